// LightBeam CPU oracle -- TEST INFRASTRUCTURE ONLY.
//
// A plain, slow, single-threaded fp64 implementation of the decoding method of
// LightBeam (arXiv 2603.14002): lexicon-constrained CTC prefix beam search
// (Alg. 1, Sec. 3.4, App. E.1-E.2) with homophone sub-beams and 4-gram backoff
// shallow fusion at word boundaries (Sec. 3.4.1, Eq. (1), App. E.3) and delayed
// fusion that replaces the word-level scores at fixed frame intervals
// (Sec. 3.4.2, Eq. (2), App. E.4).
//
// Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
// load this library.  It shares no code, header or constant table with the HIP
// decoder; prefixes are exact symbol vectors in std::map, the lexicon is a set
// of phoneme prefixes, the LM is a set of sorted tuple arrays searched by
// binary search, and every score is a double.
//
// Readings of the paper taken here (each is listed in the design notes):
//  * Recombination of equal prefixes uses log-sum-exp, with separate
//    blank-ending / non-blank-ending scores per prefix (classical CTC prefix
//    search).  A doubled phoneme (v == last symbol) extends only from the
//    blank-ending score.
//  * The token bonus beta is added once per new phoneme, the word bonus gamma
//    once per new separator, never on a stay.
//  * The n-gram LM is applied after top-K and theta pruning, to entries created
//    in this frame by a separator extension with no surviving same-prefix
//    entry ("stay wins" for word-level state).
//  * LM scores are log10 values, converted with ln(10) before the weight omega.
//  * Delayed fusion after frame t when t % I == 0 and t > 0 replaces every
//    sub-beam score of the top-F entries by phi * S_fus(words), then re-sorts
//    the sub-beams (stable); at the end a final fusion covers all entries,
//    entries inside a word are dropped if any entry ends at a word boundary
//    (else all are kept, with their completed words) and the rest are ranked.
//  * Ties are broken by a 64-bit key of the prefix (splitmix64 chain), and
//    sub-beam ties by (parent sub-beam index, word id).
//  * Options: recombination by max instead of log-sum-exp (the best alignment,
//    App. E.1); raw per-frame scores normalised by a log-softmax first;
//    lexicon entries that spell a given word id (pronunciation variants,
//    App. I; a spelling's homophones are its distinct word ids, ascending);
//    end-of-sentence marks tried at the final fusion (each sub-beam takes its
//    best mark under the synthetic scorer, the first of equals, and the mark
//    follows the output words); fusion scores from a scorer the caller passes
//    in (a function of the word sequence), in place of the synthetic one.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <map>
#include <set>
#include <string>
#include <vector>

namespace {

constexpr int kBlank = 0;
constexpr int kSep = 40;
constexpr int kClasses = 41;
constexpr int kNone = -1;
const double kNegInf = -std::numeric_limits<double>::infinity();
const double kInf = std::numeric_limits<double>::infinity();
const double kLn10 = 2.302585092994045684017991454684364208;

thread_local std::string g_err;

// log(exp(x) + exp(y)) without overflow.
double lse2(double x, double y) {
  if (x == kNegInf && y == kNegInf) return kNegInf;
  double m = x > y ? x : y;
  return m + std::log1p(std::exp(-std::fabs(x - y)));
}

double lse_list(const std::vector<double>& v) {
  double acc = kNegInf;
  for (double x : v) acc = lse2(acc, x);
  return acc;
}

// The combination of two path scores that reach the same prefix: their
// log-sum-exp (all alignments), or their maximum (the best alignment, the
// recombination of App. E.1).
double comb2(bool use_max, double x, double y) { return use_max ? std::max(x, y) : lse2(x, y); }

double comb_list(bool use_max, const std::vector<double>& v) {
  double acc = kNegInf;
  for (double x : v) acc = comb2(use_max, acc, x);
  return acc;
}

// SplitMix64 output function for state x (Steele, Lea & Flood, OOPSLA 2014):
// advance by the golden-ratio increment, then the variant-13 finaliser.
uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Tie-break key of a collapsed symbol sequence: key(()) = 0,
// key(y + v) = splitmix64(key(y) XOR v).
uint64_t prefix_key(const std::vector<int>& y) {
  uint64_t k = 0;
  for (int s : y) k = splitmix64(k ^ static_cast<uint64_t>(s));
  return k;
}

struct Params {
  int beam;
  int subbeams;
  double alpha, beta, gamma, omega, phi, theta, lam;
  int fusion_interval;  // 0 = no fusion
  int fusion_top_f;     // 0 = all entries
  int fusion_mode;      // 0 = synthetic bigram scorer, 1 = the n-gram LM's own score (pin),
                        // 2 = the caller's scorer (an external LLM stand-in)
  int finalize;         // 1 = end of utterance (final fusion, drop mid-word); 0 = rank the live beam
  int merge_max;        // 0 = contributions to a prefix combine by log-sum-exp; 1 = by max (App. E.1)
  int raw_logits;       // 0 = inputs are log-probabilities; 1 = raw scores, log-softmax per frame first
  int eos_count;        // end-of-sentence marks tried at the final fusion (synthetic scorer), 0..3
  int eos_ids[3];       // their word ids
  uint64_t fusion_seed;
  double fusion_lo, fusion_hi;
  double (*scorer)(const int32_t* words, int32_t n, void* ctx);  // fusion_mode 2
  void* scorer_ctx;
};

// ------------------------------------------------------------------ lexicon

struct Lexicon {
  std::set<std::vector<int>> prefixes;                  // every prefix of every word (incl. empty)
  std::map<std::vector<int>, std::vector<int>> words;   // phoneme string -> ascending word ids
};

// ------------------------------------------------------------------ 4-gram backoff LM

struct Order {
  int n = 0;
  int64_t count = 0;
  std::vector<int32_t> ids;  // [count][n], sorted lexicographically, unique
  std::vector<float> logp;   // log10 p
  std::vector<float> bo;     // log10 backoff (empty for the top order)

  // row of the tuple t (size n), or -1
  int64_t find(const int32_t* t) const {
    int64_t lo = 0, hi = count;
    while (lo < hi) {
      int64_t mid = lo + (hi - lo) / 2;
      const int32_t* r = &ids[static_cast<size_t>(mid) * n];
      int c = 0;
      for (int i = 0; i < n && c == 0; ++i) c = (r[i] < t[i]) ? -1 : (r[i] > t[i] ? 1 : 0);
      if (c == 0) return mid;
      if (c < 0) lo = mid + 1; else hi = mid;
    }
    return -1;
  }
};

struct LM {
  int vocab = 0, bos = 0, unk = 0;
  Order ord[4];

  // ARPA / Katz backoff query, in log10:
  //   log10 P(w | u_1..u_m) = p(u_1..u_m, w)                     if that n-gram exists
  //                         = p(w), or p(<unk>) if w is unknown     if m == 0
  //                         = bo(u_1..u_m) + log10 P(w | u_2..u_m)  otherwise (bo = 0 if absent)
  double log10p(const std::vector<int>& ctx, int w) const {
    const int m = static_cast<int>(ctx.size());
    std::vector<int32_t> t(ctx.begin(), ctx.end());
    t.push_back(w);
    int64_t r = ord[m].find(t.data());
    if (r >= 0) return static_cast<double>(ord[m].logp[r]);
    if (m == 0) {
      int32_t u = unk;
      int64_t ru = ord[0].find(&u);
      return ru >= 0 ? static_cast<double>(ord[0].logp[ru]) : kNegInf;
    }
    int64_t rc = ord[m - 1].find(ctx.data());
    double bo = rc >= 0 ? static_cast<double>(ord[m - 1].bo[rc]) : 0.0;
    std::vector<int> shorter(ctx.begin() + 1, ctx.end());
    return bo + log10p(shorter, w);
  }

  // last <= 3 words of (<s>, words...)
  std::vector<int> context(const std::vector<int>& words) const {
    std::vector<int> full;
    full.push_back(bos);
    full.insert(full.end(), words.begin(), words.end());
    size_t k = std::min<size_t>(3, full.size());
    return std::vector<int>(full.end() - k, full.end());
  }
};

struct Model {
  Lexicon lex;
  LM lm;
};

// ------------------------------------------------------------------ hypotheses

struct Sub {
  double Lw;               // cumulative word-level score (natural log, weighted)
  std::vector<int> words;  // word ids of this orthographic reading
  int eos = -1;            // end-of-sentence mark chosen at the final fusion (-1: none)
};

struct Hyp {
  std::vector<int> y;      // collapsed symbols over 1..40
  double a_b = kNegInf;    // log score of alignments ending in blank
  double a_nb = kNegInf;   // log score of alignments ending in the last symbol
  std::vector<Sub> subs;   // <= o orthographic sub-beams, best first
};

int last_symbol(const std::vector<int>& y) { return y.empty() ? kNone : y.back(); }

// Phonemes after the last separator (the word being spelled).
std::vector<int> partial_word(const std::vector<int>& y) {
  size_t i = y.size();
  while (i > 0 && y[i - 1] != kSep) --i;
  return std::vector<int>(y.begin() + i, y.end());
}

// Set once per decode: how a_b and a_nb combine into a prefix's acoustic score.
thread_local bool g_merge_max = false;
double acoustic(const Hyp& h) { return comb2(g_merge_max, h.a_b, h.a_nb); }
double total(const Hyp& h) { return acoustic(h) + h.subs[0].Lw; }

// Is symbol v (1..40) a lexicon-valid extension of a prefix whose current
// partial word is P?  Phonemes must keep P a word prefix; the separator needs
// P to be a complete (non-empty) word.
bool valid_extension(const Lexicon& lex, const std::vector<int>& P, int v) {
  if (v == kSep) return !P.empty() && lex.words.count(P) > 0;
  std::vector<int> q = P;
  q.push_back(v);
  return lex.prefixes.count(q) > 0;
}

struct Margins {
  double topk = kInf, theta = kInf, homophone = kInf, lam = kInf, fusion = kInf, ranking = kInf;
  double last_topk = kInf;  // the K-th vs (K+1)-th candidate of the last frame
};

struct Stats {
  int64_t expansions = 0, word_events = 0, lm_queries = 0, fusion_events = 0;
};

double bigram_score(const Params& p, int a, int b) {
  uint64_t h = splitmix64(p.fusion_seed ^ ((static_cast<uint64_t>(static_cast<uint32_t>(a)) << 32) |
                                           static_cast<uint64_t>(static_cast<uint32_t>(b))));
  double u = static_cast<double>(h >> 48) * (1.0 / 65536.0);
  return p.fusion_lo + (p.fusion_hi - p.fusion_lo) * u;
}

// Full-sequence fusion score of a word sequence (natural log): the seeded
// synthetic word-bigram scorer that stands in for the LLM, (mode 1) the n-gram
// LM's own ln-scaled sentence score, or (mode 2) whatever the caller's scorer
// returns for the sequence.
double fusion_score(const Model& M, const Params& p, const std::vector<int>& words) {
  if (p.fusion_mode == 2) {
    const int32_t none = 0;
    return p.scorer(words.empty() ? &none : words.data(), static_cast<int32_t>(words.size()), p.scorer_ctx);
  }
  double s = 0.0;
  if (p.fusion_mode == 1) {
    std::vector<int> prefix;
    for (int w : words) {
      s += kLn10 * M.lm.log10p(M.lm.context(prefix), w);
      prefix.push_back(w);
    }
    return s;
  }
  int prev = M.lm.bos;
  for (int w : words) {
    s += bigram_score(p, prev, w);
    prev = w;
  }
  return s;
}

// (total desc, key asc) order over hypotheses
struct Ranked {
  double total;
  uint64_t key;
  size_t idx;
};
bool ranked_before(const Ranked& a, const Ranked& b) {
  if (a.total != b.total) return a.total > b.total;
  return a.key < b.key;
}

std::vector<Ranked> rank(const std::vector<Hyp>& beam) {
  std::vector<Ranked> r;
  for (size_t i = 0; i < beam.size(); ++i) r.push_back({total(beam[i]), prefix_key(beam[i].y), i});
  std::sort(r.begin(), r.end(), ranked_before);
  return r;
}

// Delayed fusion (Eq. (2), App. E.4): the fusion score replaces the word-level
// score of every sub-beam of the selected entries; sub-beams are re-ranked.
// At the end of the utterance (final = true) each sub-beam's sequence is also
// tried with every end-of-sentence mark appended; the best mark's score is the
// sub-beam's, and the mark is kept for the output (the first of equals wins).
void apply_fusion(const Model& M, const Params& p, std::vector<Hyp>& beam, int top_f, Margins& mg,
                  Stats& st, bool final = false) {
  std::vector<Ranked> r = rank(beam);
  size_t nf = (top_f <= 0) ? r.size() : std::min<size_t>(top_f, r.size());
  if (nf < r.size()) mg.fusion = std::min(mg.fusion, r[nf - 1].total - r[nf].total);
  const bool eos = final && p.eos_count > 0 && p.fusion_mode == 0;
  for (size_t i = 0; i < nf; ++i) {
    Hyp& h = beam[r[i].idx];
    for (Sub& s : h.subs) {
      double f = fusion_score(M, p, s.words);
      if (eos) {
        const int last = s.words.empty() ? M.lm.bos : s.words.back();
        double best = kNegInf;
        for (int k = 0; k < p.eos_count; ++k) {
          const double v = bigram_score(p, last, p.eos_ids[k]);
          if (v > best) {
            best = v;
            s.eos = p.eos_ids[k];
          }
        }
        f += best;
      }
      s.Lw = p.phi * f;
    }
    std::stable_sort(h.subs.begin(), h.subs.end(),
                     [](const Sub& a, const Sub& b) { return a.Lw > b.Lw; });
    ++st.fusion_events;
  }
}

// Shallow fusion with the n-gram LM at a word boundary (Eq. (1), App. E.3):
// every (parent sub-beam, homophone) pair is scored, the top o survive, and
// survivors more than lambda below the best are dropped.
std::vector<Sub> apply_ngram(const Model& M, const Params& p, const std::vector<Sub>& parent,
                             const std::vector<int>& homophones, Margins& mg, Stats& st) {
  struct C {
    double Lw;
    int j;
    int w;
  };
  const double c_omega = p.omega * kLn10;
  std::vector<C> cand;
  for (size_t j = 0; j < parent.size(); ++j) {
    std::vector<int> ctx = M.lm.context(parent[j].words);
    for (int w : homophones) {
      double lp = M.lm.log10p(ctx, w);
      cand.push_back({parent[j].Lw + c_omega * lp, static_cast<int>(j), w});
      ++st.lm_queries;
    }
  }
  std::sort(cand.begin(), cand.end(), [](const C& a, const C& b) {
    if (a.Lw != b.Lw) return a.Lw > b.Lw;
    if (a.j != b.j) return a.j < b.j;
    return a.w < b.w;
  });
  size_t keep = std::min<size_t>(p.subbeams, cand.size());
  if (cand.size() > keep) mg.homophone = std::min(mg.homophone, cand[keep - 1].Lw - cand[keep].Lw);
  const double cut = cand[0].Lw - p.lam;
  std::vector<Sub> out;
  for (size_t i = 0; i < keep; ++i) {
    mg.lam = std::min(mg.lam, std::fabs(cand[i].Lw - cut));
    if (cand[i].Lw < cut) continue;
    Sub s;
    s.Lw = cand[i].Lw;
    s.words = parent[cand[i].j].words;
    s.words.push_back(cand[i].w);
    out.push_back(std::move(s));
  }
  return out;
}

struct Output {
  std::vector<Hyp> hyps;  // ranked
  Margins mg;
  Stats st;
  std::vector<double> frame_lse;
};

Output decode(const Model& M, const Params& p, const float* logits, int T, bool want_frame_lse) {
  Output out;
  std::vector<Hyp> beam(1);
  beam[0].y = {};
  beam[0].a_b = 0.0;
  beam[0].a_nb = kNegInf;
  beam[0].subs = {Sub{0.0, {}}};

  g_merge_max = p.merge_max != 0;
  const bool mx = g_merge_max;
  for (int t = 0; t < T; ++t) {
    double D[kClasses];
    double lp[kClasses];
    for (int v = 0; v < kClasses; ++v) lp[v] = static_cast<double>(logits[t * kClasses + v]);
    if (p.raw_logits) {
      // log-softmax over the frame's classes
      double m = kNegInf;
      for (int v = 0; v < kClasses; ++v) m = std::max(m, lp[v]);
      double s = 0.0;
      for (int v = 0; v < kClasses; ++v) s += std::exp(lp[v] - m);
      const double ls = std::log(s);
      for (int v = 0; v < kClasses; ++v) lp[v] = (lp[v] - m) - ls;
    }
    for (int v = 0; v < kClasses; ++v) D[v] = p.alpha * lp[v];
    out.st.expansions += static_cast<int64_t>(beam.size()) * kClasses;

    // Fan-out (Alg. 1): every entry stays (blank / repeated last symbol) or
    // extends by a lexicon-valid symbol.  Contributions to one prefix are
    // collected per prefix and merged by log-sum-exp.
    struct Cand {
      std::vector<double> b, nb;
      const Hyp* stay = nullptr;
      const Hyp* ext = nullptr;
      int ext_v = kNone;
    };
    std::map<std::vector<int>, Cand> C;
    for (const Hyp& h : beam) {
      const double pr = comb2(mx, h.a_b, h.a_nb);
      const int last = last_symbol(h.y);
      Cand& cs = C[h.y];
      cs.b.push_back(pr + D[kBlank]);
      if (last != kNone) cs.nb.push_back(h.a_nb + D[last]);
      cs.stay = &h;
      const std::vector<int> P = partial_word(h.y);
      for (int v = 1; v <= kSep; ++v) {
        if (!valid_extension(M.lex, P, v)) continue;
        std::vector<int> y2 = h.y;
        y2.push_back(v);
        const double base = (v == last) ? h.a_b : pr;
        const double bonus = (v == kSep) ? p.gamma : p.beta;
        Cand& ce = C[y2];
        ce.nb.push_back((base + D[v]) + bonus);
        ce.ext = &h;
        ce.ext_v = v;
      }
    }

    // Merge, then select the top K by (total desc, key asc) and prune by theta.
    struct Merged {
      const std::vector<int>* y;
      const Cand* c;
      double a_b, a_nb, total;
      uint64_t key;
    };
    std::vector<Merged> ms;
    for (const auto& kv : C) {
      Merged m;
      m.y = &kv.first;
      m.c = &kv.second;
      m.a_b = comb_list(mx, kv.second.b);
      m.a_nb = comb_list(mx, kv.second.nb);
      const Hyp* src = kv.second.stay ? kv.second.stay : kv.second.ext;
      m.total = comb2(mx, m.a_b, m.a_nb) + src->subs[0].Lw;
      m.key = prefix_key(kv.first);
      if (m.total == kNegInf) continue;
      ms.push_back(m);
    }
    std::sort(ms.begin(), ms.end(), [](const Merged& a, const Merged& b) {
      if (a.total != b.total) return a.total > b.total;
      return a.key < b.key;
    });
    size_t keep = std::min<size_t>(p.beam, ms.size());
    if (ms.size() > keep) out.mg.topk = std::min(out.mg.topk, ms[keep - 1].total - ms[keep].total);
    out.mg.last_topk = ms.size() > keep ? ms[keep - 1].total - ms[keep].total : kInf;
    const double cut = ms.empty() ? kNegInf : ms[0].total - p.theta;

    std::vector<Hyp> next;
    for (size_t i = 0; i < keep; ++i) {
      const Merged& m = ms[i];
      out.mg.theta = std::min(out.mg.theta, std::fabs(m.total - cut));
      if (m.total < cut) continue;
      Hyp h;
      h.y = *m.y;
      h.a_b = m.a_b;
      h.a_nb = m.a_nb;
      if (m.c->stay) {
        h.subs = m.c->stay->subs;
      } else if (m.c->ext_v == kSep) {
        // New word: homophones of the word just completed.
        std::vector<int> word(m.y->begin(), m.y->end() - 1);
        word = partial_word(word);
        const std::vector<int>& homs = M.lex.words.at(word);
        ++out.st.word_events;
        h.subs = apply_ngram(M, p, m.c->ext->subs, homs, out.mg, out.st);
      } else {
        h.subs = m.c->ext->subs;
      }
      next.push_back(std::move(h));
    }
    beam.swap(next);

    if (p.fusion_interval > 0 && t % p.fusion_interval == 0 && t > 0)
      apply_fusion(M, p, beam, p.fusion_top_f, out.mg, out.st);

    if (want_frame_lse) {
      double acc = kNegInf;
      for (const Hyp& h : beam) acc = lse2(acc, lse2(h.a_b, h.a_nb));
      out.frame_lse.push_back(acc);
    }
  }

  // End of the utterance: final fusion over every entry; entries that stop
  // inside a word are dropped when at least one entry ends at a word boundary
  // (otherwise every entry is kept, with its completed words); the rest are
  // ranked.  Without finalisation the live beam is ranked as it stands (the
  // state a streaming decoder reports mid-stream).
  if (p.finalize && p.fusion_interval > 0) apply_fusion(M, p, beam, 0, out.mg, out.st, true);
  bool any_complete = false;
  for (const Hyp& h : beam) any_complete = any_complete || partial_word(h.y).empty();
  std::vector<Hyp> done;
  for (Hyp& h : beam)
    if (!p.finalize || !any_complete || partial_word(h.y).empty()) done.push_back(std::move(h));
  std::vector<Ranked> r = rank(done);
  for (size_t i = 0; i + 1 < r.size(); ++i)
    out.mg.ranking = std::min(out.mg.ranking, r[i].total - r[i + 1].total);
  for (const Ranked& x : r) out.hyps.push_back(done[x.idx]);
  return out;
}

}  // namespace

// ------------------------------------------------------------------ C API (for ctypes)

extern "C" {

struct orc_params {
  int32_t beam;
  int32_t subbeams;
  double alpha, beta, gamma, omega, phi, theta, lam;
  int32_t fusion_interval;
  int32_t fusion_top_f;
  int32_t fusion_mode;
  int32_t finalize;
  int32_t merge_max;
  int32_t raw_logits;
  int32_t eos_count;
  int32_t eos_ids[3];
  uint64_t fusion_seed;
  double fusion_lo, fusion_hi;
  double (*scorer)(const int32_t* words, int32_t n, void* ctx);  // fusion_mode 2
  void* scorer_ctx;
};

const char* orc_last_error(void) { return g_err.c_str(); }

// Builds the lexicon sets and copies the LM.  Each order's tuples must be
// sorted lexicographically and unique (checked).  Returns NULL on error.
// Lexicon: n_entries pronunciations (CSR lex_offsets / lex_phonemes); entry e
// spells word entry_word[e] (entry_word NULL: word e).
void* orc_create(int32_t n_entries, const int32_t* lex_offsets, const int32_t* lex_phonemes, const int32_t* entry_word,
                 int32_t vocab_size, int32_t bos_id, int32_t unk_id, const int64_t* counts,
                 const int32_t* ids1, const float* p1, const float* bo1,
                 const int32_t* ids2, const float* p2, const float* bo2,
                 const int32_t* ids3, const float* p3, const float* bo3,
                 const int32_t* ids4, const float* p4) {
  Model* M = new Model();
  for (int32_t e = 0; e < n_entries; ++e) {
    std::vector<int> ph(lex_phonemes + lex_offsets[e], lex_phonemes + lex_offsets[e + 1]);
    if (ph.empty()) {
      g_err = "empty word";
      delete M;
      return nullptr;
    }
    for (size_t k = 0; k <= ph.size(); ++k) M->lex.prefixes.insert(std::vector<int>(ph.begin(), ph.begin() + k));
    M->lex.words[ph].push_back(entry_word ? entry_word[e] : e);
  }
  // homophones of a spelling: distinct word ids, ascending
  for (auto& kv : M->lex.words) {
    std::sort(kv.second.begin(), kv.second.end());
    kv.second.erase(std::unique(kv.second.begin(), kv.second.end()), kv.second.end());
  }
  M->lm.vocab = vocab_size;
  M->lm.bos = bos_id;
  M->lm.unk = unk_id;
  const int32_t* ids[4] = {ids1, ids2, ids3, ids4};
  const float* lp[4] = {p1, p2, p3, p4};
  const float* bo[4] = {bo1, bo2, bo3, nullptr};
  for (int n = 1; n <= 4; ++n) {
    Order& o = M->lm.ord[n - 1];
    o.n = n;
    o.count = counts[n - 1];
    o.ids.assign(ids[n - 1], ids[n - 1] + o.count * n);
    o.logp.assign(lp[n - 1], lp[n - 1] + o.count);
    if (n < 4) o.bo.assign(bo[n - 1], bo[n - 1] + o.count);
    for (int64_t i = 1; i < o.count; ++i) {
      const int32_t* a = &o.ids[(i - 1) * n];
      const int32_t* b = &o.ids[i * n];
      if (!std::lexicographical_compare(a, a + n, b, b + n)) {
        g_err = "order " + std::to_string(n) + " not sorted/unique at row " + std::to_string(i);
        delete M;
        return nullptr;
      }
    }
  }
  return M;
}

void orc_destroy(void* h) { delete static_cast<Model*>(h); }

static Params to_params(const orc_params* q) {
  Params p;
  p.beam = q->beam;
  p.subbeams = q->subbeams;
  p.alpha = q->alpha;
  p.beta = q->beta;
  p.gamma = q->gamma;
  p.omega = q->omega;
  p.phi = q->phi;
  p.theta = q->theta;
  p.lam = q->lam;
  p.fusion_interval = q->fusion_interval;
  p.fusion_top_f = q->fusion_top_f;
  p.fusion_mode = q->fusion_mode;
  p.finalize = q->finalize;
  p.merge_max = q->merge_max;
  p.raw_logits = q->raw_logits;
  p.eos_count = q->eos_count;
  for (int k = 0; k < 3; ++k) p.eos_ids[k] = q->eos_ids[k];
  p.fusion_seed = q->fusion_seed;
  p.fusion_lo = q->fusion_lo;
  p.fusion_hi = q->fusion_hi;
  p.scorer = q->scorer;
  p.scorer_ctx = q->scorer_ctx;
  return p;
}

// Decodes one utterance of T frames (logits float32 [T][41], log-softmax).
// Writes up to max_hyps ranked hypotheses; returns how many were produced
// (before truncation to max_hyps), or -1 on error.
//   out_words [max_hyps][max_words] / out_nwords: best sub-beam's word ids
//   out_total, out_acoustic: total score and its acoustic part (fp64)
//   out_labels [max_hyps][max_labels] / out_nlabels: collapsed symbol sequence
//   out_keys: 64-bit prefix key of each hypothesis
//   out_margins [7]: min decision margins (top-K, theta, top-o, lambda, top-F, ranking)
//                    and the last frame's top-K margin
//   out_frame_lse [T] (optional): log-sum-exp of the beam's acoustic scores after each frame
//   out_stats [4]: expansions, word events, LM queries, fused entries
//   (optional, with max_subs > 0) every sub-beam of each hypothesis, best first:
//   out_nsub [max_hyps], out_sub_L [max_hyps][max_subs] word-level scores,
//   out_sub_nw [max_hyps][max_subs] and out_sub_words [max_hyps][max_subs][max_words]
int32_t orc_decode(void* h, const orc_params* q, const float* logits, int32_t T, int32_t max_hyps,
                   int32_t max_words, int32_t max_labels, int32_t* out_words, int32_t* out_nwords,
                   double* out_total, double* out_acoustic, int32_t* out_labels,
                   int32_t* out_nlabels, uint64_t* out_keys, double* out_margins,
                   double* out_frame_lse, int64_t* out_stats, int32_t max_subs, int32_t* out_nsub,
                   double* out_sub_L, int32_t* out_sub_nw, int32_t* out_sub_words) {
  if (!h || !q || !logits || T < 0 || q->beam < 1 || q->subbeams < 1 || q->fusion_mode < 0 ||
      q->fusion_mode > 2 || (q->fusion_mode == 2 && !q->scorer)) {
    g_err = "invalid argument";
    return -1;
  }
  const Model& M = *static_cast<const Model*>(h);
  Params p = to_params(q);
  Output o = decode(M, p, logits, T, out_frame_lse != nullptr);
  const int32_t n = static_cast<int32_t>(o.hyps.size());
  for (int32_t i = 0; i < n && i < max_hyps; ++i) {
    const Hyp& x = o.hyps[i];
    std::vector<int> ws = x.subs[0].words;
    if (x.subs[0].eos >= 0) ws.push_back(x.subs[0].eos);
    if (out_nwords) out_nwords[i] = static_cast<int32_t>(ws.size());
    if (out_words)
      for (int32_t k = 0; k < max_words; ++k)
        out_words[static_cast<int64_t>(i) * max_words + k] = k < static_cast<int32_t>(ws.size()) ? ws[k] : -1;
    if (out_total) out_total[i] = total(x);
    if (out_acoustic) out_acoustic[i] = acoustic(x);
    if (out_nlabels) out_nlabels[i] = static_cast<int32_t>(x.y.size());
    if (out_labels)
      for (int32_t k = 0; k < max_labels; ++k)
        out_labels[static_cast<int64_t>(i) * max_labels + k] = k < static_cast<int32_t>(x.y.size()) ? x.y[k] : -1;
    if (out_keys) out_keys[i] = prefix_key(x.y);
    if (max_subs > 0 && out_nsub) {
      const int32_t ns = std::min<int32_t>(max_subs, static_cast<int32_t>(x.subs.size()));
      out_nsub[i] = ns;
      for (int32_t j = 0; j < ns; ++j) {
        const Sub& sb = x.subs[j];
        const int64_t r = static_cast<int64_t>(i) * max_subs + j;
        if (out_sub_L) out_sub_L[r] = sb.Lw;
        if (out_sub_nw) out_sub_nw[r] = static_cast<int32_t>(sb.words.size());
        if (out_sub_words)
          for (int32_t k = 0; k < max_words; ++k)
            out_sub_words[r * max_words + k] = k < static_cast<int32_t>(sb.words.size()) ? sb.words[k] : -1;
      }
    }
  }
  if (out_margins) {
    const double m[7] = {o.mg.topk, o.mg.theta, o.mg.homophone, o.mg.lam, o.mg.fusion, o.mg.ranking,
                         o.mg.last_topk};
    std::memcpy(out_margins, m, sizeof(m));
  }
  if (out_frame_lse)
    for (int32_t t = 0; t < T; ++t) out_frame_lse[t] = o.frame_lse[t];
  if (out_stats) {
    out_stats[0] = o.st.expansions;
    out_stats[1] = o.st.word_events;
    out_stats[2] = o.st.lm_queries;
    out_stats[3] = o.st.fusion_events;
  }
  return n;
}

// log10 P(w | ctx) by the backoff rule (ctx: up to 3 words, oldest first).
double orc_log10p(void* h, const int32_t* ctx, int32_t n_ctx, int32_t w) {
  const Model& M = *static_cast<const Model*>(h);
  std::vector<int> c(ctx, ctx + n_ctx);
  return M.lm.log10p(c, w);
}

// Fusion score of a word sequence under the parameters' fusion mode.
double orc_fusion_score(void* h, const orc_params* q, const int32_t* words, int32_t n) {
  const Model& M = *static_cast<const Model*>(h);
  Params p = to_params(q);
  if (p.fusion_mode == 2 && !p.scorer) return std::numeric_limits<double>::quiet_NaN();
  return fusion_score(M, p, std::vector<int>(words, words + n));
}

uint64_t orc_splitmix64(uint64_t x) { return splitmix64(x); }

uint64_t orc_prefix_key(const int32_t* y, int32_t n) {
  return prefix_key(std::vector<int>(y, y + n));
}

}  // extern "C"
