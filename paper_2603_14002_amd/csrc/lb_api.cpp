// C ABI of the LightBeam gfx950 decoder: validation, one-time table build and
// upload, buffer allocation, and the per-frame launch sequence of Alg. 1.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/lightbeam.h"
#include "lb_device.h"
#include "lb_launch.h"

using namespace lb;

static_assert(sizeof(lb_params) == 160, "lb_params layout");
static_assert(sizeof(lb_ngram_desc) == 144, "lb_ngram_desc layout");
static_assert(sizeof(lb_lexicon_desc) == 32, "lb_lexicon_desc layout");
static_assert(sizeof(lb_stats) == 320, "lb_stats layout");

namespace {

thread_local std::string g_err;

lb_status fail(lb_status st, const std::string& msg) {
  g_err = msg;
  return st;
}

#define LB_HIP(call)                                                                  \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess)                                                             \
      return fail(e_ == hipErrorOutOfMemory ? LB_ERR_OUT_OF_MEMORY : LB_ERR_HIP,      \
                  std::string(#call) + ": " + hipGetErrorString(e_));                 \
  } while (0)

// Lexicon trie flattened to CSR in breadth-first order, so that the children
// of a node are contiguous and ordered by phoneme (App. E.2 flattens the trie
// into a transition table; a child bitmask + first-child index gives the same
// transitions in 16 B per node).
struct HostTrie {
  std::vector<TrieNode> nodes;  // + sentinel
  std::vector<int32_t> words;
  uint32_t max_homophones = 0;
};

HostTrie build_trie(const lb_lexicon_desc& lex) {
  std::vector<std::array<int32_t, 40>> ch(1);
  ch[0].fill(-1);
  std::vector<std::vector<int32_t>> at(1);
  for (int32_t w = 0; w < lex.n_entries; ++w) {
    int32_t n = 0;
    for (int32_t k = lex.offsets[w]; k < lex.offsets[w + 1]; ++k) {
      const int p = lex.phonemes[k];
      if (ch[n][p] < 0) {
        ch[n][p] = static_cast<int32_t>(ch.size());
        ch.emplace_back();
        ch.back().fill(-1);
        at.emplace_back();
      }
      n = ch[n][p];
    }
    at[n].push_back(lex.entry_word ? lex.entry_word[w] : w);
  }
  // a node's words: distinct ids, ascending (two entries of one word may share a spelling)
  for (auto& v : at) {
    std::sort(v.begin(), v.end());
    v.erase(std::unique(v.begin(), v.end()), v.end());
  }
  const size_t N = ch.size();
  std::vector<int32_t> order;  // BFS order of old ids
  std::vector<int32_t> newid(N, -1);
  order.reserve(N);
  order.push_back(0);
  newid[0] = 0;
  for (size_t h = 0; h < order.size(); ++h) {
    const int32_t o = order[h];
    for (int p = 1; p <= 39; ++p) {
      const int32_t c = ch[o][p];
      if (c >= 0) {
        newid[c] = static_cast<int32_t>(order.size());
        order.push_back(c);
      }
    }
  }
  HostTrie t;
  t.nodes.resize(N + 1);
  uint32_t woff = 0;
  for (size_t k = 0; k < N; ++k) {
    const int32_t o = order[k];
    TrieNode& tn = t.nodes[k];
    tn.mask = 0;
    tn.first_child = 0;
    bool first = true;
    for (int p = 1; p <= 39; ++p) {
      if (ch[o][p] >= 0) {
        tn.mask |= 1ull << p;
        if (first) {
          tn.first_child = static_cast<uint32_t>(newid[ch[o][p]]);
          first = false;
        }
      }
    }
    if (k != 0 && !at[o].empty()) tn.mask |= 1ull << kSep;
    tn.mask |= static_cast<uint64_t>(at[o].size()) << kWordCountShift;
    tn.word_off = woff;
    t.max_homophones = std::max<uint32_t>(t.max_homophones, static_cast<uint32_t>(at[o].size()));
    for (int32_t w : at[o]) t.words.push_back(w);
    woff += static_cast<uint32_t>(at[o].size());
  }
  t.nodes[N].mask = 0;
  t.nodes[N].first_child = 0;
  t.nodes[N].word_off = woff;
  return t;
}

uint64_t buckets_for(int64_t count, double lf) {
  if (count <= 0) return 1;
  const double slots = std::ceil(static_cast<double>(count) / lf);
  return std::max<uint64_t>(1, static_cast<uint64_t>(std::ceil(slots / 4.0)));
}

struct EventPair {
  hipEvent_t a, b;
  int kind;
};

// kernel kinds of lb_stats.launches / kernel_ms
enum { kKindDecode = 0, kKindOutput = 1, kKindFuseSelect = 2, kKindFuseExport = 3, kKindFuseApply = 4, kKindBegin = 5,
       kKinds = 8 };

}  // namespace

struct lb_decoder {
  lb_params p{};
  DevParams P{};
  DevState S{};
  KArgs* dargs = nullptr;  // device copy of P and S for the decode kernel
  void* static_scratch = nullptr;  // this device's static lookup scratch (lb_decode_batch_noalloc)
  int block = 64;       // workgroup size of the fusion / output kernels (>= beam)
  std::vector<void*> allocs;
  int64_t launches[kKinds] = {};
  uint32_t profile_mask = 0;  // kernel kinds timed with HIP events (bit k = kind k), LB_PROFILE_PHASES
  // the decode kernel's options
  uint32_t decode_opts() const { return (profile_mask & LB_PROFILE_PHASES) ? kOptPhaseTimers : 0u; }
  std::vector<EventPair> pending;
  std::vector<hipEvent_t> pool;
  double kernel_ms[kKinds] = {};
  int64_t timed[kKinds] = {};
  // external fusion round trip (LB_FUSION_EXTERNAL): host mirrors of the
  // streams' frame counters and the state of an interrupted decode call
  struct {
    int pending = 0;  // 0 none, 1 fusion frame, 2 end of utterance
    bool in_call = false, requested = false, final_done = false;
    int32_t resume_tau = 0;
    const float* logits = nullptr;
    const int32_t* lengths = nullptr;
    int32_t B = 0, Tc = 0;
    uint32_t flags = 0;
    std::vector<int64_t> t0;
    std::vector<int32_t> len, flag;
    int32_t* d_flag = nullptr;
  } ext;

  template <typename T>
  lb_status alloc(T** ptr, size_t count) {
    void* q = nullptr;
    const size_t bytes = std::max<size_t>(count, 1) * sizeof(T);
    hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess)
      return fail(LB_ERR_OUT_OF_MEMORY, "hipMalloc(" + std::to_string(bytes) + " B) failed: " + hipGetErrorString(e));
    allocs.push_back(q);
    *ptr = static_cast<T*>(q);
    return LB_OK;
  }

  hipEvent_t get_event() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }

  void harvest() {
    for (EventPair& ep : pending) {
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, ep.a, ep.b) == hipSuccess) {
        kernel_ms[ep.kind] += ms;
        timed[ep.kind] += 1;
      } else {
        (void)hipGetLastError();  // an unusable pair is skipped; leave no error behind for the caller
      }
      pool.push_back(ep.a);
      pool.push_back(ep.b);
    }
    pending.clear();
  }

  ~lb_decoder() {
    for (EventPair& ep : pending) {
      (void)hipEventDestroy(ep.a);
      (void)hipEventDestroy(ep.b);
    }
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
    for (void* q : allocs) (void)hipFree(q);
  }
};

namespace {

lb_status validate(const lb_lexicon_desc* lex, const lb_ngram_desc* lm, const lb_params* p) {
  if (!lex || !lm || !p) return fail(LB_ERR_INVALID_ARG, "null descriptor");
  if (lex->n_entries < 1 || !lex->offsets || !lex->phonemes) return fail(LB_ERR_INVALID_ARG, "empty lexicon");
  if (lex->offsets[0] != 0) return fail(LB_ERR_INVALID_ARG, "lexicon offsets[0] != 0");
  for (int32_t w = 0; w < lex->n_entries; ++w) {
    if (lex->offsets[w + 1] <= lex->offsets[w])
      return fail(LB_ERR_INVALID_ARG, "word " + std::to_string(w) + " has no phonemes");
    for (int32_t k = lex->offsets[w]; k < lex->offsets[w + 1]; ++k)
      if (lex->phonemes[k] < 1 || lex->phonemes[k] > 39)
        return fail(LB_ERR_INVALID_ARG, "phoneme out of 1..39 in word " + std::to_string(w));
  }
  if (lex->entry_word) {
    for (int32_t e = 0; e < lex->n_entries; ++e)
      if (lex->entry_word[e] < 0 || lex->entry_word[e] >= lm->vocab_size)
        return fail(LB_ERR_INVALID_ARG, "entry " + std::to_string(e) + ": word id outside the LM vocabulary");
  } else if (lm->vocab_size < lex->n_entries + 1) {
    return fail(LB_ERR_INVALID_ARG, "LM vocabulary smaller than the lexicon");
  }
  if (lm->bos_id < 0 || lm->bos_id >= lm->vocab_size || lm->unk_id < 0 || lm->unk_id >= lm->vocab_size)
    return fail(LB_ERR_INVALID_ARG, "bos/unk id out of range");
  for (int n = 0; n < 4; ++n) {
    if (lm->count[n] < 0) return fail(LB_ERR_INVALID_ARG, "negative n-gram count");
    if (lm->count[n] > 0 && (!lm->ids[n] || !lm->log10p[n] || (n < 3 && !lm->backoff[n])))
      return fail(LB_ERR_INVALID_ARG, "missing n-gram arrays for order " + std::to_string(n + 1));
  }
  if (p->beam < 1 || p->beam > LB_MAX_BEAM) return fail(LB_ERR_INVALID_ARG, "beam must be in 1..256");
  if (p->subbeams < 1 || p->subbeams > LB_MAX_SUBBEAMS) return fail(LB_ERR_INVALID_ARG, "subbeams must be in 1..4");
  if (p->max_batch < 1 || p->max_frames < 1 || p->max_words_out < 1)
    return fail(LB_ERR_INVALID_ARG, "max_batch, max_frames and max_words_out must be >= 1");
  if (p->fusion_source < LB_FUSION_NONE || p->fusion_source > LB_FUSION_EXTERNAL)
    return fail(LB_ERR_INVALID_ARG, "unknown fusion_source");
  if (p->fusion_source != LB_FUSION_NONE && p->fusion_interval < 1)
    return fail(LB_ERR_INVALID_ARG, "fusion needs fusion_interval >= 1");
  if (p->merge != LB_MERGE_LOGSUMEXP && p->merge != LB_MERGE_MAX)
    return fail(LB_ERR_INVALID_ARG, "merge must be LB_MERGE_LOGSUMEXP or LB_MERGE_MAX");
  if (p->input != LB_INPUT_LOGPROBS && p->input != LB_INPUT_LOGITS)
    return fail(LB_ERR_INVALID_ARG, "input must be LB_INPUT_LOGPROBS or LB_INPUT_LOGITS");
  if (p->fusion_top_f < 0) return fail(LB_ERR_INVALID_ARG, "fusion_top_f < 0");
  if (p->eos_count < 0 || p->eos_count > 3) return fail(LB_ERR_INVALID_ARG, "eos_count must be in 0..3");
  if (p->eos_count > 0 && p->fusion_source != LB_FUSION_SYNTH_BIGRAM)
    return fail(LB_ERR_INVALID_ARG, "end-of-sentence marks are scored by the synthetic fusion scorer only");
  for (int k = 0; k < p->eos_count; ++k)
    if (p->eos_ids[k] < 0 || p->eos_ids[k] >= lm->vocab_size)
      return fail(LB_ERR_INVALID_ARG, "eos_ids outside the LM vocabulary");
  const double lf = p->lm_load_factor == 0.0 ? 0.25 : p->lm_load_factor;
  if (!(lf > 0.0 && lf <= 0.9)) return fail(LB_ERR_INVALID_ARG, "lm_load_factor must be in (0, 0.9]");
  for (double x : {p->alpha, p->beta, p->gamma, p->omega, p->phi, p->theta, p->lambda, p->fusion_lo, p->fusion_hi})
    if (!std::isfinite(x)) return fail(LB_ERR_INVALID_ARG, "non-finite parameter");
  if (p->theta < 0 || p->lambda < 0) return fail(LB_ERR_INVALID_ARG, "theta and lambda must be >= 0");
  if (p->arena_nodes_per_stream < 0) return fail(LB_ERR_INVALID_ARG, "arena_nodes_per_stream < 0");
  return LB_OK;
}

// Explicit-continuation index of one order: entries (key = context id << 32 |
// node word offset, homophone index) grouped by key into an open-addressing
// table with the n-gram tables' bucket layout, probe order and load factor.
struct PresEntry {
  uint64_t key;
  uint32_t h;
  bool operator<(const PresEntry& o) const { return key != o.key ? key < o.key : h < o.h; }
};

lb_status upload_pres(lb_decoder* d, std::vector<PresEntry>& ent, double lf, PresTable* out) {
  lb_status st;
  std::sort(ent.begin(), ent.end());
  ent.erase(std::unique(ent.begin(), ent.end(),
                        [](const PresEntry& a, const PresEntry& b) { return a.key == b.key && a.h == b.h; }),
            ent.end());
  size_t nkeys = 0;
  for (size_t i = 0; i < ent.size(); ++i) nkeys += (i == 0 || ent[i].key != ent[i - 1].key) ? 1 : 0;
  const uint64_t nb = buckets_for(static_cast<int64_t>(nkeys), lf);
  std::vector<PresSlot> slots(nb * 4, PresSlot{kEmptyKey, 0, 0});
  std::vector<uint32_t> lists;
  for (size_t i = 0; i < ent.size();) {
    size_t j = i;
    while (j < ent.size() && ent[j].key == ent[i].key) ++j;
    const uint32_t n = static_cast<uint32_t>(j - i);
    uint32_t a = ent[i].h;
    if (n > 1) {
      a = static_cast<uint32_t>(lists.size());
      for (size_t k = i; k < j; ++k) lists.push_back(ent[k].h);
    }
    uint64_t bk = bucket_of(ent[i].key, nb);
    for (;;) {
      int s = 0;
      while (s < 4 && slots[bk * 4 + s].key != kEmptyKey) ++s;
      if (s < 4) {
        slots[bk * 4 + s] = PresSlot{ent[i].key, a, n};
        break;
      }
      bk = (bk + 1 == nb) ? 0 : bk + 1;
    }
    i = j;
  }
  if (lists.size() >= 0xFFFFFFFFull) return fail(LB_ERR_CAPACITY, "continuation index too large");
  PresSlot* ds = nullptr;
  uint32_t* dl = nullptr;
  if ((st = d->alloc(&ds, slots.size())) != LB_OK) return st;
  if ((st = d->alloc(&dl, lists.size())) != LB_OK) return st;
  LB_HIP(hipMemcpy(ds, slots.data(), slots.size() * sizeof(PresSlot), hipMemcpyHostToDevice));
  if (!lists.empty()) LB_HIP(hipMemcpy(dl, lists.data(), lists.size() * sizeof(uint32_t), hipMemcpyHostToDevice));
  out->slots = ds;
  out->nbuckets = nb;
  out->lists = dl;
  return LB_OK;
}

lb_status build_tables(lb_decoder* d, const HostTrie& trie, const lb_ngram_desc* lm, double lf,
                       uint32_t heavy_min) {
  lb_status st;
  // trie
  TrieNode* dtrie = nullptr;
  int32_t* dwords = nullptr;
  if ((st = d->alloc(&dtrie, trie.nodes.size())) != LB_OK) return st;
  if ((st = d->alloc(&dwords, trie.words.size())) != LB_OK) return st;
  LB_HIP(hipMemcpy(dtrie, trie.nodes.data(), trie.nodes.size() * sizeof(TrieNode), hipMemcpyHostToDevice));
  LB_HIP(hipMemcpy(dwords, trie.words.data(), trie.words.size() * sizeof(int32_t), hipMemcpyHostToDevice));
  d->S.trie = dtrie;
  d->S.trie_words = dwords;

  // unigrams, dense by id; ids without an entry score as <unk> with backoff 0
  const int32_t V = lm->vocab_size;
  std::vector<Unigram> uni(V);
  float p_unk = -HUGE_VALF;
  for (int64_t e = 0; e < lm->count[0]; ++e)
    if (lm->ids[0][e] == lm->unk_id) p_unk = lm->log10p[0][e];
  for (int32_t v = 0; v < V; ++v) uni[v] = Unigram{p_unk, 0.0f};
  for (int64_t e = 0; e < lm->count[0]; ++e) {
    const int32_t v = lm->ids[0][e];
    if (v < 0 || v >= V) return fail(LB_ERR_INVALID_ARG, "unigram id out of range");
    uni[v] = Unigram{lm->log10p[0][e], lm->backoff[0][e]};
  }
  Unigram* duni = nullptr;
  if ((st = d->alloc(&duni, V)) != LB_OK) return st;
  LB_HIP(hipMemcpy(duni, uni.data(), V * sizeof(Unigram), hipMemcpyHostToDevice));
  d->S.uni = duni;

  // each node's words in (unigram log10 p desc, index asc) order, and, for the
  // heavy nodes, every (node, index) a word id occupies
  std::vector<WordRank> wrank(trie.words.size());
  std::vector<uint32_t> mem_off(static_cast<size_t>(V) + 1, 0);
  std::vector<std::pair<uint32_t, uint32_t>> mem;  // (node word offset, index) by word id
  for (size_t k = 0; k + 1 < trie.nodes.size(); ++k) {
    const uint32_t wo = trie.nodes[k].word_off;
    const uint32_t H = static_cast<uint32_t>(trie.nodes[k].mask >> kWordCountShift);
    for (uint32_t h = 0; h < H; ++h) {
      const int32_t w = trie.words[wo + h];
      wrank[wo + h] = WordRank{w, uni[w].logp, uni[w].bo, h};
      if (H >= heavy_min) mem_off[static_cast<size_t>(w) + 1] += 1;
    }
    std::stable_sort(wrank.begin() + wo, wrank.begin() + wo + H,
                     [](const WordRank& a, const WordRank& b) { return a.logp > b.logp; });
  }
  for (int32_t v = 0; v < V; ++v) mem_off[v + 1] += mem_off[v];
  mem.resize(mem_off[V]);
  {
    std::vector<uint32_t> fill(mem_off.begin(), mem_off.end() - 1);
    for (size_t k = 0; k + 1 < trie.nodes.size(); ++k) {
      const uint32_t wo = trie.nodes[k].word_off;
      const uint32_t H = static_cast<uint32_t>(trie.nodes[k].mask >> kWordCountShift);
      if (H < heavy_min) continue;
      for (uint32_t h = 0; h < H; ++h) mem[fill[trie.words[wo + h]]++] = {wo, h};
    }
  }
  WordRank* dwrank = nullptr;
  if ((st = d->alloc(&dwrank, wrank.size())) != LB_OK) return st;
  LB_HIP(hipMemcpy(dwrank, wrank.data(), wrank.size() * sizeof(WordRank), hipMemcpyHostToDevice));
  d->S.wrank = dwrank;
  const bool any_heavy = !mem.empty();
  std::vector<PresEntry> pres[3];
  // an n-gram (context id, w) marks w at each heavy node that holds it
  auto mark = [&](int n, uint32_t ctx, int32_t w) {
    if (w < 0 || w >= V) return;
    for (uint32_t m = mem_off[w]; m < mem_off[w + 1]; ++m)
      pres[n - 2].push_back(PresEntry{(static_cast<uint64_t>(ctx) << 32) | mem[m].first, mem[m].second});
  };

  // orders 2..4: open-addressing tables filled on the device
  NgramTable* tabs[3] = {&d->S.t2, &d->S.t3, &d->S.t4};
  for (int n = 2; n <= 4; ++n) {
    const uint64_t nb = buckets_for(lm->count[n - 1], lf);
    if (nb * 4 >= 0xFFFFFFFFull) return fail(LB_ERR_CAPACITY, "n-gram table too large for 32-bit slot ids");
    Slot* slots = nullptr;
    if ((st = d->alloc(&slots, nb * 4)) != LB_OK) return st;
    LB_HIP(hipMemset(slots, 0xFF, nb * 4 * sizeof(Slot)));
    tabs[n - 2]->slots = slots;
    tabs[n - 2]->nbuckets = nb;
  }
  uint32_t* dflags = d->S.flags;
  const int64_t kChunk = 1 << 24;
  int32_t* sids = nullptr;
  float* slp = nullptr;
  float* sbo = nullptr;
  uint32_t* sctx = nullptr;
  int64_t maxc = 0;
  for (int n = 2; n <= 4; ++n) maxc = std::max(maxc, lm->count[n - 1]);
  const int64_t chunk = std::min<int64_t>(kChunk, std::max<int64_t>(maxc, 1));
  LB_HIP(hipMalloc(&sids, chunk * 4 * sizeof(int32_t)));
  LB_HIP(hipMalloc(&slp, chunk * sizeof(float)));
  LB_HIP(hipMalloc(&sbo, chunk * sizeof(float)));
  LB_HIP(hipMalloc(&sctx, chunk * sizeof(uint32_t)));
  std::vector<uint32_t> hctx;
  hipError_t err = hipSuccess;
  for (int n = 2; n <= 4 && err == hipSuccess; ++n) {
    const int64_t cnt = lm->count[n - 1];
    for (int64_t s = 0; s < cnt && err == hipSuccess; s += chunk) {
      const int64_t m = std::min(chunk, cnt - s);
      const int32_t* ids = lm->ids[n - 1] + s * n;
      err = hipMemcpy(sids, ids, m * n * sizeof(int32_t), hipMemcpyHostToDevice);
      if (err == hipSuccess) err = hipMemcpy(slp, lm->log10p[n - 1] + s, m * sizeof(float), hipMemcpyHostToDevice);
      if (err == hipSuccess && n < 4)
        err = hipMemcpy(sbo, lm->backoff[n - 1] + s, m * sizeof(float), hipMemcpyHostToDevice);
      if (err == hipSuccess)
        err = launch_build_order(n, sids, slp, n < 4 ? sbo : nullptr, m, V, d->S.t2, d->S.t3, *tabs[n - 2], dflags,
                                 any_heavy && n > 2 ? sctx : nullptr, nullptr);
      if (err == hipSuccess) err = hipDeviceSynchronize();
      if (err == hipSuccess && any_heavy) {
        if (n == 2) {
          for (int64_t e = 0; e < m; ++e) mark(2, static_cast<uint32_t>(ids[e * 2]), ids[e * 2 + 1]);
        } else {
          hctx.resize(m);
          err = hipMemcpy(hctx.data(), sctx, m * sizeof(uint32_t), hipMemcpyDeviceToHost);
          for (int64_t e = 0; e < m && err == hipSuccess; ++e)
            if (hctx[e] != kNone) mark(n, hctx[e], ids[e * n + n - 1]);
        }
      }
    }
  }
  (void)hipFree(sids);
  (void)hipFree(slp);
  (void)hipFree(sbo);
  (void)hipFree(sctx);
  if (err != hipSuccess) return fail(LB_ERR_HIP, std::string("n-gram table build: ") + hipGetErrorString(err));
  uint32_t flags = 0;
  LB_HIP(hipMemcpy(&flags, dflags, sizeof(flags), hipMemcpyDeviceToHost));
  if (flags & kFlagBuildRange) return fail(LB_ERR_INVALID_ARG, "n-gram word id out of range");
  if (flags & kFlagBuildContext) return fail(LB_ERR_INVALID_ARG, "n-gram whose context is not an n-gram of the lower order");
  if (flags & kFlagBuildDup) return fail(LB_ERR_INVALID_ARG, "duplicate n-gram");
  if (flags & kFlagBuildFull) return fail(LB_ERR_CAPACITY, "n-gram hash table full");
  PresTable* ptabs[3] = {&d->S.p2, &d->S.p3, &d->S.p4};
  for (int k = 0; k < 3; ++k) {
    if ((st = upload_pres(d, pres[k], lf, ptabs[k])) != LB_OK) return st;
    std::vector<PresEntry>().swap(pres[k]);
  }

  // root of the word-history arena: the empty history, context <s>
  HistNode root{};
  root.blk = kNone;
  root.word = lm->bos_id;
  root.c2 = kNone;
  root.c3 = kNone;
  root.bo1 = uni[lm->bos_id].bo;
  root.bo2 = 0.0f;
  root.bo3 = 0.0f;
  root.sfus = 0.0;
  root.depth = 0;
  for (int i = 0; i < kHistBlock - 1; ++i) root.w[i] = -1;
  LB_HIP(hipMemcpy(d->S.arena, &root, sizeof(root), hipMemcpyHostToDevice));
  return LB_OK;
}

void record_start(lb_decoder* d, EventPair* ep, int kind) {
  ep->kind = kind;
  ep->a = d->get_event();
  ep->b = d->get_event();
  if (ep->a && ep->b) set_launch_events(ep->a, ep->b);
}

void record_stop(lb_decoder* d, EventPair* ep) {
  set_launch_events(nullptr, nullptr);
  if (ep->a && ep->b) d->pending.push_back(*ep);
}

// Launches through fn(); with kind's bit in the profiling mask the launch
// carries start / stop events.
template <typename F>
hipError_t timed_launch(lb_decoder* d, EventPair* ep, int kind, F&& fn) {
  const bool timed = (d->profile_mask >> kind) & 1u;
  if (timed) record_start(d, ep, kind);
  const hipError_t e = fn();
  if (timed) record_stop(d, ep);
  d->launches[kind]++;
  return e;
}

}  // namespace

extern "C" {

const char* lb_last_error(void) { return g_err.c_str(); }

#ifndef LB_BUILD_ID
#define LB_BUILD_ID "unknown"
#endif
const char* lb_build_id(void) { return LB_BUILD_ID; }

lb_status lb_create(const lb_lexicon_desc* lex, const lb_ngram_desc* lm, const lb_params* params,
                    lb_decoder** out) {
  g_err.clear();
  if (!out) return fail(LB_ERR_INVALID_ARG, "out is null");
  *out = nullptr;
  lb_status st = validate(lex, lm, params);
  if (st != LB_OK) return st;
  lb_decoder* d = new (std::nothrow) lb_decoder();
  if (!d) return fail(LB_ERR_OUT_OF_MEMORY, "host allocation failed");
  d->p = *params;
  const lb_params& p = d->p;
  const double lf = p.lm_load_factor == 0.0 ? 0.25 : p.lm_load_factor;
  const int K = p.beam, O = p.subbeams, B = p.max_batch;
  d->block = K <= 64 ? 64 : (K <= 128 ? 128 : 256);
  uint64_t cap = p.arena_nodes_per_stream > 0
                     ? static_cast<uint64_t>(p.arena_nodes_per_stream)
                     : static_cast<uint64_t>(p.max_frames) * K * O + O;
  if (1 + cap * B >= 0xFFFFFFFFull) {
    delete d;
    return fail(LB_ERR_CAPACITY, "word-history arena exceeds 32-bit node ids; lower max_frames or max_batch");
  }
  // the lexicon trie (host), whose largest homophone set bounds the queries of a frame
  HostTrie trie = build_trie(*lex);
  if (trie.max_homophones >= (1u << (64 - kWordCountShift))) {
    delete d;
    return fail(LB_ERR_INVALID_ARG, "more than 65535 words share one phoneme spelling");
  }
  const uint64_t scap = static_cast<uint64_t>(K) * O * std::max<uint32_t>(1, trie.max_homophones);
  if (scap >= 0x7FFFFFFFull) {
    delete d;
    return fail(LB_ERR_CAPACITY, "per-frame n-gram query bound exceeds 31 bits; lower beam or subbeams");
  }
  if (trie.words.size() >= (1ull << 30)) {
    delete d;
    return fail(LB_ERR_INVALID_ARG, "lexicon too large (2^30 words)");
  }
  DevState& S = d->S;
  const size_t BK = static_cast<size_t>(B) * K;
  if ((st = d->alloc(&S.key, BK)) != LB_OK || (st = d->alloc(&S.pkey, BK)) != LB_OK ||
      (st = d->alloc(&S.ab, BK)) != LB_OK || (st = d->alloc(&S.anb, BK)) != LB_OK ||
      (st = d->alloc(&S.pt, BK)) != LB_OK ||
      (st = d->alloc(&S.node, BK)) != LB_OK || (st = d->alloc(&S.meta, BK)) != LB_OK ||
      (st = d->alloc(&S.Lw, BK * O)) != LB_OK || (st = d->alloc(&S.hist, BK * O)) != LB_OK ||
      (st = d->alloc(&S.nbeam, B)) != LB_OK || (st = d->alloc(&S.t0, B)) != LB_OK ||
      (st = d->alloc(&S.arena_n, B)) != LB_OK || (st = d->alloc(&S.arena, 1 + cap * B)) != LB_OK ||
      (st = d->alloc(&S.scrL, static_cast<size_t>(B) * scap)) != LB_OK ||
      (st = d->alloc(&S.scrS, static_cast<size_t>(B) * scap)) != LB_OK ||
      (st = d->alloc(&S.scrE, static_cast<size_t>(B) * K * kMaxSub * kMaxExplicit)) != LB_OK ||
      (st = d->alloc(&S.flags, 1)) != LB_OK || (st = d->alloc(&S.counters, static_cast<size_t>(B) * kNumCounters)) != LB_OK ||
      (st = d->alloc(&S.fsel, BK)) != LB_OK || (st = d->alloc(&S.fsel_n, B)) != LB_OK ||
      (st = d->alloc(&d->ext.d_flag, B)) != LB_OK) {
    std::string msg = g_err;
    delete d;
    return fail(st, msg);
  }
  S.arena_cap = cap;
  S.scap = scap;
  d->ext.t0.assign(B, 0);
  d->ext.len.assign(B, 0);
  d->ext.flag.assign(B, 0);
  auto init = [&]() -> lb_status {
    LB_HIP(hipMemset(S.nbeam, 0, B * sizeof(int32_t)));
    LB_HIP(hipMemset(S.t0, 0, B * sizeof(int64_t)));
    LB_HIP(hipMemset(S.arena_n, 0, B * sizeof(uint32_t)));
    LB_HIP(hipMemset(S.flags, 0, sizeof(uint32_t)));
    LB_HIP(hipMemset(S.counters, 0, static_cast<size_t>(B) * kNumCounters * sizeof(unsigned long long)));
    return LB_OK;
  };
  const uint32_t heavy_min = p.heavy_homophones == 0 ? static_cast<uint32_t>(kHeavyDefault)
                             : (p.heavy_homophones < 0 ? 0xFFFFFFFFu : static_cast<uint32_t>(p.heavy_homophones));
  if ((st = init()) != LB_OK || (st = build_tables(d, trie, lm, lf, heavy_min)) != LB_OK) {
    std::string msg = g_err;
    delete d;
    return fail(st, msg);
  }
  DevParams& P = d->P;
  P.K = K;
  P.O = O;
  P.W = p.max_words_out;
  P.fusion_source = p.fusion_source;
  P.fusion_interval = p.fusion_interval;
  P.fusion_top_f = p.fusion_top_f;
  P.bos = lm->bos_id;
  P.merge_max = p.merge == LB_MERGE_MAX ? 1 : 0;
  P.raw_input = p.input == LB_INPUT_LOGITS ? 1 : 0;
  P.eos_count = p.eos_count;
  for (int k = 0; k < 3; ++k) P.eos_ids[k] = p.eos_ids[k];
  P.heavy_min = heavy_min;
  P.alpha = p.alpha;
  P.beta = p.beta;
  P.gamma = p.gamma;
  P.comega = p.omega * kLn10;
  P.phi = p.phi;
  P.theta = p.theta;
  P.lam = p.lambda;
  P.seed = p.fusion_seed;
  P.lo = p.fusion_lo;
  P.hi = p.fusion_hi;
  {
    const KArgs ka{P, S};
    hipError_t e = hipSuccess;
    if ((st = d->alloc(&d->dargs, 1)) != LB_OK ||
        (e = hipMemcpy(d->dargs, &ka, sizeof(KArgs), hipMemcpyHostToDevice)) != hipSuccess) {
      std::string msg = st != LB_OK ? g_err : std::string("hipMemcpy: ") + hipGetErrorString(e);
      delete d;
      return fail(st != LB_OK ? st : LB_ERR_HIP, msg);
    }
  }
  // the device address of this device's static lookup scratch, for the calls
  // that allocate nothing (a failure here only disables those calls)
  if (static_scratch_address(&d->static_scratch) != hipSuccess) {
    d->static_scratch = nullptr;
    (void)hipGetLastError();
  }
  *out = d;
  return LB_OK;
}

void lb_destroy(lb_decoder* dec) { delete dec; }

lb_status lb_decode_batch(lb_decoder* d, const float* logits, const int32_t* lengths, int32_t batch,
                          int32_t frames, uint32_t flags, void* stream, int32_t* out_hyps, float* out_scores) {
  g_err.clear();
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  if (batch < 1 || batch > d->p.max_batch) return fail(LB_ERR_INVALID_ARG, "batch must be in 1..max_batch");
  if (frames < 0) return fail(LB_ERR_INVALID_ARG, "frames < 0");
  if ((frames > 0 && !logits) || !lengths || !out_hyps || !out_scores)
    return fail(LB_ERR_INVALID_ARG, "null device pointer");
  if (flags & ~static_cast<uint32_t>(LB_BEGIN | LB_END)) return fail(LB_ERR_INVALID_ARG, "unknown flags");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const DevParams& P = d->P;
  const DevState& S = d->S;
  const bool external = P.fusion_source == LB_FUSION_EXTERNAL;
  EventPair ep{};
  auto launch = [&](int kind, auto&& fn) -> hipError_t { return timed_launch(d, &ep, kind, fn); };
  auto& X = d->ext;
  int32_t start = 0;
  bool resuming = false;
  if (external) {
    if (X.in_call) {
      resuming = true;
      // resuming a call that returned LB_NEED_FUSION
      if (logits != X.logits || lengths != X.lengths || batch != X.B || frames != X.Tc || flags != X.flags)
        return fail(LB_ERR_STATE, "a decode call awaiting fusion scores must be repeated with the same arguments");
      if (X.pending) return fail(LB_ERR_STATE, "fusion scores for the pending request have not been supplied");
      start = X.resume_tau;
    } else {
      // the frame counters of the streams decide where fusion happens: read the lengths
      LB_HIP(hipMemcpyAsync(X.len.data(), lengths, batch * sizeof(int32_t), hipMemcpyDeviceToHost, st));
      LB_HIP(hipStreamSynchronize(st));
      for (int32_t b = 0; b < batch; ++b)
        if (X.len[b] < 0 || X.len[b] > frames) return fail(LB_ERR_INVALID_ARG, "lengths must be in 0..frames");
      if (flags & LB_BEGIN)
        for (int32_t b = 0; b < batch; ++b) X.t0[b] = 0;
      X.in_call = true;
      X.final_done = false;
      X.logits = logits;
      X.lengths = lengths;
      X.B = batch;
      X.Tc = frames;
      X.flags = flags;
    }
  }
  if (!resuming && (flags & LB_BEGIN)) LB_HIP(launch(kKindBegin, [&] { return launch_begin(P, S, batch, st); }));
  // frames [start, stop) in one launch; with the external scorer, stop follows
  // the first frame at which some stream fuses
  int32_t stop = frames, fuse_tau = -1;
  if (external) {
    const int64_t I = P.fusion_interval;
    for (int32_t b = 0; b < batch; ++b) {
      // first frame tau >= start of stream b with t = t0 + tau > 0 a multiple of I
      const int64_t t_lo = std::max<int64_t>(X.t0[b] + start, 1);
      const int64_t tau = ((t_lo + I - 1) / I) * I - X.t0[b];
      if (tau < X.len[b] && (fuse_tau < 0 || tau < fuse_tau)) fuse_tau = static_cast<int32_t>(tau);
    }
    if (fuse_tau >= 0) stop = fuse_tau + 1;
  }
  // the output is written by the decode launch itself when nothing else
  // follows it in this call (no fusion round trip), else by k_output
  const int32_t fin = (flags & LB_END) ? 1 : 0;
  const bool out_here = start < stop && fuse_tau < 0 && !(external && fin && !X.final_done);
  if (start < stop)
    LB_HIP(launch(kKindDecode, [&] {
      return launch_decode(P.K, d->dargs, logits, lengths, batch, frames, start, stop, out_here ? fin : 0,
                           out_here ? out_hyps : nullptr, out_here ? out_scores : nullptr,
                           d->decode_opts(), nullptr, st);
    }));
  if (fuse_tau >= 0) {
    for (int32_t b = 0; b < batch; ++b) {
      const int64_t t = X.t0[b] + fuse_tau;
      X.flag[b] = (fuse_tau < X.len[b] && t > 0 && t % P.fusion_interval == 0) ? 1 : 0;
    }
    LB_HIP(hipMemcpyAsync(X.d_flag, X.flag.data(), batch * sizeof(int32_t), hipMemcpyHostToDevice, st));
    LB_HIP(hipStreamSynchronize(st));
    X.pending = 1;
    X.requested = false;
    X.resume_tau = fuse_tau + 1;
    return LB_NEED_FUSION;
  }
  if (external && (flags & LB_END) && !X.final_done) {
    for (int32_t b = 0; b < batch; ++b) X.flag[b] = 2;
    LB_HIP(hipMemcpyAsync(X.d_flag, X.flag.data(), batch * sizeof(int32_t), hipMemcpyHostToDevice, st));
    LB_HIP(hipStreamSynchronize(st));
    X.pending = 2;
    X.requested = false;
    X.final_done = true;
    X.resume_tau = frames;
    return LB_NEED_FUSION;
  }
  if (!out_here)
    LB_HIP(launch(kKindOutput, [&] { return launch_output(d->block, P, S, lengths, batch, frames, fin, out_hyps, out_scores, st); }));
  if (external) {
    for (int32_t b = 0; b < batch; ++b) X.t0[b] += X.len[b];
    X.in_call = false;
  }
  return LB_OK;
}

lb_status lb_decode_batch_noalloc(lb_decoder* d, const float* logits, const int32_t* lengths, int32_t batch,
                                  int32_t frames, uint32_t flags, void* stream, int32_t* out_hyps,
                                  float* out_scores) {
  g_err.clear();
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  if (batch < 1 || batch > d->p.max_batch) return fail(LB_ERR_INVALID_ARG, "batch must be in 1..max_batch");
  if (frames < 0) return fail(LB_ERR_INVALID_ARG, "frames < 0");
  if ((frames > 0 && !logits) || !lengths || !out_hyps || !out_scores)
    return fail(LB_ERR_INVALID_ARG, "null device pointer");
  if (flags & ~static_cast<uint32_t>(LB_BEGIN | LB_END)) return fail(LB_ERR_INVALID_ARG, "unknown flags");
  const DevParams& P = d->P;
  const DevState& S = d->S;
  if (P.fusion_source == LB_FUSION_EXTERNAL)
    return fail(LB_ERR_INVALID_ARG, "lb_decode_batch_noalloc does not run the external fusion round trip "
                                    "(it reads the lengths to the host); use lb_decode_batch");
  const size_t need = scratch_layout(static_cast<size_t>(batch), S.scap, static_cast<size_t>(P.K)).bytes;
  if (need > kStaticScratchBytes)
    return fail(LB_ERR_CAPACITY, "lb_decode_batch_noalloc: " + std::to_string(batch) + " streams need " +
                                     std::to_string(need) + " B of lookup scratch, the static scratch holds " +
                                     std::to_string(kStaticScratchBytes) +
                                     " B; decode fewer streams per call or use lb_decode_batch");
  if (!d->static_scratch) return fail(LB_ERR_HIP, "the static lookup scratch has no device address on this device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  // the same launches as lb_decode_batch, without event timing (which creates events)
  if (flags & LB_BEGIN) {
    LB_HIP(launch_begin(P, S, batch, st));
    d->launches[kKindBegin]++;
  }
  const int32_t fin = (flags & LB_END) ? 1 : 0;
  if (frames > 0) {
    LB_HIP(launch_decode(P.K, d->dargs, logits, lengths, batch, frames, 0, frames, fin, out_hyps, out_scores,
                         d->decode_opts(), d->static_scratch, st));
    d->launches[kKindDecode]++;
  } else {
    LB_HIP(launch_output(d->block, P, S, lengths, batch, frames, fin, out_hyps, out_scores, st));
    d->launches[kKindOutput]++;
  }
  return LB_OK;
}

lb_status lb_fusion_request(lb_decoder* d, int32_t* words, int32_t* n_words, void* stream) {
  g_err.clear();
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  if (!d->ext.pending) return fail(LB_ERR_STATE, "no fusion request is pending");
  if (!words || !n_words) return fail(LB_ERR_INVALID_ARG, "null device pointer");
  hipStream_t st = static_cast<hipStream_t>(stream);
  EventPair ep{};
  auto launch = [&](int kind, auto&& fn) -> hipError_t { return timed_launch(d, &ep, kind, fn); };
  LB_HIP(launch(kKindFuseSelect, [&] { return launch_fuse_select(d->block, d->P, d->S, d->ext.d_flag, d->ext.B, st); }));
  LB_HIP(launch(kKindFuseExport, [&] { return launch_fuse_export(d->block, d->P, d->S, words, n_words, d->ext.B, st); }));
  d->ext.requested = true;
  return LB_OK;
}

lb_status lb_fusion_scores(lb_decoder* d, const float* fusion_logprobs, void* stream) {
  g_err.clear();
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  if (!d->ext.pending) return fail(LB_ERR_STATE, "no fusion request is pending");
  if (!fusion_logprobs) return fail(LB_ERR_INVALID_ARG, "null device pointer");
  hipStream_t st = static_cast<hipStream_t>(stream);
  EventPair ep{};
  auto launch = [&](int kind, auto&& fn) -> hipError_t { return timed_launch(d, &ep, kind, fn); };
  if (!d->ext.requested)
    LB_HIP(launch(kKindFuseSelect, [&] { return launch_fuse_select(d->block, d->P, d->S, d->ext.d_flag, d->ext.B, st); }));
  LB_HIP(launch(kKindFuseApply, [&] { return launch_fuse_apply(d->block, d->P, d->S, fusion_logprobs, d->ext.B, st); }));
  d->ext.pending = 0;
  d->ext.requested = false;
  return LB_OK;
}

lb_status lb_measure_gather(const void* table, uint64_t table_lines, uint64_t n_lines, uint64_t seed,
                            uint32_t* out, uint64_t out_len, void* stream) {
  g_err.clear();
  if (!table || !out) return fail(LB_ERR_INVALID_ARG, "null device pointer");
  if (table_lines < 1 || n_lines < 1) return fail(LB_ERR_INVALID_ARG, "table_lines and n_lines must be >= 1");
  if (out_len < gather_probe_threads(n_lines))
    return fail(LB_ERR_INVALID_ARG, "out needs " + std::to_string(gather_probe_threads(n_lines)) + " entries");
  LB_HIP(launch_gather_probe(table, table_lines, n_lines, seed, out, static_cast<hipStream_t>(stream)));
  return LB_OK;
}

lb_status lb_get_status(lb_decoder* d, void* stream) {
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  LB_HIP(hipStreamSynchronize(static_cast<hipStream_t>(stream)));
  uint32_t flags = 0;
  LB_HIP(hipMemcpy(&flags, d->S.flags, sizeof(flags), hipMemcpyDeviceToHost));
  if (flags & kFlagArena) return fail(LB_ERR_CAPACITY, "word-history arena overflow (raise arena_nodes_per_stream)");
  if (flags & kFlagWords) return fail(LB_ERR_CAPACITY, "hypothesis longer than max_words_out (output truncated)");
  if (flags & kFlagSelect) return fail(LB_ERR_CAPACITY, "internal top-K selection overflow");
  if (flags & kFlagLength)
    return fail(LB_ERR_INVALID_ARG, "a decode call's lengths were outside 0..frames (decoded and counted as clamped)");
  return LB_OK;
}

lb_status lb_get_stats(lb_decoder* d, lb_stats* out) {
  if (!d || !out) return fail(LB_ERR_INVALID_ARG, "null argument");
  LB_HIP(hipDeviceSynchronize());
  std::vector<unsigned long long> c(static_cast<size_t>(d->p.max_batch) * kNumCounters);
  LB_HIP(hipMemcpy(c.data(), d->S.counters, c.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
  std::memset(out, 0, sizeof(*out));
  for (int b = 0; b < d->p.max_batch; ++b) {
    const unsigned long long* x = &c[static_cast<size_t>(b) * kNumCounters];
    out->expansions += static_cast<int64_t>(x[kCntExpansions]);
    out->word_events += static_cast<int64_t>(x[kCntWordEvents]);
    out->lm_queries += static_cast<int64_t>(x[kCntLmQueries]);
    out->fused += static_cast<int64_t>(x[kCntFused]);
    out->frames += static_cast<int64_t>(x[kCntFrames]);
    out->probe_lines += static_cast<int64_t>(x[kCntProbeLines]);
    out->lm_lookups += static_cast<int64_t>(x[kCntLookups]);
    out->index_lines += static_cast<int64_t>(x[kCntPresLines]);
    for (int k = 0; k < kPhases; ++k) out->phase_cycles[k] += static_cast<int64_t>(x[kCntPhase0 + k]);
  }
  d->harvest();
  for (int k = 0; k < kKinds; ++k) {
    out->launches[k] = d->launches[k];
    out->kernel_ms[k] = d->kernel_ms[k];
    out->timed[k] = d->timed[k];
  }
  return LB_OK;
}

lb_status lb_reset_stats(lb_decoder* d) {
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  LB_HIP(hipDeviceSynchronize());
  LB_HIP(hipMemset(d->S.counters, 0, static_cast<size_t>(d->p.max_batch) * kNumCounters * sizeof(unsigned long long)));
  d->harvest();
  for (int k = 0; k < kKinds; ++k) {
    d->launches[k] = 0;
    d->kernel_ms[k] = 0;
    d->timed[k] = 0;
  }
  return LB_OK;
}

lb_status lb_set_profiling(lb_decoder* d, uint32_t kernel_mask) {
  if (!d) return fail(LB_ERR_INVALID_ARG, "decoder is null");
  d->profile_mask = kernel_mask;
  return LB_OK;
}

}  // extern "C"
