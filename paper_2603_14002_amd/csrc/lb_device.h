// Device-side data layout and helpers of the LightBeam gfx950 decoder.
//
// HBM layout (all buffers allocated once in lb_create, for max_batch streams):
//   trie        TrieNode[S+1]   16 B/node: child mask (bits 1..39 phonemes, bit 40
//                               separator when the node ends a word, bits 48..63
//                               the number of words ending there), index of the
//                               first child (children are contiguous, in phoneme
//                               order), offset of the node's words in trie_words
//   trie_words  int32[]         word ids ending at each node, ascending
//   uni         Unigram[vocab]  dense log10 p / backoff by word id
//   t2, t3, t4  Slot[4*nbuckets] open-addressing hash tables of orders 2..4; a
//                               bucket is one 64-B line of four 16-B slots
//                               {key, log10 p, backoff}; key = (context, word)
//                               where context is the word id (order 2) or the
//                               slot index of the context n-gram (orders 3, 4)
//   beams       SoA [max_batch][K] (sub-beam arrays [max_batch][K][O])
//   arena       HistNode[1 + max_batch*cap]: word-history nodes; node 0 is the
//               empty history (context <s>), stream b owns [1+b*cap, 1+(b+1)*cap)
//   scrL, scrS  [max_batch][K*O*Hmax] per-stream n-gram lookup results of a
//               frame (Hmax: the largest homophone set)
//   wrank       WordRank[] parallel to trie_words: each node's words again, in
//               (unigram log10 p desc, index asc) order
//   p2, p3, p4  explicit-continuation index of the heavy nodes (many homophones):
//               (context, node) -> the node's homophones h whose n-gram
//               (context, word h) exists, for contexts of orders 1, 2, 3
//               (word id, 2-gram slot, 3-gram slot); same bucket layout as t2..t4
//   scrE        [max_batch][K*4*kMaxExplicit] per-stream explicit homophone
//               lists of a frame's heavy query groups
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lb {

constexpr int kClasses = 41;
constexpr int kSep = 40;
constexpr int kMaxBeam = 256;
constexpr int kMaxSub = 4;
constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr uint64_t kEmptyKey = ~0ull;
constexpr uint64_t kNoParent = 0xFFFFFFFFFFFFFFFEull;  // parent key of the empty prefix
constexpr uint32_t kRootNode = 0;                      // trie root
constexpr uint32_t kRootHist = 0;                      // empty word history
constexpr double kLn10 = 2.302585092994045684017991454684364208;
constexpr int kWordCountShift = 48;  // TrieNode::mask bits 48..63: words ending at the node
constexpr int kMaxExplicit = 16;     // a heavy group with more explicit homophones takes the full path
constexpr int kHeavyDefault = 3;     // default homophone count from which a node is heavy

// overflow / error flag bits (DevState::flags)
constexpr uint32_t kFlagArena = 1u;
constexpr uint32_t kFlagWords = 2u;
constexpr uint32_t kFlagSelect = 4u;
constexpr uint32_t kFlagBuildRange = 8u;
constexpr uint32_t kFlagBuildContext = 16u;
constexpr uint32_t kFlagBuildDup = 32u;
constexpr uint32_t kFlagBuildFull = 64u;
constexpr uint32_t kFlagLength = 128u;  // a decode call's length outside 0..frames (clamped)

// phases of a decode frame timed by the phase counters: recombination and stay
// scores, top-K selection, new beam, grouping of the n-gram queries (with the
// continuation index), the n-gram lookups, ranking of the completed words and
// history nodes, the rest of the frame (fusion, trie-node store, next row);
// kPhOther: beam load, write-back and output outside the frame loop
enum { kPhRecomb = 0, kPhTopK = 1, kPhNewBeam = 2, kPhGroup = 3, kPhLookup = 4, kPhRank = 5, kPhFusion = 6,
       kPhOther = 7, kPhases = 8 };
constexpr uint32_t kOptPhaseTimers = 1u;  // k_decode option: per-phase clock cycles

// per-stream counters (DevState::counters, [max_batch][kNumCounters])
enum { kCntExpansions = 0, kCntWordEvents = 1, kCntLmQueries = 2, kCntFused = 3, kCntFrames = 4,
       kCntProbeLines = 5, kCntLookups = 6, kCntPresLines = 7, kCntPhase0 = 8,
       kNumCounters = kCntPhase0 + kPhases };

struct TrieNode {
  uint64_t mask;
  uint32_t first_child;
  uint32_t word_off;
};

struct Unigram {
  float logp;
  float bo;
};

struct Slot {
  uint64_t key;
  float logp;
  float bo;
};

struct NgramTable {
  Slot* slots;
  uint64_t nbuckets;
};

// A word of a trie node: its id, unigram log10 p and backoff, and its index
// among the node's words (ascending ids).
struct WordRank {
  int32_t w;
  float logp;
  float bo;
  uint32_t h;
};

// Explicit-continuation index slot: key = (context id << 32) | node word offset;
// n homophone indices, stored in `a` itself when n == 1, else at lists[a..a+n).
struct PresSlot {
  uint64_t key;
  uint32_t a;
  uint32_t n;
};

struct PresTable {
  PresSlot* slots;
  uint64_t nbuckets;
  const uint32_t* lists;
};

// Word-history node (64 B, one line): the word sequence of an orthographic
// sub-beam plus the n-gram state after its last word: the word itself (the
// 1-word context), the slots of the 2- and 3-word contexts (kNone if absent)
// and the three backoff weights, the number of words in the chain (depth), the
// running synthetic fusion score, and what a traceback needs.  The chain is
// cut into blocks of kHistBlock words (depths 1..7, 8..14, ...): a node keeps
// the words of the earlier nodes of its own block, nearest first, in w[0 ..
// (depth - 1) % kHistBlock), and `blk`, the node that ends the previous block
// (depth kHistBlock * floor((depth - 1) / kHistBlock); the root ends block 0),
// so a traceback reads one node per block.
constexpr int kHistBlock = 7;
struct HistNode {
  uint32_t blk;
  int32_t word;
  uint32_t c2;
  uint32_t c3;
  float bo1, bo2, bo3;
  uint32_t depth;
  double sfus;
  int32_t w[kHistBlock - 1];
};
static_assert(sizeof(HistNode) == 64, "history node is one 64-B line");

// n-gram state after a queried word: slots of its 2- and 3-word contexts and
// their backoffs, the word and its unigram backoff.
struct QState {
  uint32_t c2, c3;
  float bo2, bo3;
  int32_t w;
  float bo1;
};

struct DevParams {
  int32_t K, O, W;
  int32_t fusion_source, fusion_interval, fusion_top_f;
  int32_t bos;
  int32_t merge_max;  // 1: paths into one prefix combine by max, 0: by log-sum-exp
  int32_t raw_input;  // 1: per-frame scores are raw, log-softmax them first
  int32_t eos_count;  // end-of-sentence marks tried at the final synthetic fusion
  int32_t eos_ids[3];
  uint32_t heavy_min;  // nodes with at least this many words use the explicit-continuation index
  double alpha, beta, gamma, comega, phi, theta, lam;
  uint64_t seed;
  double lo, hi;
};

struct DevState {
  // hypotheses, [B][K] (sub-beams [B][K][O])
  uint64_t* key;
  uint64_t* pkey;
  double* ab;
  double* anb;
  double* pt;  // log-sum-exp(ab, anb)
  uint32_t* node;
  uint32_t* meta;  // last symbol (bits 0..7) | number of sub-beams (bits 8..15)
  double* Lw;
  uint32_t* hist;
  int32_t* nbeam;     // [B]
  int64_t* t0;        // [B] frames decoded since LB_BEGIN
  uint32_t* arena_n;  // [B] arena nodes used
  HistNode* arena;
  uint64_t arena_cap;  // per stream
  // per-stream LM lookup results of a frame: [B][scap] log10 p and n-gram state
  double* scrL;
  QState* scrS;
  uint64_t scap;
  uint32_t* flags;
  unsigned long long* counters;  // [B][kNumCounters]
  // fusion selection for external scores: [B][K] beam index per rank, [B] count
  int32_t* fsel;
  int32_t* fsel_n;
  // lexicon
  const TrieNode* trie;
  const int32_t* trie_words;
  // n-gram LM
  const Unigram* uni;
  NgramTable t2, t3, t4;
  // heavy nodes: words in unigram order, explicit-continuation index, and the
  // per-stream explicit homophone lists of a frame ([B][K*kMaxSub*kMaxExplicit])
  const WordRank* wrank;
  PresTable p2, p3, p4;
  uint32_t* scrE;
};

// Layout of the n-gram lookup scratch of a decode call over nb streams, when it
// is one contiguous buffer: nb x scap lookup results (f64 log10 P), then nb x
// scap n-gram states (QState), then nb x K*kMaxSub*kMaxExplicit explicit
// homophone indices (u32); each region starts on a 256-B boundary.
struct ScratchLayout {
  size_t off_state, off_explicit, bytes;
};
__host__ __device__ inline ScratchLayout scratch_layout(size_t nb, size_t scap, size_t K) {
  auto up = [](size_t x) { return (x + 255) & ~static_cast<size_t>(255); };
  ScratchLayout l;
  l.off_state = up(nb * scap * sizeof(double));
  l.off_explicit = l.off_state + up(nb * scap * sizeof(QState));
  l.bytes = l.off_explicit + up(nb * K * kMaxSub * kMaxExplicit * sizeof(uint32_t));
  return l;
}

// The decode kernel's parameters and state, kept in device memory (written
// once by lb_create) and read through a constant-memory pointer.
struct KArgs {
  DevParams P;
  DevState S;
};
#define LB_CONST __attribute__((address_space(4)))

// SplitMix64 output for state x (Steele, Lea & Flood, OOPSLA 2014).
__host__ __device__ inline uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// 64-bit rolling key of a collapsed prefix: key(y v) = splitmix64(key(y) ^ v), key(()) = 0.
__host__ __device__ inline uint64_t prefix_step(uint64_t k, int v) {
  return splitmix64(k ^ static_cast<uint64_t>(v));
}

// Bucket of an n-gram key: multiply-high range reduction of a mixed hash.
__host__ __device__ inline uint64_t bucket_of(uint64_t key, uint64_t nbuckets) {
  const uint64_t h = splitmix64(key ^ 0xD6E8FEB86659FD93ull);
#if defined(__HIP_DEVICE_COMPILE__)
  return __umul64hi(h, nbuckets);
#else
  return static_cast<uint64_t>((static_cast<unsigned __int128>(h) * nbuckets) >> 64);
#endif
}

// log1p(e) for e in [0, 1], the only arguments a log-sum-exp of two scores
// gives it: 2 atanh(s) with s = e / (2 + e) in [0, 1/3].  s is carried as
// q + lo: the rounding of 2 + e (recovered exactly: den - 2 is exact by
// Sterbenz' lemma) and that of the quotient (its residual, by a fused
// multiply-add) go into lo.  atanh(s) - s = s^3 (1/3 + s^2/5 + s^4/7 + ...),
// cut after the s^33 term: with s^2 <= 1/9 the rest is below 2e-17 of the
// sum.  Checked on 2e7 random arguments against an 80-bit log1p: correctly
// rounded in 99 % of them, never off by more than 0.7 ulp; about half the
// instructions of the general routine, which a two-input log-sum-exp in
// every hypothesis of every frame makes worth it.
// The series' coefficient of s^(2n+3) is 1/(2n+3), n = 0..kAtanhTerms-1;
// coef(n) returns it (a compile-time constant, or a table the caller keeps:
// the decode kernel reads them from LDS, which loads them into vector
// registers without a vector move per constant half).
constexpr int kAtanhTerms = 16;
template <class Coef>
__host__ __device__ inline double log1p_unit(double e, Coef coef) {
  const double den = 2.0 + e;
  const double err = e - (den - 2.0);  // 2 + e == den + err exactly
  const double r = 1.0 / den;
  const double q = e * r;
  const double lo = fma(-q, err, fma(-q, den, e)) * r;
  const double u = q * q;
  double p = coef(kAtanhTerms - 1);
#pragma unroll
  for (int n = kAtanhTerms - 2; n >= 0; --n) p = fma(p, u, coef(n));
  return 2.0 * q + 2.0 * (lo + (q * u) * p);
}
__host__ __device__ inline double log1p_unit(double e) {
  return log1p_unit(e, [](int n) { return 1.0 / (2 * n + 3); });
}

template <class Coef>
__device__ inline double lse2(double x, double y, Coef coef) {
  if (x == -HUGE_VAL && y == -HUGE_VAL) return -HUGE_VAL;
  const double m = x > y ? x : y;
  return m + log1p_unit(exp(-fabs(x - y)), coef);
}
__device__ inline double lse2(double x, double y) {
  return lse2(x, y, [](int n) { return 1.0 / (2 * n + 3); });
}

// Synthetic word-bigram fusion score Bg(a, b), natural log.
__device__ inline double bigram_score(const DevParams& P, int a, int b) {
  const uint64_t h = splitmix64(P.seed ^ ((static_cast<uint64_t>(static_cast<uint32_t>(a)) << 32) |
                                          static_cast<uint64_t>(static_cast<uint32_t>(b))));
  const double u = static_cast<double>(h >> 48) * (1.0 / 65536.0);
  return P.lo + (P.hi - P.lo) * u;
}

// Order-preserving map of a double to uint64 (larger double -> larger integer).
__device__ inline uint64_t order_bits(double x) {
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(x));
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

}  // namespace lb
