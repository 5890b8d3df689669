// HIP kernels of the LightBeam gfx950 decoder (wave64, CDNA4).
//
// A decode call is one launch of k_decode on the caller's stream: one
// workgroup per stream runs Alg. 1 over the call's frames with the stream's
// beam resident in LDS (fan-out, recombination, theta / top-K pruning, trie
// advance, Eq. (1) with the hashed 4-gram LM, Eq. (2) with the synthetic
// scorer).  The output -- each stream's hypotheses ranked, their word ids and
// scores written (after the final fusion at the end of an utterance) -- is
// written by the call's last k_decode launch, or by k_output when the call
// ends without one.  k_fuse_select,
// k_fuse_export and k_fuse_apply carry the round trip to an external fusion
// scorer; k_build_order fills the n-gram hash tables; k_begin resets streams.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <mutex>
#include <type_traits>

#include "lb_device.h"
#include "lb_launch.h"

namespace lb {

namespace {

constexpr double kNegInf = -HUGE_VAL;
constexpr int kBoundaryCap = 256;   // candidates resolved exactly inside the boundary bin
constexpr int kMaxLevels = 16;      // refinement levels of the top-K selection
constexpr uint32_t kGroupHeavy = 0x80000000u;  // query group scored through its explicit homophones

// ------------------------------------------------------------------ block helpers

// Workgroup barrier that orders LDS only: it waits for the wave's LDS
// operations, not for its outstanding global loads and stores (those are
// waited for where their registers are used, and by a full __syncthreads
// where global memory is handed between threads).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Cross-lane moves inside rows of 16 lanes (DPP): lane i reads lane i^1
// (quad_perm [1,0,3,2]), lane i^2 (quad_perm [2,3,0,1]), the mirror lane in
// its half-row (7-i) and in its row (15-i).  Applying an associative,
// commutative operation after each of the four leaves every lane with the
// result over its row; the four rows are then combined through readlane.  A
// lane whose source lane is inactive receives `ident` (the operation's
// identity).
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

template <int CTRL>
__device__ __forceinline__ int dpp_i32(int x, int ident) {
  return __builtin_amdgcn_update_dpp(ident, x, CTRL, 0xF, 0xF, false);
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x, double ident) {
  return __hiloint2double(dpp_i32<CTRL>(__double2hiint(x), __double2hiint(ident)),
                          dpp_i32<CTRL>(__double2loint(x), __double2loint(ident)));
}

__device__ __forceinline__ double readlane_f64(double x, int lane) {
  return __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(x), lane),
                          __builtin_amdgcn_readlane(__double2loint(x), lane));
}

// Wavefront maximum of *mx and minimum of *mn, in every lane.
__device__ __forceinline__ void wave_minmax(double* mx, double* mn) {
  double a = *mx, c = *mn;
#define LB_MM_STEP(C)                    \
  a = fmax(a, dpp_f64<C>(a, -HUGE_VAL)); \
  c = fmin(c, dpp_f64<C>(c, HUGE_VAL));
  LB_MM_STEP(kDppXor1)
  LB_MM_STEP(kDppXor2)
  LB_MM_STEP(kDppHalfMirror)
  LB_MM_STEP(kDppMirror)
#undef LB_MM_STEP
  *mx = fmax(fmax(readlane_f64(a, 0), readlane_f64(a, 16)), fmax(readlane_f64(a, 32), readlane_f64(a, 48)));
  *mn = fmin(fmin(readlane_f64(c, 0), readlane_f64(c, 16)), fmin(readlane_f64(c, 32), readlane_f64(c, 48)));
}

// Wavefront maximum of x, in every lane.
__device__ __forceinline__ double wave_max(double x) {
  x = fmax(x, dpp_f64<kDppXor1>(x, -HUGE_VAL));
  x = fmax(x, dpp_f64<kDppXor2>(x, -HUGE_VAL));
  x = fmax(x, dpp_f64<kDppHalfMirror>(x, -HUGE_VAL));
  x = fmax(x, dpp_f64<kDppMirror>(x, -HUGE_VAL));
  return fmax(fmax(readlane_f64(x, 0), readlane_f64(x, 16)), fmax(readlane_f64(x, 32), readlane_f64(x, 48)));
}

// Wavefront sum of x, in every lane.
__device__ __forceinline__ double wave_sum(double x) {
  x += dpp_f64<kDppXor1>(x, 0.0);
  x += dpp_f64<kDppXor2>(x, 0.0);
  x += dpp_f64<kDppHalfMirror>(x, 0.0);
  x += dpp_f64<kDppMirror>(x, 0.0);
  return (readlane_f64(x, 0) + readlane_f64(x, 16)) + (readlane_f64(x, 32) + readlane_f64(x, 48));
}

// One DPP step of the wavefront arg-max of (L desc, q asc).
template <int CTRL>
__device__ __forceinline__ void argmax_step(double* L, int* q) {
  const double oL = dpp_f64<CTRL>(*L, -HUGE_VAL);
  const int oq = dpp_i32<CTRL>(*q, 0x7FFFFFFF);
  const bool take = oL > *L || (oL == *L && oq < *q);
  *L = take ? oL : *L;
  *q = take ? oq : *q;
}

// Wavefront arg-max of (L desc, q asc), in every lane.
__device__ __forceinline__ void wave_argmax(double* L, int* q) {
  argmax_step<kDppXor1>(L, q);
  argmax_step<kDppXor2>(L, q);
  argmax_step<kDppHalfMirror>(L, q);
  argmax_step<kDppMirror>(L, q);
  double bL = readlane_f64(*L, 0);
  int bq = __builtin_amdgcn_readlane(*q, 0);
#pragma unroll
  for (int r = 16; r < 64; r += 16) {
    const double oL = readlane_f64(*L, r);
    const int oq = __builtin_amdgcn_readlane(*q, r);
    if (oL > bL || (oL == bL && oq < bq)) {
      bL = oL;
      bq = oq;
    }
  }
  *L = bL;
  *q = bq;
}

template <int BLOCK>
__device__ inline double block_max(double v, double* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  lds_barrier();
  double r = red[0];
#pragma unroll
  for (int k = 1; k < BLOCK / 64; ++k) r = fmax(r, red[k]);
  lds_barrier();
  return r;
}

// Block-wide maximum of `mx` and minimum of `mn` in one reduction (SYNC as in
// block_scan).
template <int BLOCK, bool SYNC = true>
__device__ inline void block_minmax(double mx, double mn, double* red, double* out_max, double* out_min) {
  wave_minmax(&mx, &mn);
  constexpr int NW = BLOCK / 64;
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = mx;
    red[NW + (threadIdx.x >> 6)] = mn;
  }
  lds_barrier();
  double a = red[0], c = red[NW];
#pragma unroll
  for (int k = 1; k < NW; ++k) {
    a = fmax(a, red[k]);
    c = fmin(c, red[NW + k]);
  }
  if (SYNC) lds_barrier();
  *out_max = a;
  *out_min = c;
}

// Inclusive prefix sum over the wavefront: shifts by 1, 2, 4, 8 inside each
// row of 16 lanes (lanes shifted in from outside the row add 0), then rows 1
// and 3 add the last lane of the row before them, and rows 2 and 3 add lane 31.
__device__ __forceinline__ int wave_scan_incl(int v) {
  int x = v;
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
  return x;
}

// Exclusive prefix sum over the block; *total receives the block sum.  With
// SYNC = false the trailing barrier is left out: `red` must then not be
// written again before the next barrier.
template <int BLOCK, bool SYNC = true>
__device__ inline int block_scan(int v, int* red, int* total) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int x = wave_scan_incl(v);
  if (lane == 63) red[w] = x;
  lds_barrier();
  int base = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < BLOCK / 64; ++k) {
    const int t = red[k];
    base += (k < w) ? t : 0;
    tot += t;
  }
  if (SYNC) lds_barrier();
  *total = tot;
  return base + x - v;
}

// (score desc, key asc)
__device__ inline bool ranks_before(double sa, uint64_t ka, double sb, uint64_t kb) {
  return sa > sb || (sa == sb && ka < kb);
}

// In-place bitonic sort of N entries (N a power of two, at most the block
// size) by (score desc, key asc); every thread of the block calls it.
template <int N>
__device__ inline void bitonic_sort(double* sc, uint64_t* ky, uint32_t* val) {
  const int i = threadIdx.x;
  for (int k = 2; k <= N; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int ixj = i ^ j;
      if (i < N && ixj > i) {
        const bool up = (i & k) == 0;
        const bool swap = up ? ranks_before(sc[ixj], ky[ixj], sc[i], ky[i])
                             : ranks_before(sc[i], ky[i], sc[ixj], ky[ixj]);
        if (swap) {
          const double s = sc[i];
          sc[i] = sc[ixj];
          sc[ixj] = s;
          const uint64_t kk = ky[i];
          ky[i] = ky[ixj];
          ky[ixj] = kk;
          const uint32_t vv = val[i];
          val[i] = val[ixj];
          val[ixj] = vv;
        }
      }
      lds_barrier();
    }
  }
}

// ------------------------------------------------------------------ n-gram tables

// Looks `key` up; `lines` counts the 64-B bucket lines read.
__device__ inline bool probe(const NgramTable& t, uint64_t key, uint32_t* slot, float* lp, float* bo,
                             uint32_t* lines) {
  if (t.nbuckets == 0) return false;
  uint64_t bk = bucket_of(key, t.nbuckets);
  for (uint64_t it = 0; it < t.nbuckets; ++it) {
    ++*lines;
    const uint4* line = reinterpret_cast<const uint4*>(t.slots + bk * 4);
    uint4 q[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) q[s] = line[s];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint64_t k = static_cast<uint64_t>(q[s].x) | (static_cast<uint64_t>(q[s].y) << 32);
      if (k == key) {
        *slot = static_cast<uint32_t>(bk * 4 + s);
        *lp = __uint_as_float(q[s].z);
        *bo = __uint_as_float(q[s].w);
        return true;
      }
      if (k == kEmptyKey) return false;
    }
    bk = (bk + 1 == t.nbuckets) ? 0 : bk + 1;
  }
  return false;
}

// 0 = inserted, 1 = duplicate key, 2 = table full
__device__ inline int insert(const NgramTable& t, uint64_t key, float lp, float bo) {
  uint64_t bk = bucket_of(key, t.nbuckets);
  for (uint64_t it = 0; it < t.nbuckets; ++it) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      Slot* sl = t.slots + bk * 4 + s;
      const unsigned long long prev =
          atomicCAS(reinterpret_cast<unsigned long long*>(&sl->key), kEmptyKey, key);
      if (prev == kEmptyKey) {
        sl->logp = lp;
        sl->bo = bo;
        return 0;
      }
      if (prev == key) return 1;
    }
    bk = (bk + 1 == t.nbuckets) ? 0 : bk + 1;
  }
  return 2;
}

// Inserts a chunk of order-`order` n-grams; each n-gram's context id (the word
// id for order 2, the slot of its context n-gram for orders 3 and 4) goes to
// ctx_out[e] when ctx_out is given (kNone on error).
__global__ void k_build_order(int order, const int32_t* __restrict__ ids, const float* __restrict__ lp,
                              const float* __restrict__ bo, int64_t count, int32_t vocab, NgramTable t2,
                              NgramTable t3, NgramTable dst, uint32_t* flags, uint32_t* ctx_out) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < count; e += stride) {
    const int32_t* r = ids + e * order;
    if (ctx_out) ctx_out[e] = kNone;
    bool ok = true;
    for (int k = 0; k < order; ++k) ok = ok && r[k] >= 0 && r[k] < vocab;
    if (!ok) {
      atomicOr(flags, kFlagBuildRange);
      continue;
    }
    uint64_t ctx = static_cast<uint32_t>(r[0]);
    if (order >= 3) {
      uint32_t s2, nl = 0;
      float a, c;
      if (!probe(t2, (static_cast<uint64_t>(r[0]) << 32) | static_cast<uint32_t>(r[1]), &s2, &a, &c, &nl)) {
        atomicOr(flags, kFlagBuildContext);
        continue;
      }
      ctx = s2;
      if (order == 4) {
        uint32_t s3;
        if (!probe(t3, (static_cast<uint64_t>(s2) << 32) | static_cast<uint32_t>(r[2]), &s3, &a, &c, &nl)) {
          atomicOr(flags, kFlagBuildContext);
          continue;
        }
        ctx = s3;
      }
    }
    const uint64_t key = (ctx << 32) | static_cast<uint32_t>(r[order - 1]);
    if (ctx_out) ctx_out[e] = static_cast<uint32_t>(ctx);
    const int st = insert(dst, key, lp[e], bo ? bo[e] : 0.0f);
    if (st == 1) atomicOr(flags, kFlagBuildDup);
    if (st == 2) atomicOr(flags, kFlagBuildFull);
  }
}

// ------------------------------------------------------------------ stream reset

__global__ void k_begin(DevParams P, DevState S, int32_t B) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  const size_t i = static_cast<size_t>(b) * P.K;
  S.nbeam[b] = 1;
  S.key[i] = 0;
  S.pkey[i] = kNoParent;
  S.ab[i] = 0.0;
  S.anb[i] = kNegInf;
  S.pt[i] = lse2(0.0, kNegInf);
  S.node[i] = kRootNode;
  S.meta[i] = 1u << 8;  // no last symbol, one sub-beam
  S.Lw[i * P.O] = 0.0;
  S.hist[i * P.O] = kRootHist;
  S.t0[b] = 0;
  S.arena_n[b] = 0;
}

// ------------------------------------------------------------------ n-gram lookup

// One 64-B bucket: four 16-B slots {key lo, key hi, log10 p, backoff}.
struct Bucket {
  uint4 s0, s1, s2, s3;
};

// (NgramTable and PresTable share the bucket layout: 16-B slots {u64 key, u32, u32})
template <typename Table>
__device__ __forceinline__ Bucket load_bucket(const Table& t, uint64_t bk) {
  const uint4* line = reinterpret_cast<const uint4*>(t.slots + bk * 4);
  Bucket q;
  q.s0 = line[0];
  q.s1 = line[1];
  q.s2 = line[2];
  q.s3 = line[3];
  return q;
}

__device__ __forceinline__ uint64_t slot_key(const uint4& v) {
  return static_cast<uint64_t>(v.x) | (static_cast<uint64_t>(v.y) << 32);
}

// Scans a bucket for `key`: 1 found (slot index and the slot's two values set),
// 0 absent, -1 bucket full.
__device__ __forceinline__ int scan_bucket(const Bucket& q, uint64_t key, uint64_t bk, uint32_t* slot, uint32_t* z,
                                           uint32_t* w) {
#define LB_SCAN_SLOT(V, K)                              \
  {                                                     \
    const uint64_t kk = slot_key(V);                    \
    if (kk == key) {                                    \
      *slot = static_cast<uint32_t>(bk * 4 + (K));      \
      *z = (V).z;                                       \
      *w = (V).w;                                       \
      return 1;                                         \
    }                                                   \
    if (kk == kEmptyKey) return 0;                      \
  }
  LB_SCAN_SLOT(q.s0, 0)
  LB_SCAN_SLOT(q.s1, 1)
  LB_SCAN_SLOT(q.s2, 2)
  LB_SCAN_SLOT(q.s3, 3)
#undef LB_SCAN_SLOT
  return -1;
}

// Resolves a lookup whose first bucket `bk` is already loaded; linear probing
// continues bucket by bucket while buckets are full.
template <typename Table>
__device__ __forceinline__ bool resolve(const Table& t, uint64_t key, uint64_t bk, const Bucket& first,
                                        uint32_t* slot, uint32_t* z, uint32_t* w, uint32_t* lines) {
  int r = scan_bucket(first, key, bk, slot, z, w);
  for (uint64_t it = 1; r < 0 && it < t.nbuckets; ++it) {
    bk = (bk + 1 == t.nbuckets) ? 0 : bk + 1;
    ++*lines;
    r = scan_bucket(load_bucket(t, bk), key, bk, slot, z, w);
  }
  return r == 1;
}

// log10 P(w | the last three words of history ctx) by Katz backoff over the
// hashed tables (Eq. (1), App. E.3), and the n-gram state after w.  The three
// bucket lines (orders 2, 3, 4) and the unigram are loaded together, then
// resolved; `lines` counts the bucket lines read.
struct LmResult {
  double lp;
  QState st;
};

// The n-gram context of a history node: its last word, the slots of its 2- and
// 3-word contexts and the three backoffs.
struct Ctx {
  int32_t word;
  uint32_t c2, c3;
  float bo1, bo2, bo3;
};

__device__ __forceinline__ Ctx ctx_of(const HistNode& h) {
  Ctx c;
  c.word = h.word;
  c.c2 = h.c2;
  c.c3 = h.c3;
  c.bo1 = h.bo1;
  c.bo2 = h.bo2;
  c.bo3 = h.bo3;
  return c;
}

__device__ __forceinline__ LmResult lm_lookup(const DevState& S, int32_t w, const Ctx& ctx, uint32_t* lines) {
  const uint64_t k2 = (static_cast<uint64_t>(static_cast<uint32_t>(ctx.word)) << 32) | static_cast<uint32_t>(w);
  const uint64_t k3 = (static_cast<uint64_t>(ctx.c2) << 32) | static_cast<uint32_t>(w);
  const uint64_t k4 = (static_cast<uint64_t>(ctx.c3) << 32) | static_cast<uint32_t>(w);
  const bool has3 = ctx.c2 != kNone;
  const bool has4 = ctx.c3 != kNone;
  const uint64_t b2 = bucket_of(k2, S.t2.nbuckets);
  const uint64_t b3 = has3 ? bucket_of(k3, S.t3.nbuckets) : 0;
  const uint64_t b4 = has4 ? bucket_of(k4, S.t4.nbuckets) : 0;
  const Bucket q2 = load_bucket(S.t2, b2);
  const Bucket q3 = has3 ? load_bucket(S.t3, b3) : Bucket{};
  const Bucket q4 = has4 ? load_bucket(S.t4, b4) : Bucket{};
  const Unigram u = S.uni[w];
  *lines += 1u + (has3 ? 1u : 0u) + (has4 ? 1u : 0u);
  uint32_t s2 = kNone, s3 = kNone, s4 = kNone;
  uint32_t z2 = 0, y2 = 0, z3 = 0, y3 = 0, z4 = 0, y4 = 0;
  const bool f2 = resolve(S.t2, k2, b2, q2, &s2, &z2, &y2, lines);
  const bool f3 = has3 && resolve(S.t3, k3, b3, q3, &s3, &z3, &y3, lines);
  const bool f4 = has4 && resolve(S.t4, k4, b4, q4, &s4, &z4, &y4, lines);
  const float p2 = __uint_as_float(z2), bb2 = __uint_as_float(y2), p3 = __uint_as_float(z3),
              bb3 = __uint_as_float(y3), p4 = __uint_as_float(z4);
  // log10 P(w | context) by backoff, innermost order first
  double lp;
  if (f4) {
    lp = static_cast<double>(p4);
  } else {
    double l3;
    if (f3) {
      l3 = static_cast<double>(p3);
    } else {
      const double l2 = f2 ? static_cast<double>(p2) : static_cast<double>(ctx.bo1) + static_cast<double>(u.logp);
      l3 = static_cast<double>(ctx.bo2) + l2;
    }
    lp = static_cast<double>(ctx.bo3) + l3;
  }
  LmResult r;
  r.lp = lp;
  r.st.c2 = f2 ? s2 : kNone;
  r.st.c3 = f3 ? s3 : kNone;
  r.st.bo2 = f2 ? bb2 : 0.0f;
  r.st.bo3 = f3 ? bb3 : 0.0f;
  r.st.w = w;
  r.st.bo1 = u.bo;
  return r;
}

// Identity of an n-gram query group: the context of a history node (its 3-word
// context slot if the LM has that trigram, else its 2-word context slot, else
// its last word; the backoff weights are functions of these) and the trie
// node of the completed word (by its first word offset, < 2^30).
__device__ __forceinline__ unsigned long long group_key(const Ctx& ctx, uint32_t woff) {
  const uint64_t tag = ctx.c3 != kNone ? 2u : (ctx.c2 != kNone ? 1u : 0u);
  const uint64_t id = ctx.c3 != kNone ? ctx.c3 : (ctx.c2 != kNone ? ctx.c2 : static_cast<uint32_t>(ctx.word));
  return (tag << 62) | (id << 30) | woff;
}

// The homophones of the node at word offset `woff` that have an explicit
// n-gram with context `ctx`, from the explicit-continuation index of orders 2,
// 3 and 4 (contexts: the last word, the 2-word slot, the 3-word slot).  The
// first buckets of the three probes are loaded together.  Order n's result is
// hit[n-2] = {a, count}: the index is `a` itself when count == 1, else
// lists[a..a+count).
struct PresHit {
  uint32_t a, n;
};

__device__ __forceinline__ void pres_lookup(const DevState& S, const Ctx& ctx, uint32_t woff, PresHit* hit,
                                            uint32_t* lines) {
  const uint64_t k2 = (static_cast<uint64_t>(static_cast<uint32_t>(ctx.word)) << 32) | woff;
  const uint64_t k3 = (static_cast<uint64_t>(ctx.c2) << 32) | woff;
  const uint64_t k4 = (static_cast<uint64_t>(ctx.c3) << 32) | woff;
  const bool has3 = ctx.c2 != kNone;
  const bool has4 = ctx.c3 != kNone;
  const uint64_t b2 = bucket_of(k2, S.p2.nbuckets);
  const uint64_t b3 = has3 ? bucket_of(k3, S.p3.nbuckets) : 0;
  const uint64_t b4 = has4 ? bucket_of(k4, S.p4.nbuckets) : 0;
  const Bucket q2 = load_bucket(S.p2, b2);
  const Bucket q3 = has3 ? load_bucket(S.p3, b3) : Bucket{};
  const Bucket q4 = has4 ? load_bucket(S.p4, b4) : Bucket{};
  *lines += 1u + (has3 ? 1u : 0u) + (has4 ? 1u : 0u);
  uint32_t slot;
  hit[0] = PresHit{0, 0};
  hit[1] = PresHit{0, 0};
  hit[2] = PresHit{0, 0};
  resolve(S.p2, k2, b2, q2, &slot, &hit[0].a, &hit[0].n, lines);
  if (has3) resolve(S.p3, k3, b3, q3, &slot, &hit[1].a, &hit[1].n, lines);
  if (has4) resolve(S.p4, k4, b4, q4, &slot, &hit[2].a, &hit[2].n, lines);
}

// ------------------------------------------------------------------ decoding loop

// A stream's hypotheses in LDS (structure of arrays); the fields of each
// hypothesis' trie node travel with it.
template <int KMAX>
struct BeamLds {
  uint64_t key[KMAX];
  uint64_t pkey[KMAX];
  uint64_t tmask[KMAX];  // trie child mask, separator bit, word count << 48
  double ab[KMAX];
  double anb[KMAX];
  double pt[KMAX];  // log-sum-exp(ab, anb)
  double Lw[KMAX * kMaxSub];
  uint32_t hist[KMAX * kMaxSub];
  uint32_t node[KMAX];
  uint32_t meta[KMAX];   // last symbol | number of sub-beams << 8
  uint32_t first[KMAX];  // the trie node's first child
  uint32_t woff[KMAX];   // the trie node's first word in trie_words
};

template <int NT, int N>
__device__ __forceinline__ void emit_output(const DevParams& P, const DevState& S, int b, const int32_t* lengths,
                                            int32_t Tc, int32_t fin, int32_t* out_hyps, float* out_scores, double* sc,
                                            uint64_t* ky, uint32_t* ix, int32_t* sScan);

// Frames [tau0, min(tau1, length)) of Alg. 1 for every stream: one workgroup
// per stream, which keeps the stream's beam in LDS from frame to frame.  Each
// frame:
//   * fan-out of every hypothesis by blank, repeat and each lexicon-valid
//     symbol (trie child mask), token / word bonuses, recombination of equal
//     prefixes by log-sum-exp, theta pruning, top-K selection (score bins,
//     exact rank inside the boundary bin), beam update, trie-state advance;
//     hypothesis i is owned by LPB consecutive lanes: lane s of it handles the
//     extensions v = 1+s, 1+s+LPB, ... and lane 0 also the merged stay;
//   * Eq. (1) for the hypotheses that completed a word (in batches of NEB
//     words): the (word, sub-beam) pairs are grouped by (n-gram context, trie
//     node); each group is looked up once per homophone, or, for a node with
//     many homophones, only for those the explicit-continuation index lists
//     (the others back off to their unigrams); the lookups are spread over all
//     threads; each word's top-o (one thread per word, or a wavefront for a
//     word with a large fully looked-up group) survive lambda pruning and
//     receive word-history nodes;
//   * Eq. (2) with the synthetic scorer on fusion frames.
// After the last frame the beam goes back to global memory, and, when out_hyps
// is given, the workgroup also writes the stream's output (emit_output; out_fin:
// the end of the utterance).
// WPE: wavefronts per SIMD the register allocation aims for (four workgroups
// of 256 threads per CU need 4).  DB: the hypotheses are double-buffered in
// LDS; otherwise one buffer is rewritten in place (every source entry is read
// before any new entry is written), which lets two K = 256 workgroups share a
// CU.  HSF: LDS hash slots per hypothesis for the prefix keys (more slots,
// shorter linear probe chains, more LDS).  The decoder's parameters and state
// (P, S) are read from their device copy A_ in constant memory.  opts bit 0
// (kOptPhaseTimers): thread 0 adds the clock cycles of each phase of the
// frame to the stream's phase counters (kCntPhase0 + kPh*).  scratch: when
// given, the n-gram lookup scratch of the call's streams (scratch_layout)
// instead of the decoder's own buffers.
template <int KMAX, int LPB, int WPE, bool DB, int HSF>
__global__ __launch_bounds__(KMAX * LPB) __attribute__((amdgpu_waves_per_eu(WPE))) void k_decode(
    const KArgs LB_CONST* A_, const float* __restrict__ logits, const int32_t* __restrict__ lengths, int32_t Tc,
    int32_t tau0, int32_t tau1, int32_t out_fin, int32_t* __restrict__ out_hyps, float* __restrict__ out_scores,
    uint32_t opts, unsigned char* __restrict__ scratch) {
  // P and S are read through a pointer that is made opaque in every frame, so
  // that each field is loaded (scalar, from the constant cache) where it is
  // used instead of staying live in scalar registers across the whole loop
  const KArgs LB_CONST* A = A_;
#define P (*(const DevParams*)(&A->P))
#define S (*(const DevState*)(&A->S))

  constexpr int BLOCK = KMAX * LPB;
  // LDS hash slots for the current prefix keys: a load of at most 1/4 keeps the
  // linear probe chains short (at 1/2, a parent that is not in the beam took
  // ~2.5 probes, and the whole frame 6 % longer)
  constexpr int HS = HSF * KMAX;
  static_assert(HSF >= 4 && (HSF & (HSF - 1)) == 0, "hash slots: a power of two, load at most 1/4");
  static_assert(KMAX <= 256, "a hash slot holds its hypothesis in 8 bits");
  constexpr int NW = BLOCK / 64;
  constexpr int NC = (kSep + LPB - 1) / LPB;  // extension slots per lane
  // top-K in one pass over the slots, with the bin range from bounds taken in
  // the recombination phase, where a lane owns 5 or more slots; with fewer
  // slots per lane a first pass for the exact range costs less than the bounds
  constexpr bool kOnePass = NC >= 5;
  static_assert(LPB <= 16 && LPB * NC < 64, "a lane's slots stay below symbol 64");
  static_assert(NC + 2 < 64, "a lane's candidates (its slots, the stay and the repeat) fit the sets sel_bits and bnd");
  // the candidate sets of a lane: 32 bits where its positions fit
  using CandSet = typename std::conditional<(NC + 2 <= 32), uint32_t, uint64_t>::type;
  constexpr int NPM = KMAX * kMaxSub;  // (completed word, sub-beam) pairs per frame, at most
  constexpr int NPL = NPM < 256 ? NPM : 256;  // pairs grouped at once
  constexpr int NEB = NPL / kMaxSub;          // completed words per batch
  // score bins of the top-K selection: 1024 at K = 256; 512 for the smaller
  // beams' fewer candidates (c5: 25.69 against 25.83 ms with 1024; c4 9.91
  // against 9.80 with 512)
  constexpr int kBinBits = KMAX >= 256 ? 10 : 9;
  constexpr int kBins = 1 << kBinBits;
  constexpr int SEL_BYTES = kBins * 4 + kBoundaryCap * 16;
  constexpr int LM_BYTES = 64 * NPL + 16;
  constexpr int UNI_BYTES = SEL_BYTES > LM_BYTES ? SEL_BYTES : LM_BYTES;
  static_assert(20 * KMAX <= SEL_BYTES, "fusion sort scratch");
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int len = lengths[b];
  const int tend = len < tau1 ? len : tau1;

  __shared__ BeamLds<KMAX> sBeam[DB ? 2 : 1];
  __shared__ double sD[64];  // classes 0..40; 41..63 are zero (slots past the separator)
  __shared__ double sDmax;   // the largest of sD[1..40]
  __shared__ double sAb2[KMAX], sAnb2[KMAX], sPt2[KMAX], sStay[KMAX];
  __shared__ uint64_t sMask[KMAX];
  // the prefix keys of the frame's hypotheses: inserted when the hypotheses
  // are written (in the previous frame, or when the beam is loaded), cleared
  // once this frame's parent lookups are done (the frame's later barriers
  // separate the clear from the next inserts)
  __shared__ unsigned long long sHKey[HS];
  __shared__ uint8_t sHIdx[HS];  // the slot's hypothesis (KMAX <= 256)
  // top-K selection scratch; the LM step and the fusion sort reuse it
  __shared__ __align__(16) unsigned char sSel[UNI_BYTES];
  __shared__ double sLvHi[kMaxLevels], sLvInv[kMaxLevels];
  __shared__ int32_t sLvBeta[kMaxLevels], sLvShift[kMaxLevels];
  __shared__ uint32_t sSelSrc[KMAX];
  // hypotheses that completed a word this frame
  __shared__ uint32_t sEvBeam[KMAX], sEvWoff[KMAX], sEvH[KMAX];
  __shared__ int32_t sNG, sHeavy, sNLarge;
  __shared__ int32_t sLarge[KMAX];  // completed words ranked by a whole wavefront
  __shared__ double sRed[2 * NW], sRedB[3 * NW];
  __shared__ int32_t sScan[NW], sScanB[NW], sScanC[NW], sScanD[NW];
  __shared__ int32_t sBucket, sAbove, sBucketCnt, sBCount, sAthr, sNBinned;
  // counters: probed lines, completed words, LM queries, index lines (summed over
  // the threads at the end), expansions, fused hypotheses, lookups (added by
  // thread 0 as they occur: kept here, not in every thread's registers)
  __shared__ unsigned long long sCnt[7];
  // phase cycles of thread 0 (kPh*), and the last timestamp
  __shared__ unsigned long long sPhase[kPhases + 1];
  // the log-sum-exp's series coefficients (log1p_unit), read from LDS
  __shared__ double sAtanh[kAtanhTerms];
  const bool timing = (opts & kOptPhaseTimers) != 0;
  // closes the current phase as phase k (taken after the barrier that ends it)
  auto mark = [&](int k) {
    if (timing && threadIdx.x == 0) {
      const unsigned long long now = __builtin_amdgcn_s_memtime();
      sPhase[k] += now - sPhase[kPhases];
      sPhase[kPhases] = now;
    }
  };

  uint32_t* const sHisto = reinterpret_cast<uint32_t*>(sSel);
  double* const sBScore = reinterpret_cast<double*>(sSel + kBins * 4);
  uint64_t* const sBKey = reinterpret_cast<uint64_t*>(sSel + kBins * 4 + kBoundaryCap * 8);
  // write-back staging of the sub-beams (one-buffer instances), past the
  // grouping keys that the write-back clears
  double* const sStL = reinterpret_cast<double*>(sSel + 8 * NPL);
  uint32_t* const sStH = reinterpret_cast<uint32_t*>(sStL + KMAX * kMaxSub);
  static_assert(DB || 8 * NPL + 12 * KMAX * kMaxSub <= UNI_BYTES, "write-back staging fits the shared scratch");
  // the output (when this launch writes it) sorts in the shared scratch
  auto output = [&](const DevParams& Pr, const DevState& Sr) {
    emit_output<BLOCK, KMAX>(Pr, Sr, b, lengths, Tc, out_fin, out_hyps, out_scores, reinterpret_cast<double*>(sSel),
                             reinterpret_cast<uint64_t*>(sSel + 8 * KMAX),
                             reinterpret_cast<uint32_t*>(sSel + 16 * KMAX), sScan);
  };
  if (tau0 >= tend) {  // no frames of this stream in the launch
    if (out_hyps) output(P, S);
    return;
  }

  const size_t gb = static_cast<size_t>(b) * P.K;
  const int O = P.O;
  const bool synth = P.fusion_source == 1;
  const bool fuse_frames = synth && P.fusion_interval > 0;
  const int64_t t0 = S.t0[b];
  const uint32_t arena0 = 1u + static_cast<uint32_t>(static_cast<uint64_t>(b) * S.arena_cap);

  // ---- the stream's beam into LDS
  int n = S.nbeam[b];
  if (tid < n) {
    BeamLds<KMAX>& B0 = sBeam[0];
    const size_t g = gb + tid;
    B0.key[tid] = S.key[g];
    B0.pkey[tid] = S.pkey[g];
    B0.ab[tid] = S.ab[g];
    B0.anb[tid] = S.anb[g];
    B0.pt[tid] = S.pt[g];
    const uint32_t node = S.node[g];
    const uint32_t meta = S.meta[g];
    B0.node[tid] = node;
    B0.meta[tid] = meta;
    const int nsub = (meta >> 8) & 0xFF;
    for (int j = 0; j < nsub; ++j) {
      B0.Lw[tid * kMaxSub + j] = S.Lw[g * O + j];
      B0.hist[tid * kMaxSub + j] = S.hist[g * O + j];
    }
    const TrieNode tn = S.trie[node];
    B0.tmask[tid] = tn.mask;
    B0.first[tid] = tn.first_child;
    B0.woff[tid] = tn.word_off;
  }
  if (tid < 7) sCnt[tid] = 0;
  if (tid < kAtanhTerms) sAtanh[tid] = 1.0 / (2 * tid + 3);
  if (timing && tid == 0) {
    for (int k = 0; k < kPhases; ++k) sPhase[k] = 0;
    sPhase[kPhases] = __builtin_amdgcn_s_memtime();
  }
  uint32_t arena_n = S.arena_n[b];
  int cur = 0;  // the current buffer (DB)
  for (int q = tid; q < HS; q += BLOCK) sHKey[q] = kEmptyKey;
  // a new hypothesis' prefix key into the hash table, with its index r
  auto insert_key = [&](uint64_t key, int r) {
    uint32_t s = static_cast<uint32_t>(key) & (HS - 1);
    for (;;) {
      const unsigned long long prev = atomicCAS(&sHKey[s], kEmptyKey, key);
      if (prev == kEmptyKey) {
        sHIdx[s] = static_cast<uint8_t>(r);
        break;
      }
      s = (s + 1) & (HS - 1);
    }
  };
  uint32_t lines = 0, plines = 0, c_words = 0;  // per thread
  uint64_t c_queries = 0;
  const ScratchLayout slay = scratch_layout(gridDim.x, S.scap, P.K);
  double* const scrL = (scratch ? reinterpret_cast<double*>(scratch) : S.scrL) + static_cast<size_t>(b) * S.scap;
  QState* const scrS =
      (scratch ? reinterpret_cast<QState*>(scratch + slay.off_state) : S.scrS) + static_cast<size_t>(b) * S.scap;
  uint32_t* const scrE = (scratch ? reinterpret_cast<uint32_t*>(scratch + slay.off_explicit) : S.scrE) +
                         static_cast<size_t>(b) * P.K * kMaxSub * kMaxExplicit;
  // D = alpha * log-probs of a frame into sD, by wavefront 0 (every lane):
  // raw scores are first normalised by a log-softmax over the 41 classes
  auto set_row = [&](const DevParams& Pr, float xin) {
    double x = lane < kClasses ? static_cast<double>(xin) : kNegInf;
    if (Pr.raw_input) {
      double m = x, unused = x;
      wave_minmax(&m, &unused);
      const double sum = wave_sum(lane < kClasses ? exp(x - m) : 0.0);
      x = (x - m) - log(sum);
    }
    const double dv = lane < kClasses ? Pr.alpha * x : 0.0;
    sD[lane] = dv;
    const double dm = wave_max(lane >= 1 && lane < kClasses ? dv : kNegInf);
    if (lane == 0) sDmax = dm;
  };
  // the first frame's row now; each frame loads the next frame's row early and
  // writes it to sD after the frame's last global wait
  if (wave == 0)
    set_row(P, lane < kClasses ? logits[(static_cast<size_t>(b) * Tc + tau0) * kClasses + lane] : 0.0f);
  float dnext = 0.0f;
  lds_barrier();
  // the loaded hypotheses' keys and trie masks for the first frame
  if (tid < n) {
    insert_key(sBeam[0].key[tid], tid);
    sMask[tid] = sBeam[0].tmask[tid];
  }
  lds_barrier();
  mark(kPhOther);

  for (int tau = tau0; tau < tend; ++tau) {
    // the thread index is made opaque to the optimizer in every frame so that
    // values derived from it are not hoisted out of the loop (they would stay
    // live in registers across all frames)
    int tid = threadIdx.x;
    asm volatile("" : "+v"(tid));
    asm volatile("" : "+s"(A));
    const int lane = tid & 63;
    const int wave = tid >> 6;
    BeamLds<KMAX>& C = sBeam[DB ? cur : 0];        // the frame's hypotheses
    BeamLds<KMAX>& N = sBeam[DB ? (cur ^ 1) : 0];  // the new ones (the same buffer when !DB)

    // the next frame's log-probs are loaded meanwhile
    if (tid < kClasses && tau + 1 < tend) dnext = logits[(static_cast<size_t>(b) * Tc + tau + 1) * kClasses + tid];
    unsigned long long* const hkey = sHKey;  // the frame's prefix keys (inserted with the hypotheses)
    for (int d = tid; d < kBins; d += BLOCK) sHisto[d] = 0;
    if (tid == 0) sBCount = 0;
    uint64_t my_pkey = kNoParent;
    uint32_t my_meta = 0;
    if (tid < n) {
      my_pkey = C.pkey[tid];
      my_meta = C.meta[tid];
    }

    // ---- recombination: a hypothesis whose parent prefix is also live receives
    // the parent's extension by its last symbol; that extension is removed from
    // the parent's fan-out.  Stay candidates: blank-stay, repeat-stay, merged
    // parent extension.
    double st = kNegInf, up = kNegInf;  // this hypothesis' stay score and extension bound
    if (tid < n) {
      int par = -1;
      if (my_pkey != kNoParent) {
        uint32_t s = static_cast<uint32_t>(my_pkey) & (HS - 1);
        for (int probes = 0; probes < HS; ++probes) {
          const unsigned long long k = hkey[s];
          if (k == kEmptyKey) break;
          if (k == my_pkey) {
            par = static_cast<int>(sHIdx[s]);
            break;
          }
          s = (s + 1) & (HS - 1);
        }
        if (par >= 0) atomicAnd(reinterpret_cast<unsigned long long*>(&sMask[par]), ~(1ull << (my_meta & 0xFF)));
      }
      const int last = my_meta & 0xFF;
      const double ab2 = C.pt[tid] + sD[0];
      const double rep = last ? C.anb[tid] + sD[last] : kNegInf;
      double ext = kNegInf;
      if (par >= 0) {
        const double base = (last == static_cast<int>(C.meta[par] & 0xFF)) ? C.ab[par] : C.pt[par];
        ext = (base + sD[last]) + (last == kSep ? P.gamma : P.beta);
      }
      // anb2 = merge(rep, ext), then pt2 = merge(ab2, anb2); merge is
      // log-sum-exp, or max for the best-alignment recombination
      double x = rep, y = ext, anb2 = 0.0;
#pragma unroll 1
      for (int pass = 0; pass < 2; ++pass) {
        const double l = P.merge_max ? fmax(x, y) : lse2(x, y, [&](int k) { return sAtanh[k]; });
        if (pass == 0) {
          anb2 = l;
          x = ab2;
          y = l;
        } else {
          y = l;
        }
      }
      const double pt2 = y;
      sAb2[tid] = ab2;
      sAnb2[tid] = anb2;
      sPt2[tid] = pt2;
      st = pt2 + C.Lw[tid * kMaxSub];
      sStay[tid] = st;
      // no extension of this hypothesis scores above this (each of the additions
      // rounds monotonically, base <= pt, log-prob <= sDmax, bonus <= the larger)
      if constexpr (kOnePass) up = ((C.pt[tid] + sDmax) + fmax(P.beta, P.gamma)) + C.Lw[tid * kMaxSub];
    }
    if constexpr (kOnePass) {
      // per wavefront: an upper bound of every candidate (sRedB[w]), the best
      // stay (sRedB[NW + w]) and the lowest (sRedB[2 NW + w]), for the top-K's
      // bin range (a wavefront past the last hypothesis, e.g. the upper half
      // of the block when there is one thread per hypothesis here but two
      // lanes per hypothesis later, has the neutral values without reducing)
      if (wave * 64 < n) {
        double hi = fmax(st, up), nlo = -st;
        wave_minmax(&hi, &nlo);
        const double nmin = wave_max(tid < n ? -st : -HUGE_VAL);
        if (lane == 0) {
          sRedB[wave] = hi;
          sRedB[NW + wave] = -nlo;
          sRedB[2 * NW + wave] = -nmin;
        }
      } else if (lane == 0) {
        sRedB[wave] = kNegInf;
        sRedB[NW + wave] = kNegInf;
        sRedB[2 * NW + wave] = HUGE_VAL;
      }
    }
    lds_barrier();
    mark(kPhRecomb);
    for (int s = tid; s < HS; s += BLOCK) sHKey[s] = kEmptyKey;  // for the new hypotheses' keys
    // Workgroups that share a CU: the CU's arbitration favours the older
    // wavefronts, so the workgroup dispatched second (the later half of the
    // grid, when workgroups are dispatched to the CUs in order) fell behind
    // (c4: 9.8 against 11.1 ms on average) and the launch waited for it.  It
    // gets the higher issue priority in 3 frames of 4, the first one in the
    // 4th (c4: 12.3 -> 11.7 ms; alternating 1:1 gave 12.1).
    if ((blockIdx.x >= gridDim.x / 2) ? (tau & 3) != 0 : (tau & 3) == 0)
      __builtin_amdgcn_s_setprio(1);
    else
      __builtin_amdgcn_s_setprio(0);

    // ---- this lane's candidates: slot k is the extension by v = 1 + ln + LPB*k,
    // plus the merged stay on lane 0; scores are recomputed in every pass (same
    // operations, same result)
    const int hi_ = tid / LPB;
    const int ln = tid - hi_ * LPB;
    const bool live = hi_ < n;
    uint64_t c_key = 0, c_rel = 0;
    double c_stay = kNegInf, c_ab = 0.0, c_p = 0.0, c_L = 0.0;
    int c_rep = -1;
    if (live) {
      c_ab = C.ab[hi_];
      c_p = C.pt[hi_];
      c_L = C.Lw[hi_ * kMaxSub];
      // slot k <-> symbol 1 + ln + LPB*k: bit LPB*k of c_rel is its mask bit
      // (slots past the separator are invalid: the mask is cut to bits 1..40,
      // its bits 48..63 hold the node's word count)
      c_rel = (sMask[hi_] & ((2ull << kSep) - 1ull)) >> (1 + ln);
      c_rep = static_cast<int>(C.meta[hi_] & 0xFF) - 1 - ln;  // LPB*k of the repeat symbol
      c_key = C.key[hi_];
      if (ln == 0) c_stay = sStay[hi_];
    }
    // the separator (symbol kSep = 1 + ln + LPB*k) can only be slot
    // (kSep - 1) / LPB of lane (kSep - 1) % LPB: with k known at compile time
    // (the unrolled slot loops) the bonus of every other slot is beta without
    // a select
    constexpr int kSepSlot = (kSep - 1) / LPB;
    const bool sep_lane = ln == (kSep - 1) % LPB;
    // (the bonuses are read once here: inside the slot loops a constant-memory
    // load per slot would wait together with the LDS loads)
    const double bon_ph = P.beta, bon_sep = P.gamma;
    auto bonus_at = [&](int k) -> double { return (k == kSepSlot && sep_lane) ? bon_sep : bon_ph; };
    // the repeat extension (the hypothesis' last symbol again, from its
    // blank-ending part) is a candidate of its own, position NC + 1, and its
    // slot is left out of the slot loops, whose extensions all start from pt
    int c_rk = -1;            // its slot on this lane (-1: not on this lane, or invalid)
    double c_rps = kNegInf;   // its score
    if (c_rep >= 0 && c_rep % LPB == 0 && ((c_rel >> c_rep) & 1ull)) {
      c_rk = c_rep / LPB;
      c_rps = ((c_ab + sD[1 + ln + c_rep]) + bonus_at(c_rk)) + c_L;
      c_rel &= ~(1ull << c_rep);
    }
    auto score_now = [&](int k) -> double {
      const bool valid = (c_rel >> (LPB * k)) & 1ull;
      const double sc = ((c_p + sD[1 + ln + LPB * k]) + bonus_at(k)) + c_L;
      return valid ? sc : kNegInf;
    };
    auto key_of = [&](int v) -> uint64_t { return v == 0 ? c_key : prefix_step(c_key, v); };
    // position k of the lane: slot k (k < NC), the stay (NC), the repeat (NC + 1)
    auto pos_v = [&](int k) -> int { return k == NC ? 0 : 1 + ln + LPB * (k == NC + 1 ? c_rk : k); };
    auto pos_score = [&](int k) -> double { return k == NC ? c_stay : (k == NC + 1 ? c_rps : score_now(k)); };

    // ---- top-K and the theta cut.  Level 0 bins the candidates at or above L0
    // by (U - score) over [L0, U] into kBins, where U is at least every
    // candidate's score and L0 at most every candidate that can be selected:
    // at most the cut (best - theta) or at most the K-th candidate (with a
    // full beam the K stays are candidates, so the K-th candidate scores at
    // least the lowest stay).  The map is monotone, so bins above the one
    // holding the K-th candidate are taken whole, and the bins above the
    // cut's bin hold only candidates above the cut.  U and L0 come from the
    // recombination phase's bounds (U: the stays and each hypothesis'
    // extension bound; L0: the best stay - theta, or the lowest stay if the
    // beam is full and that is higher), so one pass over the slots bins them;
    // the exact best is taken only where the cut might bind (below), and then
    // the members of the cut's bin are tested against the cut exactly.
    // Without a finite stay (and in the instances without bounds) a first
    // pass finds best and the lowest candidate: U = best, L0 = max(best -
    // theta, lowest).  The bin holding the K-th candidate is resolved exactly
    // by rank on (score desc, key asc) when it holds at most kBoundaryCap
    // candidates; otherwise it is re-binned over its own score range (deeper
    // levels), and when its scores are all equal, by the bits of the key
    // (smaller key first).
    const double theta = P.theta;
    double U = kNegInf, Bst = kNegInf, Smin = kNegInf;
    if constexpr (kOnePass) {
      U = sRedB[0];
      Bst = sRedB[NW];
      Smin = sRedB[2 * NW];
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        U = fmax(U, sRedB[w]);
        Bst = fmax(Bst, sRedB[NW + w]);
        Smin = fmin(Smin, sRedB[2 * NW + w]);
      }
    }
    double L0 = Bst - theta;
    if (n >= P.K) L0 = fmax(L0, Smin);  // (a stay of -inf leaves Smin at -inf)
    // with a first pass the best is exact before the binning (and every binned
    // candidate is at or above the cut)
    const bool first_pass = Bst == kNegInf;  // no bounds, or no finite stay (uniform)
    double best = kNegInf;
    if (first_pass) {
      double mx = fmax(c_stay, c_rps);
      double mn = fmin(c_stay != kNegInf ? c_stay : HUGE_VAL, c_rps != kNegInf ? c_rps : HUGE_VAL);
#pragma unroll
      for (int k = 0; k < NC; ++k) {
        const double sc = score_now(k);
        mx = fmax(mx, sc);
        mn = fmin(mn, sc != kNegInf ? sc : HUGE_VAL);
      }
      double lowest;
      block_minmax<BLOCK, false>(mx, mn, sRed, &best, &lowest);
      U = best;
      L0 = fmax(best - theta, lowest);
    }
    const double inv0 = U > L0 ? static_cast<double>(kBins) / (U - L0) : 0.0;
    const int shift0 = U > L0 ? -1 : 64 - kBinBits;
    auto bin_score = [&](double hi, double inv, double s) -> int {
      const double x = (hi - s) * inv;
      return x >= static_cast<double>(kBins - 1) ? kBins - 1 : static_cast<int>(x);
    };
    // level 0: (U - s) * inv0 as one fused multiply-add of s, clamped to the
    // bins; each step rounds monotonically, so a higher score never takes a
    // higher bin (U bounds every candidate, so the value is at least about 0)
    const double ninv0 = -inv0, uinv0 = U * inv0;
    auto bin_lv0 = [&](double s) -> int {
      return static_cast<int>(fmax(fmin(fma(s, ninv0, uinv0), static_cast<double>(kBins - 1)), 0.0));
    };
    auto bin0 = [&](int v, double s) -> int {
      return shift0 < 0 ? bin_lv0(s) : static_cast<int>((key_of(v) >> shift0) & (kBins - 1));
    };
    // deeper levels (rare): parameters in LDS
    auto bin_at = [&](int l, int v, double s) -> int {
      const int sh = sLvShift[l];
      if (sh >= 0) return static_cast<int>((key_of(v) >> sh) & (kBins - 1));
      return bin_score(sLvHi[l], sLvInv[l], s);
    };
    // finds the bin holding the need-th candidate of sHisto (sBucket, sAbove,
    // sBucketCnt) and, for bthr < kBins, the number of candidates in the bins
    // above bin bthr (sAthr); returns the number of binned candidates.  The
    // first wavefront scans the bins, kBins / 64 per lane, so one barrier ends it.
    auto find_bin = [&](int need_in, int bthr) -> int {
      constexpr int PERW = kBins / 64;
      static_assert(PERW % 4 == 0, "bins per lane in 16-B loads");
      if (wave == 0) {
        int h[PERW];
        const uint4* hp = reinterpret_cast<const uint4*>(sHisto + lane * PERW);
#pragma unroll
        for (int q = 0; q < PERW / 4; ++q) {
          const uint4 x4 = hp[q];
          h[4 * q] = static_cast<int>(x4.x);
          h[4 * q + 1] = static_cast<int>(x4.y);
          h[4 * q + 2] = static_cast<int>(x4.z);
          h[4 * q + 3] = static_cast<int>(x4.w);
        }
        int local = 0;
#pragma unroll
        for (int q = 0; q < PERW; ++q) local += h[q];
        const int incl = wave_scan_incl(local);
        const int before = incl - local;
        if (lane == 63) sNBinned = incl;
        if (need_in > 0 && before < need_in && incl >= need_in) {
          int acc = before;
          bool found = false;
#pragma unroll
          for (int q = 0; q < PERW; ++q) {
            if (!found && acc + h[q] >= need_in) {
              sBucket = lane * PERW + q;
              sAbove = acc;
              sBucketCnt = h[q];
              found = true;
            }
            acc += h[q];
          }
        }
        if (bthr < kBins && lane == bthr / PERW) {
          int acc = before;
#pragma unroll
          for (int q = 0; q < PERW; ++q) acc += (lane * PERW + q < bthr) ? h[q] : 0;
          sAthr = acc;
        }
      }
      lds_barrier();
      return sNBinned;
    };

    // level-0 bin of each of the lane's candidates, kept packed 16 bits per slot
    // (0xFFFF: no candidate); exact scores are recomputed only inside the boundary bin
    uint32_t binp[(NC + 1) / 2];
    // (with several lanes per hypothesis the candidates' inputs are made opaque
    // here so that their scores are recomputed below instead of being kept live
    // across the block reduction; the one-lane instance has the registers)
    if constexpr (LPB > 1) asm volatile("" : "+v"(c_ab), "+v"(c_p), "+v"(c_L), "+v"(c_rel), "+v"(c_key));
    uint32_t bin_stay = 0xFFFFu, bin_rep = 0xFFFFu;
    if (c_stay >= L0) bin_stay = static_cast<uint32_t>(bin0(0, c_stay));  // (-inf: no stay)
    if (c_rps >= L0) bin_rep = static_cast<uint32_t>(bin0(pos_v(NC + 1), c_rps));
    // the bins first, then the histogram: with no LDS write among them, the
    // slots' log-prob loads are issued together instead of each waiting behind
    // the previous slot's atomic
    if (shift0 < 0) {
#pragma unroll
      for (int k = 0; k < NC; ++k) {
        // branch-free: the score and bin of the slot, valid or not (a bin in
        // range either way), then a select
        const bool valid = (c_rel >> (LPB * k)) & 1ull;
        const double sc = ((c_p + sD[1 + ln + LPB * k]) + bonus_at(k)) + c_L;
        const bool in = valid && sc >= L0;
        const uint32_t bn = in ? static_cast<uint32_t>(bin_lv0(sc)) : 0xFFFFu;
        if (k & 1)
          binp[k >> 1] |= bn << 16;
        else
          binp[k >> 1] = bn;
      }
    } else {
      // every candidate in range has the same score: bins by key bits
#pragma unroll
      for (int k = 0; k < NC; ++k) {
        const double sc = score_now(k);
        const bool in = sc >= L0;
        const uint32_t bn = in ? static_cast<uint32_t>(bin0(1 + ln + LPB * k, sc)) : 0xFFFFu;
        if (k & 1)
          binp[k >> 1] |= bn << 16;
        else
          binp[k >> 1] = bn;
      }
    }
    if (bin_stay != 0xFFFFu) atomicAdd(&sHisto[bin_stay], 1u);
    if (bin_rep != 0xFFFFu) atomicAdd(&sHisto[bin_rep], 1u);
#pragma unroll
    for (int k = 0; k < NC; ++k) {
      const uint32_t bn = (binp[k >> 1] >> ((k & 1) * 16)) & 0xFFFFu;
      if (bn != 0xFFFFu) atomicAdd(&sHisto[bn], 1u);
    }
    lds_barrier();
    // With bounds, the exact best is needed only if the K-th candidate may lie
    // at or below U - theta (>= best - theta): when it lies in a bin above that
    // value's, every candidate up to it is above the cut, which cannot bind.
    int nbinned = 0, bthr = kBins;
    bool exact_cut = first_pass;
    if (!first_pass) {
      const double thr_hi = U - theta;
      const int bhi = (shift0 < 0 && thr_hi > L0) ? bin_lv0(thr_hi) : kBins;
      nbinned = find_bin(P.K, kBins);
      if (!(nbinned >= P.K && sBucket < bhi)) {
        double mx = fmax(c_stay, c_rps);
#pragma unroll
        for (int k = 0; k < NC; ++k) mx = fmax(mx, score_now(k));
        best = block_max<BLOCK>(mx, sRed);
        exact_cut = true;
      }
    }
    const double thr = best - theta;  // (read only with exact_cut)
    if (exact_cut) {
      // the cut's bin (kBins: every binned candidate is at or above the cut)
      bthr = (shift0 < 0 && thr > L0) ? bin_lv0(thr) : kBins;
      nbinned = find_bin(P.K, bthr);
    }
    // three cases: the K-th candidate lies above the cut's bin (resolve its
    // bin); every candidate is selected; or the cut's bin decides (its members
    // at or above the cut, as many as are still needed)
    int beta0 = kBins, nlev = 1, need = 0, nbc = 0, cntb = 0;
    bool all_bin = false, resolve = false, cutbin = false;
    if (nbinned >= P.K && sBucket < bthr) {
      beta0 = sBucket;
      need = P.K - sAbove;
      cntb = sBucketCnt;
      resolve = true;
    } else if (bthr < kBins) {
      beta0 = bthr;
      need = P.K - sAthr;
      cutbin = true;
    }
    // level 0 decides every candidate outside the boundary bin: above it taken,
    // below it dropped; bnd marks this lane's candidates inside it (bit k: slot
    // k, bit NC: the stay)
    CandSet sel_bits = 0;  // bit 0: the stay, bit k+1: slot k
    CandSet bnd = 0;
    // lowest set bit and population count of a candidate set
    auto set_ffs = [](CandSet m) -> int {
      if constexpr (sizeof(CandSet) == 4) return __ffs(m) - 1;
      else return __ffsll(static_cast<unsigned long long>(m)) - 1;
    };
    auto set_popc = [](CandSet m) -> int {
      if constexpr (sizeof(CandSet) == 4) return __popc(m);
      else return __popcll(m);
    };
    // (branch-free: 0xFFFF, no candidate, is above every bin index; the two
    // sets are updated separately so that they stay in registers)
    auto classify = [&](uint32_t bn, int bit, int bbit) {
      sel_bits |= static_cast<CandSet>(static_cast<int>(bn) < beta0) << bit;
      bnd |= static_cast<CandSet>(static_cast<int>(bn) == beta0) << bbit;
    };
    classify(bin_stay, 0, NC);
    classify(bin_rep, NC + 1, NC + 1);
#pragma unroll
    for (int k = 0; k < NC; ++k) classify((binp[k >> 1] >> ((k & 1) * 16)) & 0xFFFFu, k + 1, k);
    if (cutbin) {
      // the cut's bin: members below the cut are no candidates.  When the bin
      // is small (the usual case) its members at or above the cut go straight
      // to the exact rank, whose list also counts them; otherwise they are
      // counted first and the bin is refined like any boundary bin.
      const bool small = static_cast<int>(sHisto[bthr]) <= kBoundaryCap;  // (uniform)
#pragma unroll 1
      for (CandSet m = bnd; m; m &= m - 1) {
        const int k = set_ffs(m);
        const double sc = pos_score(k);
        if (!(sc >= thr)) {
          bnd &= ~(CandSet{1} << k);
        } else if (small) {
          const int slot = atomicAdd(&sBCount, 1);
          sBScore[slot] = sc;
          sBKey[slot] = key_of(pos_v(k));
        }
      }
      if (small) {
        lds_barrier();
        nbc = sBCount;
        cntb = nbc;
        all_bin = cntb <= need;  // else: ranked exactly below
      } else {
        int cnt = 0;
        (void)block_scan<BLOCK>(set_popc(bnd), sScanD, &cnt);
        cntb = cnt;
        if (cntb <= need)
          all_bin = true;
        else
          resolve = true;
      }
    }
    // the lane's boundary-bin candidates (v, exact score) that also lie in the
    // boundary bins of levels 1..L-1
    auto for_bnd = [&](int L, auto&& f) {
#pragma unroll 1
      for (CandSet m = bnd; m; m &= m - 1) {
        const int k = set_ffs(m);
        const int v = pos_v(k);
        const double sc = pos_score(k);
        bool in = true;
        for (int l = 1; l < L && in; ++l) in = bin_at(l, v, sc) == sLvBeta[l];
        if (in) f(k, v, sc);
      }
    };
    if (resolve) {
      int key_shift = shift0 >= 0 ? shift0 - kBinBits : 64 - kBinBits;
      bool key_level = shift0 >= 0;
      int last_shift = shift0;  // shift of the deepest level (-1: score bins)
      while (cntb != need && cntb > kBoundaryCap && !(key_level && last_shift == 0) && nlev < kMaxLevels) {
        // refine: score range of the boundary bin's members, or key bits when it is flat
        const int L = nlev;
        double bmx = kNegInf, bmn = HUGE_VAL;
        for_bnd(L, [&](int, int, double sc) {
          bmx = fmax(bmx, sc);
          bmn = fmin(bmn, sc);
        });
        double lv_hi, lv_lo;
        block_minmax<BLOCK>(bmx, bmn, sRedB, &lv_hi, &lv_lo);
        if (tid == 0) {
          sLvHi[L] = lv_hi;
          sLvInv[L] = lv_hi > lv_lo ? static_cast<double>(kBins) / (lv_hi - lv_lo) : 0.0;
          sLvShift[L] = lv_hi > lv_lo ? -1 : (key_shift > 0 ? key_shift : 0);
        }
        for (int d = tid; d < kBins; d += BLOCK) sHisto[d] = 0;
        lds_barrier();
        last_shift = sLvShift[L];
        key_level = last_shift >= 0;
        if (key_level) key_shift -= kBinBits;
        for_bnd(L, [&](int, int v, double sc) { atomicAdd(&sHisto[bin_at(L, v, sc)], 1u); });
        lds_barrier();
        (void)find_bin(need, kBins);
        if (tid == 0) sLvBeta[L] = sBucket;
        need -= sAbove;
        cntb = sBucketCnt;
        nlev = L + 1;
        lds_barrier();
      }
      if (cntb == need) {
        all_bin = true;
      } else {
        // exact rank inside the boundary bin (a flat key level of shift 0 holds one
        // key); sBCount was cleared at the start of the frame
        for_bnd(nlev, [&](int, int v, double sc) {
          const int slot = atomicAdd(&sBCount, 1);
          if (slot < kBoundaryCap) {
            sBScore[slot] = sc;
            sBKey[slot] = key_of(v);
          }
        });
        lds_barrier();
        nbc = sBCount < kBoundaryCap ? sBCount : kBoundaryCap;
        if (sBCount > kBoundaryCap && tid == 0) atomicOr(S.flags, kFlagSelect);
      }
    }
    // the boundary bin's candidates: the deeper levels, then the exact rank on
    // (score desc, key asc)
#pragma unroll 1
    for (CandSet m = bnd; m; m &= m - 1) {
      const int k = set_ffs(m);
      const int v = pos_v(k);
      const double sc = pos_score(k);
      bool take = true;
      bool decided = false;
      for (int l = 1; l < nlev && !decided; ++l) {
        const int bl = bin_at(l, v, sc);
        if (bl != sLvBeta[l]) {
          take = bl < sLvBeta[l];
          decided = true;
        }
      }
      if (!decided && !all_bin) {
        const uint64_t key = key_of(v);
        int rank = 0;
        for (int u = 0; u < nbc; ++u) rank += ranks_before(sBScore[u], sBKey[u], sc, key);
        take = rank < need;
      }
      if (take) sel_bits |= CandSet{1} << (k == NC ? 0 : (k == NC + 1 ? NC + 1 : k + 1));
    }
    int nsel = 0;
    int wpos = block_scan<BLOCK, false>(set_popc(sel_bits), sScanB, &nsel);
    if (nsel > P.K) {  // cannot happen when the selection is exact; never write past K entries
      nsel = P.K;
      if (tid == 0) atomicOr(S.flags, kFlagSelect);
    }
#pragma unroll 1
    for (CandSet m = sel_bits; m && wpos < nsel; m &= m - 1) {
      const int bit = set_ffs(m);
      const uint32_t v = static_cast<uint32_t>(pos_v(bit == 0 ? NC : (bit == NC + 1 ? NC + 1 : bit - 1)));
      sSelSrc[wpos++] = static_cast<uint32_t>(hi_) | (v << 16);
    }
    lds_barrier();
    mark(kPhTopK);

    // ---- the new hypotheses; an extension's trie node is fetched now and
    // stored after the LM step.  (The n-gram grouping table is cleared here:
    // the top-K scratch it shares is no longer read.)
    {
      unsigned long long* const gk = reinterpret_cast<unsigned long long*>(sSel);
      for (int q = tid; q < NPL; q += BLOCK) gk[q] = kEmptyKey;
      if (tid == 0) {
        sNG = 0;
        sHeavy = 0;
        sNLarge = 0;
      }
    }
    const int r = tid;
    int is_event = 0;
    uint32_t ev_woff = 0, ev_H = 0;
    bool tn_load = false;
    TrieNode tn{};
    // every new entry's fields from its source, into registers first
    uint64_t w_key = 0, w_pkey = 0, w_tmask = 0;
    double w_ab = 0.0, w_anb = 0.0, w_pt = 0.0;
    uint32_t w_node = 0, w_meta = 0, w_first = 0, w_woff = 0;
    if (r < nsel) {
      const uint32_t src = sSelSrc[r];
      const int i = src & 0xFFFF;
      const int v = src >> 16;
      const uint32_t meta_i = C.meta[i];
      if (v == 0) {
        w_key = C.key[i];
        w_pkey = C.pkey[i];
        w_ab = sAb2[i];
        w_anb = sAnb2[i];
        w_pt = sPt2[i];
        w_node = C.node[i];
        w_meta = meta_i;
        w_tmask = C.tmask[i];
        w_first = C.first[i];
        w_woff = C.woff[i];
      } else {
        const int last = meta_i & 0xFF;
        const double base = (v == last) ? C.ab[i] : C.pt[i];
        const double anb = (base + sD[v]) + (v == kSep ? P.gamma : P.beta);
        const uint64_t tm = C.tmask[i];
        w_key = prefix_step(C.key[i], v);
        w_pkey = C.key[i];
        w_ab = kNegInf;
        w_anb = anb;
        w_pt = anb;  // log-sum-exp(-inf, anb)
        uint32_t child = kRootNode;
        if (v != kSep) child = C.first[i] + __popcll(tm & ((1ull << v) - 1ull));
        w_node = child;
        w_meta = static_cast<uint32_t>(v) | (meta_i & 0xFF00u);
        tn = S.trie[child];
        tn_load = true;
        if (v == kSep) {
          is_event = 1;
          ev_woff = C.woff[i];
          ev_H = static_cast<uint32_t>(tm >> kWordCountShift);
        }
      }
      const int nsub = (meta_i >> 8) & 0xFF;
      if constexpr (DB) {
        // two buffers: the sub-beams are copied straight across
        for (int j = 0; j < nsub; ++j) {
          N.Lw[r * kMaxSub + j] = C.Lw[i * kMaxSub + j];
          N.hist[r * kMaxSub + j] = C.hist[i * kMaxSub + j];
        }
      } else {
        // in place: the sub-beams go through the free part of the shared
        // scratch (registers would spill)
        for (int j = 0; j < nsub; ++j) {
          sStL[r * kMaxSub + j] = C.Lw[i * kMaxSub + j];
          sStH[r * kMaxSub + j] = C.hist[i * kMaxSub + j];
        }
      }
    }
    if constexpr (!DB) lds_barrier();  // every source entry has been read
    if (r < nsel) {
      insert_key(w_key, r);  // for the next frame's parent lookups
      N.key[r] = w_key;
      N.pkey[r] = w_pkey;
      N.ab[r] = w_ab;
      N.anb[r] = w_anb;
      N.pt[r] = w_pt;
      N.node[r] = w_node;
      N.meta[r] = w_meta;
      if (!tn_load) {
        N.tmask[r] = w_tmask;
        sMask[r] = w_tmask;
        N.first[r] = w_first;
        N.woff[r] = w_woff;
      }
      if constexpr (!DB) {
        const int nsub = (w_meta >> 8) & 0xFF;
        for (int j = 0; j < nsub; ++j) {
          N.Lw[r * kMaxSub + j] = sStL[r * kMaxSub + j];
          N.hist[r * kMaxSub + j] = sStH[r * kMaxSub + j];
        }
      }
    }
    int nev = 0;
    const int erank = block_scan<BLOCK, false>(is_event, sScanC, &nev);
    if (is_event) {
      sEvBeam[erank] = static_cast<uint32_t>(r);
      sEvWoff[erank] = ev_woff;
      sEvH[erank] = ev_H;
    }
    mark(kPhNewBeam);

    // ---- Eq. (1).  The queries (sub-beam j, homophone h) of the completed
    // words are scored once per distinct group (n-gram context, completed-word
    // node): the pairs (word e, sub-beam j) are grouped in an LDS hash table,
    // the groups' lookups spread over all threads into the stream's scratch,
    // and each completed word ranks its queries from there.  Words are taken
    // in batches of NEB (the grouping tables hold NPL pairs).
    unsigned long long* const sGKey = reinterpret_cast<unsigned long long*>(sSel);
    int32_t* const sGId = reinterpret_cast<int32_t*>(sSel + 8 * NPL);
    int32_t* const sPairG = sGId + NPL;  // pair -> hash slot, then -> group
    uint32_t* const sGwoff = reinterpret_cast<uint32_t*>(sPairG + NPL);
    uint32_t* const sGH = sGwoff + NPL;
    Ctx* const sGctx = reinterpret_cast<Ctx*>(sGH + NPL);             // 24 B each
    int32_t* const sGoff = reinterpret_cast<int32_t*>(sGctx + NPL);  // NPL + 1 entries
    uint32_t* const sGcnt = reinterpret_cast<uint32_t*>(sGoff + NPL + 1);  // lookups | kGroupHeavy
    // heavy groups: bit (h mod 64) set for each homophone h of the explicit
    // list; past sGcnt (which ends 56 NPL + 4 bytes in), 8-B aligned
    constexpr int kGmaskOff = (56 * NPL + 4 + 7) & ~7;
    uint64_t* const sGmask = reinterpret_cast<uint64_t*>(sSel + kGmaskOff);
    static_assert(kGmaskOff + 8 * NPL <= UNI_BYTES, "grouping tables fit the shared scratch");
    static_assert(sizeof(Ctx) == 24, "group contexts are 24 B each");
#pragma unroll 1
    for (int e0 = 0; e0 < nev; e0 += NEB) {
    const int nb = nev - e0 < NEB ? nev - e0 : NEB;
    if (e0 > 0) {
      // the next batch: the previous one's scratch reads are done; fresh grouping table
      __syncthreads();
      for (int q = tid; q < NPL; q += BLOCK) sGKey[q] = kEmptyKey;
      if (tid == 0) {
        sNG = 0;
        sHeavy = 0;
        sNLarge = 0;
      }
    }
    lds_barrier();
    for (int pr = tid; pr < nb * kMaxSub; pr += BLOCK) {
      const int el = pr / kMaxSub;
      const int e = e0 + el;
      const int j = pr - el * kMaxSub;
      const uint32_t rr = sEvBeam[e];
      int slot = -1;
      if (j < static_cast<int>((N.meta[rr] >> 8) & 0xFF)) {
        const uint32_t ph = N.hist[rr * kMaxSub + j];
        const Ctx ctx = ctx_of(S.arena[ph]);
        const unsigned long long key = group_key(ctx, sEvWoff[e]);
        uint32_t q = static_cast<uint32_t>(splitmix64(key)) & (NPL - 1);
        for (;;) {
          const unsigned long long prev = atomicCAS(&sGKey[q], kEmptyKey, key);
          if (prev == kEmptyKey) {
            const int g = atomicAdd(&sNG, 1);
            sGId[q] = g;
            sGwoff[g] = sEvWoff[e];
            sGH[g] = sEvH[e];
            sGctx[g] = ctx;
            if (sEvH[e] >= P.heavy_min) sHeavy = 1;
            break;
          }
          if (prev == key) break;
          q = (q + 1) & (NPL - 1);
        }
        slot = static_cast<int>(q);
      }
      sPairG[pr] = slot;
    }
    lds_barrier();
    const int NG = sNG;
    for (int pr = tid; pr < nb * kMaxSub; pr += BLOCK) {
      const int q = sPairG[pr];
      if (q >= 0) sPairG[pr] = sGId[q];
    }
    // heavy groups (nodes with many homophones): the homophones with an explicit
    // n-gram for the group's context, from the continuation index (each once: a
    // homophone can be listed for several context orders); the others back off
    // to their unigrams and are not looked up.  A group with more than
    // kMaxExplicit listed is looked up in full.
    const bool heavy_frame = sHeavy != 0;
    for (int g = tid; g < NG; g += BLOCK) {
      const uint32_t Hg = sGH[g];
      uint32_t cnt = Hg;
      if (Hg >= P.heavy_min) {
        PresHit hit[3];
        pres_lookup(S, sGctx[g], sGwoff[g], hit, &plines);
        const uint32_t ne = hit[0].n + hit[1].n + hit[2].n;
        if (ne <= static_cast<uint32_t>(kMaxExplicit)) {
          uint32_t* const E = scrE + static_cast<size_t>(g) * kMaxExplicit;
          uint64_t bm = 0;
          uint32_t nd = 0;
          // (the list is read back only when the mask bit is already set)
          auto add = [&](uint32_t x) {
            const uint64_t bit = 1ull << (x & 63u);
            bool seen = false;
            if (bm & bit)
              for (uint32_t m = 0; m < nd; ++m) seen |= E[m] == x;
            if (!seen) {
              E[nd++] = x;
              bm |= bit;
            }
          };
#pragma unroll
          for (int o3 = 0; o3 < 3; ++o3) {
            if (hit[o3].n == 1) {
              add(hit[o3].a);
            } else {
              const uint32_t* lst = (o3 == 0 ? S.p2.lists : (o3 == 1 ? S.p3.lists : S.p4.lists)) + hit[o3].a;
              for (uint32_t m = 0; m < hit[o3].n; ++m) add(lst[m]);
            }
          }
          cnt = nd | kGroupHeavy;
          sGmask[g] = bm;
        }
      }
      sGcnt[g] = cnt;
    }
    if (heavy_frame)
      __syncthreads();  // the explicit lists (global memory) are read by other threads
    else
      lds_barrier();
    // lookup offsets of the groups
    int U = 0;
    {
      constexpr int PG = (NPL + BLOCK - 1) / BLOCK;
      int loc = 0;
#pragma unroll
      for (int q = 0; q < PG; ++q) {
        const int g = tid * PG + q;
        loc += g < NG ? static_cast<int>(sGcnt[g] & ~kGroupHeavy) : 0;
      }
      int pre = block_scan<BLOCK, false>(loc, sScanD, &U);
#pragma unroll
      for (int q = 0; q < PG; ++q) {
        const int g = tid * PG + q;
        if (g < NG) {
          sGoff[g] = pre;
          pre += static_cast<int>(sGcnt[g] & ~kGroupHeavy);
        }
      }
      if (tid == 0) sGoff[NG] = U;
    }
    if (static_cast<uint64_t>(U) > S.scap) {  // cannot happen: U <= K * O * (largest homophone set)
      if (tid == 0) atomicOr(S.flags, kFlagSelect);
      U = 0;
    }
    if (tid == 0) sCnt[6] += static_cast<unsigned long long>(U);
    // the results go to LDS when they fit in the grouping keys freed above (the
    // usual case), else to the stream's scratch in global memory; the log-probs,
    // read for every candidate (the states only for the kept ones), stay in
    // LDS up to four times as many lookups, the states then in the scratch
    constexpr int kLdsRes = 12 * NPL / 32;
    constexpr int kLdsLp = 12 * NPL / 8;
    double* const sResL = reinterpret_cast<double*>(sSel);
    QState* const sResS = reinterpret_cast<QState*>(sSel + 8 * kLdsRes);  // (only when U <= kLdsRes)
    const bool res_lds = U <= kLdsRes;
    const bool lp_lds = U <= kLdsLp;
    auto res_lp = [&](int u) -> double { return lp_lds ? sResL[u] : scrL[u]; };
    auto res_st = [&](int u) -> QState { return res_lds ? sResS[u] : scrS[u]; };
    lds_barrier();
    mark(kPhGroup);
    for (int u = tid; u < U; u += BLOCK) {
      int lo = 0, hi = NG - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (sGoff[mid] <= u) lo = mid; else hi = mid - 1;
      }
      const uint32_t k = static_cast<uint32_t>(u - sGoff[lo]);
      const uint32_t h = (sGcnt[lo] & kGroupHeavy) ? scrE[static_cast<size_t>(lo) * kMaxExplicit + k] : k;
      const int32_t w = S.trie_words[sGwoff[lo] + h];
      const LmResult res = lm_lookup(S, w, sGctx[lo], &lines);
      if (lp_lds)
        sResL[u] = res.lp;
      else
        scrL[u] = res.lp;
      if (res_lds)
        sResS[u] = res.st;
      else
        scrS[u] = res.st;
    }
    if (res_lds)
      lds_barrier();
    else
      __syncthreads();  // the lookup results (global memory) are read by other threads
    mark(kPhLookup);
    // each completed word: its top-o by (score desc, j*H + h asc), lambda
    // pruning, word-history nodes (o reserved per word, in order).  A
    // candidate's source: its lookup result in the scratch (>= 0), or, for a
    // homophone that backs off to its unigram in a heavy group, -1 - its rank
    // in the node's unigram order.  A word is ranked by one thread, unless one
    // of its sub-beams' groups was looked up in full over more than
    // kThreadMaxH homophones: those words get a wavefront each.
    // (ph: the winner's parent history, read before any of the word's
    // sub-beams is overwritten)
    auto write_node = [&](int e, int k, double L, uint32_t ph, int src) {
      const uint32_t rr = sEvBeam[e];
      QState st;
      if (src >= 0) {
        st = res_st(src);
      } else {
        const WordRank wr = S.wrank[sEvWoff[e] + static_cast<uint32_t>(-1 - src)];
        st.c2 = kNone;
        st.c3 = kNone;
        st.bo2 = 0.0f;
        st.bo3 = 0.0f;
        st.w = wr.w;
        st.bo1 = wr.bo;
      }
      const HistNode par = S.arena[ph];
      HistNode hn;
      hn.word = st.w;
      hn.c2 = st.c2;
      hn.c3 = st.c3;
      hn.bo1 = st.bo1;
      hn.bo2 = st.bo2;
      hn.bo3 = st.bo3;
      hn.depth = par.depth + 1;
      hn.sfus = synth ? par.sfus + bigram_score(P, par.word, st.w) : 0.0;
      // a parent that ends a block (the root included) starts a new one
      const bool starts = par.depth % kHistBlock == 0;
      hn.blk = starts ? ph : par.blk;
      hn.w[0] = starts ? -1 : par.word;
#pragma unroll
      for (int i = 1; i < kHistBlock - 1; ++i) hn.w[i] = starts ? -1 : par.w[i - 1];
      const uint32_t node = arena0 + arena_n + static_cast<uint32_t>(e * O + k);
      S.arena[node] = hn;
      N.Lw[rr * kMaxSub + k] = L;
      N.hist[rr * kMaxSub + k] = node;
    };
    auto close_event = [&](int e, int kept, int nsub) {
      const uint32_t rr = sEvBeam[e];
      const bool room = static_cast<uint64_t>(arena_n) + static_cast<uint64_t>(e + 1) * O <= S.arena_cap;
      if (room)
        N.meta[rr] = (N.meta[rr] & 0xFFu) | (static_cast<uint32_t>(kept) << 8);
      else
        atomicOr(S.flags, kFlagArena);
      c_words += 1;
      c_queries += static_cast<uint64_t>(nsub * sEvH[e]);
    };
    {
      constexpr uint32_t kThreadMaxH = 16;
      bool mine = false;
      if (tid < nb) {
        const int nsub = (N.meta[sEvBeam[e0 + tid]] >> 8) & 0xFF;
        bool large = false;
        for (int j = 0; j < nsub; ++j) {
          const int g = sPairG[tid * kMaxSub + j];
          large |= !(sGcnt[g] & kGroupHeavy) && sGH[g] > kThreadMaxH;
        }
        if (large)
          sLarge[atomicAdd(&sNLarge, 1)] = e0 + tid;
        else
          mine = true;
      }
      if (mine) {
        const int e = e0 + tid;
        const uint32_t rr = sEvBeam[e];
        const int H = static_cast<int>(sEvH[e]);
        const uint32_t woff = sEvWoff[e];
        const int nsub = (N.meta[rr] >> 8) & 0xFF;
        double tL[kMaxSub];
        int tq[kMaxSub], ts[kMaxSub];
#pragma unroll
        for (int k = 0; k < kMaxSub; ++k) {
          tL[k] = kNegInf;
          tq[k] = 0x7FFFFFFF;
          ts[k] = 0;
        }
        auto insert = [&](double L, int qq, int ss) {
#pragma unroll
          for (int k = 0; k < kMaxSub; ++k) {
            if (k < O && (L > tL[k] || (L == tL[k] && qq < tq[k]))) {
              const double t = tL[k];
              const int u = tq[k], v = ts[k];
              tL[k] = L;
              tq[k] = qq;
              ts[k] = ss;
              L = t;
              qq = u;
              ss = v;
            }
          }
        };
        bool any_heavy = false;
#pragma unroll
        for (int j = 0; j < kMaxSub; ++j) {
          if (j < nsub) {
            const double Lw = N.Lw[rr * kMaxSub + j];
            const int g = sPairG[(e - e0) * kMaxSub + j];
            const int off = sGoff[g];
            const uint32_t cnt = sGcnt[g];
            if (!(cnt & kGroupHeavy)) {
              for (int h = 0; h < H; ++h) insert(Lw + P.comega * res_lp(off + h), j * H + h, off + h);
            } else {
              any_heavy = true;
              const uint32_t* E = scrE + static_cast<size_t>(g) * kMaxExplicit;
              const int ne = static_cast<int>(cnt & ~kGroupHeavy);
              for (int m = 0; m < ne; ++m)
                insert(Lw + P.comega * res_lp(off + m), j * H + static_cast<int>(E[m]), off + m);
            }
          }
        }
        if (any_heavy) {
          // the heavy groups' other homophones in unigram order (scores
          // non-increasing): a sub-beam is done once its o-th such candidate
          // scores strictly above the next word's
          int nw[kMaxSub];
          double Lth[kMaxSub];
#pragma unroll
          for (int j = 0; j < kMaxSub; ++j) {
            nw[j] = 0;
            Lth[j] = HUGE_VAL;
          }
#pragma unroll 1
          for (int k = 0; k < H; ++k) {
            const WordRank wr = S.wrank[woff + k];
            bool need = false;
#pragma unroll
            for (int j = 0; j < kMaxSub; ++j) {
              if (j < nsub) {
                const int g = sPairG[(e - e0) * kMaxSub + j];
                const uint32_t cnt = sGcnt[g];
                if (cnt & kGroupHeavy) {
                  const Ctx cx = sGctx[g];
                  const double lp = static_cast<double>(cx.bo3) +
                                    (static_cast<double>(cx.bo2) +
                                     (static_cast<double>(cx.bo1) + static_cast<double>(wr.logp)));
                  const double L = N.Lw[rr * kMaxSub + j] + P.comega * lp;
                  if (nw[j] < O || !(Lth[j] > L)) {
                    need = true;
                    bool member = false;
                    if ((sGmask[g] >> (wr.h & 63u)) & 1ull) {
                      const uint32_t* E = scrE + static_cast<size_t>(g) * kMaxExplicit;
                      const int ne = static_cast<int>(cnt & ~kGroupHeavy);
                      for (int m = 0; m < ne; ++m) member |= E[m] == wr.h;
                    }
                    if (!member) {
                      insert(L, j * H + static_cast<int>(wr.h), -1 - k);
                      nw[j] += 1;
                      if (nw[j] == O) Lth[j] = L;
                    }
                  }
                }
              }
            }
            if (!need) break;
          }
        }
        int kept = 0;
#pragma unroll
        for (int k = 0; k < kMaxSub; ++k)
          if (k < O && tL[k] != kNegInf && !(tL[k] < tL[0] - P.lam)) kept = k + 1;
        const bool room = static_cast<uint64_t>(arena_n) + static_cast<uint64_t>(e + 1) * O <= S.arena_cap;
        uint32_t ph[kMaxSub];
#pragma unroll
        for (int k = 0; k < kMaxSub; ++k) ph[k] = k < kept ? N.hist[rr * kMaxSub + tq[k] / H] : 0u;
#pragma unroll
        for (int k = 0; k < kMaxSub; ++k)
          if (k < kept && room) write_node(e, k, tL[k], ph[k], ts[k]);
        close_event(e, kept, nsub);
      }
    }
    lds_barrier();  // the list of wavefront-ranked words
    const int nlarge = sNLarge;
    for (int x = wave; x < nlarge; x += NW) {
      const int e = sLarge[x];
      const uint32_t rr = sEvBeam[e];
      const uint32_t H = sEvH[e];
      const uint32_t woff = sEvWoff[e];
      const int nsub = (N.meta[rr] >> 8) & 0xFF;
      double tL[kMaxSub];
      int tq[kMaxSub], ts[kMaxSub];
#pragma unroll
      for (int k = 0; k < kMaxSub; ++k) {
        tL[k] = kNegInf;
        tq[k] = 0x7FFFFFFF;
        ts[k] = 0;
      }
      auto insert = [&](double L, int qq, int ss) {
#pragma unroll
        for (int k = 0; k < kMaxSub; ++k) {
          if (k < O && (L > tL[k] || (L == tL[k] && qq < tq[k]))) {
            const double t = tL[k];
            const int u = tq[k], v = ts[k];
            tL[k] = L;
            tq[k] = qq;
            ts[k] = ss;
            L = t;
            qq = u;
            ss = v;
          }
        }
      };
      // the sub-beams' scores, groups and result offsets (a group's results
      // are contiguous in the scratch)
      double Lw[kMaxSub];
      int gid[kMaxSub], goff[kMaxSub];
      uint32_t gcnt[kMaxSub];
      bool any_full = false, any_heavy = false;
#pragma unroll
      for (int j = 0; j < kMaxSub; ++j) {
        const int jj = j < nsub ? j : 0;
        Lw[j] = N.Lw[rr * kMaxSub + jj];
        gid[j] = sPairG[(e - e0) * kMaxSub + jj];
        goff[j] = sGoff[gid[j]];
        gcnt[j] = sGcnt[gid[j]];
        if (j < nsub) {
          any_heavy |= (gcnt[j] & kGroupHeavy) != 0;
          any_full |= (gcnt[j] & kGroupHeavy) == 0;
        }
      }
      // full groups: lane h reads homophone h of every such sub-beam
      if (any_full) {
        for (int h = lane; h < static_cast<int>(H); h += 64) {
          double a[kMaxSub];
#pragma unroll
          for (int j = 0; j < kMaxSub; ++j)
            a[j] = (j < nsub && !(gcnt[j] & kGroupHeavy)) ? res_lp(goff[j] + h) : 0.0;
#pragma unroll
          for (int j = 0; j < kMaxSub; ++j)
            if (j < nsub && !(gcnt[j] & kGroupHeavy))
              insert(Lw[j] + P.comega * a[j], j * static_cast<int>(H) + h, goff[j] + h);
        }
      }
      if (any_heavy) {
        // heavy groups: lane m holds the m-th explicit homophone (the list has
        // no repeats), a candidate with its looked-up score
        uint32_t eh[kMaxSub];
        int ne[kMaxSub];
#pragma unroll
        for (int j = 0; j < kMaxSub; ++j) {
          const bool hv = j < nsub && (gcnt[j] & kGroupHeavy);
          ne[j] = hv ? static_cast<int>(gcnt[j] & ~kGroupHeavy) : 0;
          eh[j] = lane < ne[j] ? scrE[static_cast<size_t>(gid[j]) * kMaxExplicit + lane] : kNone;
        }
#pragma unroll
        for (int j = 0; j < kMaxSub; ++j) {
          if (ne[j] > 0) {
            if (lane < ne[j])
              insert(Lw[j] + P.comega * res_lp(goff[j] + lane), j * static_cast<int>(H) + static_cast<int>(eh[j]),
                     goff[j] + lane);
          }
        }
        // the other homophones of a heavy group score bo3 + bo2 + bo1 + log10 p1(w)
        // (Katz backoff to the unigram), monotone in log10 p1: walk the node's
        // words in unigram order, 64 at a time, until every heavy sub-beam has
        // o candidates strictly above all that remain
        int cum[kMaxSub];
        Ctx cx[kMaxSub];
#pragma unroll
        for (int j = 0; j < kMaxSub; ++j) {
          cum[j] = 0;
          cx[j] = sGctx[gid[j]];
        }
#pragma unroll 1
        for (int c0 = 0; c0 < static_cast<int>(H); c0 += 64) {
          const int k = c0 + lane;
          const bool valid = k < static_cast<int>(H);
          WordRank wr = WordRank{0, 0.0f, 0.0f, kNone};
          if (valid) wr = S.wrank[woff + k];
          const int last = (static_cast<int>(H) - 1 - c0) < 63 ? static_cast<int>(H) - 1 - c0 : 63;
          bool more = false;
#pragma unroll
          for (int j = 0; j < kMaxSub; ++j) {
            if (j < nsub && (gcnt[j] & kGroupHeavy)) {
              bool member = false;
              for (int m = 0; m < ne[j]; ++m)
                member |= static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(eh[j]), m)) == wr.h;
              const double lp = static_cast<double>(cx[j].bo3) +
                                (static_cast<double>(cx[j].bo2) +
                                 (static_cast<double>(cx[j].bo1) + static_cast<double>(wr.logp)));
              const double L = Lw[j] + P.comega * lp;
              const bool cand = valid && !member;
              if (cand) insert(L, j * static_cast<int>(H) + static_cast<int>(wr.h), -1 - k);
              const double lastL = readlane_f64(L, last);
              cum[j] += __popcll(__ballot(cand && L > lastL));
              more |= cum[j] < O;
            }
          }
          if (!more) break;
        }
      }
      // O rounds of wavefront arg-max; lane k keeps the k-th winner
      double myL = kNegInf, bestL = kNegInf;
      int myq = 0, mys = 0, kept = 0;
#pragma unroll 1
      for (int k = 0; k < O; ++k) {
        double bL = tL[0];
        int bq = tq[0];
        wave_argmax(&bL, &bq);
        if (bL == kNegInf) break;
        if (k == 0) bestL = bL;
        if (bL < bestL - P.lam) break;
        const bool holder = tL[0] == bL && tq[0] == bq;  // one lane: queries are distinct
        const int hl = __builtin_ctzll(__ballot(holder));
        const int bs = __builtin_amdgcn_readlane(ts[0], hl);
        if (lane == k) {
          myL = bL;
          myq = bq;
          mys = bs;
        }
        if (holder) {
#pragma unroll
          for (int m = 0; m + 1 < kMaxSub; ++m) {
            tL[m] = tL[m + 1];
            tq[m] = tq[m + 1];
            ts[m] = ts[m + 1];
          }
          tL[kMaxSub - 1] = kNegInf;
          tq[kMaxSub - 1] = 0x7FFFFFFF;
        }
        kept = k + 1;
      }
      const bool room = static_cast<uint64_t>(arena_n) + static_cast<uint64_t>(e + 1) * O <= S.arena_cap;
      // every lane reads its parent before any lane writes (one wavefront, in order)
      const uint32_t ph = lane < kept ? N.hist[rr * kMaxSub + static_cast<uint32_t>(myq) / H] : 0u;
      if (lane < kept && room) write_node(e, lane, myL, ph, mys);
      if (lane == 0) close_event(e, kept, nsub);
    }
    mark(kPhRank);
    }
    {
      // nodes reserved this frame; past the capacity the count stays at cap + 1
      // (every later word event then sees no room and raises the flag)
      const uint64_t an = static_cast<uint64_t>(arena_n) + static_cast<uint64_t>(nev * O);
      arena_n = static_cast<uint32_t>(an <= S.arena_cap ? an : S.arena_cap + 1);
    }
    if (tid == 0) sCnt[4] += static_cast<unsigned long long>(n) * kClasses;
    n = nsel;
    __syncthreads();  // history nodes (global memory) are read by the fusion and the next frame
    mark(kPhRank);
    if (tn_load) {
      N.tmask[r] = tn.mask;
      sMask[r] = tn.mask;
      N.first[r] = tn.first_child;
      N.woff[r] = tn.word_off;
    }
    if (wave == 0 && tau + 1 < tend) set_row(P, dnext);  // this frame's row is no longer read

    // ---- Eq. (2) on fusion frames: the top-F hypotheses by (total desc, key
    // asc); each sub-beam's score becomes phi * its synthetic fusion score and
    // the sub-beams are re-ranked (stable)
    const int64_t t = t0 + tau;
    if (fuse_frames && t > 0 && t % P.fusion_interval == 0) {
      double* sc = reinterpret_cast<double*>(sSel);
      uint64_t* ky = reinterpret_cast<uint64_t*>(sSel + 8 * KMAX);
      uint32_t* ix = reinterpret_cast<uint32_t*>(sSel + 16 * KMAX);
      const int F = (P.fusion_top_f <= 0 || P.fusion_top_f >= n) ? n : P.fusion_top_f;
      const uint32_t* sel = ix;  // the selected hypotheses (any order: each is fused on its own)
      if (F < n) {
        if constexpr (KMAX >= 128) {
          // the top F as a set, from a histogram of the totals (a sort of K =
          // 256 totals takes 36 barrier-separated stages): bins of (hi -
          // total) over [lo, hi], monotone; the bin holding the F-th found by
          // one wavefront; the bins above it taken whole, and its members
          // ranked exactly among themselves by (total desc, key asc; the
          // index for exact ties, which distinct prefixes do not have)
          uint32_t* const fH = reinterpret_cast<uint32_t*>(sSel);
          double* const fT = reinterpret_cast<double*>(sSel + 4 * kBins);
          uint64_t* const fK = reinterpret_cast<uint64_t*>(sSel + 4 * kBins + 8 * KMAX);
          uint32_t* const fI = reinterpret_cast<uint32_t*>(sSel + 4 * kBins + 16 * KMAX);
          uint32_t* const fSel = fI + KMAX;
          static_assert(4 * kBins + 24 * KMAX <= UNI_BYTES, "top-F scratch");
          for (int d = tid; d < kBins; d += BLOCK) fH[d] = 0;
          if (tid == 0) {
            sBCount = 0;
            sAthr = 0;
          }
          const bool own = tid < n;
          double tot = kNegInf;
          uint64_t key = ~0ull;
          if (own) {
            tot = N.pt[tid] + N.Lw[tid * kMaxSub];
            key = N.key[tid];
          }
          double hi, lo;
          block_minmax<BLOCK>(own ? tot : kNegInf, own ? tot : HUGE_VAL, sRed, &hi, &lo);
          const double inv = hi > lo ? static_cast<double>(kBins) / (hi - lo) : 0.0;
          int bin = -1;
          if (own) {
            const double x = (hi - tot) * inv;
            bin = x < static_cast<double>(kBins - 1) ? static_cast<int>(x) : kBins - 1;  // NaN: a total of -inf
            atomicAdd(&fH[bin], 1u);
          }
          lds_barrier();
          if (wave == 0) {
            constexpr int PERW = kBins / 64;
            int h[PERW];
            const uint4* hp = reinterpret_cast<const uint4*>(fH + lane * PERW);
#pragma unroll
            for (int q = 0; q < PERW / 4; ++q) {
              const uint4 x4 = hp[q];
              h[4 * q] = static_cast<int>(x4.x);
              h[4 * q + 1] = static_cast<int>(x4.y);
              h[4 * q + 2] = static_cast<int>(x4.z);
              h[4 * q + 3] = static_cast<int>(x4.w);
            }
            int local = 0;
#pragma unroll
            for (int q = 0; q < PERW; ++q) local += h[q];
            const int incl = wave_scan_incl(local);
            const int before = incl - local;
            if (before < F && incl >= F) {
              int acc = before;
              bool found = false;
#pragma unroll
              for (int q = 0; q < PERW; ++q) {
                if (!found && acc + h[q] >= F) {
                  sBucket = lane * PERW + q;
                  sAbove = acc;
                  found = true;
                }
                acc += h[q];
              }
            }
          }
          lds_barrier();
          const int fb = sBucket, fa = sAbove;
          if (own && bin < fb) fSel[atomicAdd(&sAthr, 1)] = static_cast<uint32_t>(tid);  // positions 0..fa-1
          if (own && bin == fb) {
            const int m = atomicAdd(&sBCount, 1);
            fT[m] = tot;
            fK[m] = key;
            fI[m] = static_cast<uint32_t>(tid);
          }
          lds_barrier();
          const int nbm = sBCount;
          for (int m = tid; m < nbm; m += BLOCK) {
            const double tm = fT[m];
            const uint64_t km = fK[m];
            const uint32_t im = fI[m];
            int r = 0;
            for (int u = 0; u < nbm; ++u) {
              const double tu = fT[u];
              const uint64_t ku = fK[u];
              r += (tu > tm || (tu == tm && (ku < km || (ku == km && fI[u] < im)))) ? 1 : 0;
            }
            if (r < F - fa) fSel[fa + r] = im;
          }
          lds_barrier();
          sel = fSel;
        } else if constexpr (WPE == 1) {
          // the top F as a set by rank counting: the LPB lanes of each
          // hypothesis count, a share each, the hypotheses ranking before it
          // (total desc, key asc; the keys are distinct), and one lane places
          // it; one barrier (in the instances with registers to spare: in the
          // 128-register ones it costs a spill)
          const int hf = tid / LPB, lf = tid - hf * LPB;
          int cnt = 0;
          if (hf < n) {
            const double ti = N.pt[hf] + N.Lw[hf * kMaxSub];
            const uint64_t ki = N.key[hf];
            for (int j = lf; j < n; j += LPB) cnt += ranks_before(N.pt[j] + N.Lw[j * kMaxSub], N.key[j], ti, ki) ? 1 : 0;
          }
#pragma unroll
          for (int o = 1; o < LPB; o <<= 1) cnt += __shfl_xor(cnt, o, 64);
          if (hf < n && lf == 0 && cnt < F) ix[cnt] = static_cast<uint32_t>(hf);
          lds_barrier();
        } else {
          if (tid < KMAX) {
            sc[tid] = tid < n ? N.pt[tid] + N.Lw[tid * kMaxSub] : kNegInf;
            ky[tid] = tid < n ? N.key[tid] : ~0ull;
            ix[tid] = tid < n ? static_cast<uint32_t>(tid) : 0u;
          }
          lds_barrier();
          bitonic_sort<KMAX>(sc, ky, ix);
        }
      }
      if (tid < F) {
        const int i = F < n ? static_cast<int>(sel[tid]) : tid;
        const int nsub = (N.meta[i] >> 8) & 0xFF;
        double L[kMaxSub];
        uint32_t h[kMaxSub];
#pragma unroll
        for (int j = 0; j < kMaxSub; ++j) {
          if (j < nsub) {
            h[j] = N.hist[i * kMaxSub + j];
            L[j] = P.phi * S.arena[h[j]].sfus;
          } else {
            L[j] = kNegInf;
            h[j] = 0;
          }
        }
        // stable bubble sort, descending
#pragma unroll
        for (int pass = 0; pass < kMaxSub - 1; ++pass) {
#pragma unroll
          for (int j = 0; j + 1 < kMaxSub; ++j) {
            if (j + 1 < nsub && L[j] < L[j + 1]) {
              const double tL = L[j];
              L[j] = L[j + 1];
              L[j + 1] = tL;
              const uint32_t th = h[j];
              h[j] = h[j + 1];
              h[j + 1] = th;
            }
          }
        }
#pragma unroll
        for (int j = 0; j < kMaxSub; ++j) {
          if (j < nsub) {
            N.Lw[i * kMaxSub + j] = L[j];
            N.hist[i * kMaxSub + j] = h[j];
          }
        }
      }
      if (tid == 0) sCnt[5] += static_cast<unsigned long long>(F);
    }
    lds_barrier();
    mark(kPhFusion);
    if constexpr (DB) cur ^= 1;
  }

  // ---- the beam back to HBM
  {
    const BeamLds<KMAX>& E = sBeam[DB ? cur : 0];
    if (tid < n) {
      const size_t g = gb + tid;
      S.key[g] = E.key[tid];
      S.pkey[g] = E.pkey[tid];
      S.ab[g] = E.ab[tid];
      S.anb[g] = E.anb[tid];
      S.pt[g] = E.pt[tid];
      S.node[g] = E.node[tid];
      const uint32_t meta = E.meta[tid];
      S.meta[g] = meta;
      const int nsub = (meta >> 8) & 0xFF;
      for (int j = 0; j < nsub; ++j) {
        S.Lw[g * O + j] = E.Lw[tid * kMaxSub + j];
        S.hist[g * O + j] = E.hist[tid * kMaxSub + j];
      }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    lines += __shfl_xor(lines, o, 64);
    plines += __shfl_xor(plines, o, 64);
    c_words += __shfl_xor(c_words, o, 64);
    c_queries += __shfl_xor(c_queries, o, 64);
  }
  if (lane == 0) {
    atomicAdd(&sCnt[0], static_cast<unsigned long long>(lines));
    atomicAdd(&sCnt[1], static_cast<unsigned long long>(c_words));
    atomicAdd(&sCnt[2], static_cast<unsigned long long>(c_queries));
    atomicAdd(&sCnt[3], static_cast<unsigned long long>(plines));
  }
  __syncthreads();
  if (tid == 0) {
    S.nbeam[b] = n;
    S.arena_n[b] = arena_n;
    unsigned long long* cn = S.counters + static_cast<size_t>(b) * kNumCounters;
    cn[kCntExpansions] += sCnt[4];
    cn[kCntFrames] += static_cast<unsigned long long>(tend - tau0);
    cn[kCntWordEvents] += sCnt[1];
    cn[kCntLmQueries] += sCnt[2];
    cn[kCntFused] += sCnt[5];
    cn[kCntProbeLines] += sCnt[0] + sCnt[3];
    cn[kCntPresLines] += sCnt[3];
    cn[kCntLookups] += sCnt[6];
  }
  if (out_hyps) {
    __syncthreads();  // the beam is back in global memory
    output(P, S);
  }
  if (timing) {
    __syncthreads();
    mark(kPhOther);
    if (tid == 0) {
      unsigned long long* cn = S.counters + static_cast<size_t>(b) * kNumCounters;
      for (int k = 0; k < kPhases; ++k) cn[kCntPhase0 + k] += sPhase[k];
    }
  }
}

// ------------------------------------------------------------------ delayed fusion

// Selects the top-F hypotheses of stream b by (total desc, key asc) into
// S.fsel[b][0..F) and S.fsel_n[b] (F = all hypotheses when top_f <= 0); the
// sort covers BLOCK >= K entries (the workgroup may be larger).
#undef P
#undef S

template <int BLOCK>
__device__ __forceinline__ void select_fused(const DevParams& P, const DevState& S, int b, int top_f, double* sc, uint64_t* ky,
                             uint32_t* ix) {
  const int tid = threadIdx.x;
  const int n = S.nbeam[b];
  const size_t gb = static_cast<size_t>(b) * P.K;
  const int F = (top_f <= 0 || top_f >= n) ? n : top_f;
  if (F < n) {
    if (tid < n) {
      sc[tid] = S.pt[gb + tid] + S.Lw[(gb + tid) * P.O];
      ky[tid] = S.key[gb + tid];
      ix[tid] = tid;
    } else if (tid < BLOCK) {
      sc[tid] = kNegInf;
      ky[tid] = ~0ull;
      ix[tid] = 0;
    }
    __syncthreads();
    bitonic_sort<BLOCK>(sc, ky, ix);
  }
  if (tid < F) S.fsel[gb + tid] = (F < n) ? static_cast<int32_t>(ix[tid]) : tid;
  if (tid == 0) S.fsel_n[b] = F;
  __syncthreads();
}

// Delayed fusion on the selected hypotheses of stream b (Eq. (2)): each
// sub-beam's word-level score becomes phi * its fusion score -- the synthetic
// score kept in its history node, or the caller's ext[b][rank][j] -- and the
// sub-beams are re-ranked (stable).
// The best end-of-sentence mark after `word` by the synthetic scorer (the
// first of equal scores), or -1 without marks.
__device__ inline int32_t best_eos(const DevParams& P, int32_t word, double* score) {
  int32_t best = -1;
  double bs = kNegInf;
  for (int k = 0; k < P.eos_count; ++k) {
    const double v = bigram_score(P, word, P.eos_ids[k]);
    if (v > bs) {
      bs = v;
      best = P.eos_ids[k];
    }
  }
  *score = bs;
  return best;
}

// With `eos` (the final synthetic fusion) each sub-beam's fusion score also
// takes its best end-of-sentence mark.
template <int BLOCK>
__device__ __forceinline__ void apply_fused(const DevParams& P, const DevState& S, int b, const float* ext, bool eos = false) {
  const int tid = threadIdx.x;
  const size_t gb = static_cast<size_t>(b) * P.K;
  const int F = S.fsel_n[b];
  if (tid < F) {
    const size_t bi = gb + S.fsel[gb + tid];
    const uint32_t meta = S.meta[bi];
    const int nsub = (meta >> 8) & 0xFF;
    double L[kMaxSub];
    uint32_t h[kMaxSub];
#pragma unroll
    for (int j = 0; j < kMaxSub; ++j) {
      if (j < nsub) {
        h[j] = S.hist[bi * P.O + j];
        double f;
        if (ext) {
          f = static_cast<double>(ext[(gb + tid) * P.O + j]);
        } else {
          const HistNode hn = S.arena[h[j]];
          f = hn.sfus;
          if (eos) {
            double e;
            (void)best_eos(P, hn.word, &e);
            f += e;
          }
        }
        L[j] = P.phi * f;
      } else {
        L[j] = kNegInf;
        h[j] = 0;
      }
    }
    // stable bubble sort, descending
#pragma unroll
    for (int pass = 0; pass < kMaxSub - 1; ++pass) {
#pragma unroll
      for (int j = 0; j + 1 < kMaxSub; ++j) {
        if (j + 1 < nsub && L[j] < L[j + 1]) {
          const double tL = L[j];
          L[j] = L[j + 1];
          L[j + 1] = tL;
          const uint32_t th = h[j];
          h[j] = h[j + 1];
          h[j + 1] = th;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kMaxSub; ++j) {
      if (j < nsub) {
        S.Lw[bi * P.O + j] = L[j];
        S.hist[bi * P.O + j] = h[j];
      }
    }
  }
  if (tid == 0) {
    unsigned long long* cn = S.counters + static_cast<size_t>(b) * kNumCounters;
    cn[kCntFused] += static_cast<unsigned long long>(F);
  }
  __syncthreads();
}

// External scorer, step 1: per stream, the hypotheses to fuse (flag 1: a
// fusion frame, top-F; flag 2: end of utterance, all; 0: none).
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fuse_select(const DevParams P, const DevState S,
                                                       const int32_t* __restrict__ flag) {
  const int b = blockIdx.x;
  __shared__ double sc[BLOCK];
  __shared__ uint64_t ky[BLOCK];
  __shared__ uint32_t ix[BLOCK];
  if (flag[b] == 0) {
    if (threadIdx.x == 0) S.fsel_n[b] = 0;
    return;
  }
  select_fused<BLOCK>(P, S, b, flag[b] == 1 ? P.fusion_top_f : 0, sc, ky, ix);
}

// External scorer, step 2: word sequences of every sub-beam of the selected
// hypotheses, words [B][K][O][W] (-1 padded) and n_words [B][K][O] (-1 where
// nothing is to be scored).
// Writes -1 past each row's words: rows [nrows][W] with len[r] words in row r;
// the whole block on consecutive addresses, 16 B per store when W allows.
typedef int v4i __attribute__((ext_vector_type(4)));
template <int BLOCK>
__device__ inline void pad_rows(int32_t* rows, int nrows, int W, const int32_t* len) {
  if ((W & 3) == 0 && (reinterpret_cast<uintptr_t>(rows) & 15) == 0 && W > 0) {
    // thread t writes the 16-B column t % per of rows t / per, t / per + rstep,
    // ... (per = min(W / 4, BLOCK) columns of a row per pass, rstep rows)
    const int W4 = W >> 2;
    const int per = W4 < BLOCK ? W4 : BLOCK;  // columns per pass of a row
    const int rstep = BLOCK / per;            // rows per pass
    const int tid = threadIdx.x;
    if (tid < rstep * per) {
      for (int r = tid / per; r < nrows; r += rstep) {
        int4* row = reinterpret_cast<int4*>(rows + static_cast<size_t>(r) * W);
        const int n = len[r];
        for (int c = tid % per; c < W4; c += per) {
          const int c0 = 4 * c;
          if (c0 >= n) {
            // streamed past the caches: the rows are read by the caller, not here
            const v4i m1 = {-1, -1, -1, -1};
            __builtin_nontemporal_store(m1, reinterpret_cast<v4i*>(row + c));
          } else if (c0 + 3 >= n) {
            int32_t* e = rows + static_cast<size_t>(r) * W + c0;
            for (int q = n - c0; q < 4; ++q) e[q] = -1;
          }
        }
      }
    }
  } else {
    for (int r = 0; r < nrows; ++r) {
      int32_t* row = rows + static_cast<size_t>(r) * W;
      for (int c = len[r] + static_cast<int>(threadIdx.x); c < W; c += BLOCK) row[c] = -1;
    }
  }
}

// Writes the `depth` words of history h into row[0..min(depth, W)), one node
// read per block of kHistBlock words (the node's word and the earlier words of
// its block, then the node that ends the previous block).
__device__ inline void trace_words(const DevState& S, uint32_t h, int depth, int32_t* row, int W) {
  int d = depth;
  while (d >= 1) {
    const HistNode x = S.arena[h];
    const int nb = (d - 1) % kHistBlock;  // earlier words of the block
    if (d - 1 < W) row[d - 1] = x.word;
#pragma unroll
    for (int i = 0; i < kHistBlock - 1; ++i)
      if (i < nb && d - 2 - i < W) row[d - 2 - i] = x.w[i];
    d -= nb + 1;
    h = x.blk;
  }
}

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fuse_export(const DevParams P, const DevState S,
                                                       int32_t* __restrict__ words, int32_t* __restrict__ n_words) {
  const int b = blockIdx.x;
  const size_t gb = static_cast<size_t>(b) * P.K;
  const int F = S.fsel_n[b];
  __shared__ int32_t sLen[BLOCK * kMaxSub];  // words written per request row (BLOCK >= K)
  for (int idx = threadIdx.x; idx < P.K * P.O; idx += BLOCK) {
    const int r = idx / P.O;
    const int j = idx - r * P.O;
    const size_t slot = (gb + r) * P.O + j;
    int32_t* row = words + slot * P.W;
    int len = -1;
    if (r < F) {
      const size_t bi = gb + S.fsel[gb + r];
      const int nsub = (S.meta[bi] >> 8) & 0xFF;
      if (j < nsub) {
        const uint32_t h = S.hist[bi * P.O + j];
        len = static_cast<int>(S.arena[h].depth);
        if (len > P.W) atomicOr(S.flags, kFlagWords);
        trace_words(S, h, len, row, P.W);
        if (len > P.W) len = P.W;
      }
    }
    sLen[idx] = len < 0 ? 0 : len;
    n_words[slot] = len;
  }
  __syncthreads();
  pad_rows<BLOCK>(words + gb * P.O * P.W, P.K * P.O, P.W, sLen);
}

// External scorer, step 3: apply the caller's scores [B][K][O] to the selection.
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fuse_apply(const DevParams P, const DevState S,
                                                      const float* __restrict__ scores) {
  apply_fused<BLOCK>(P, S, blockIdx.x, scores);
}

// ------------------------------------------------------------------ output

// One stream's output: at the end of an utterance the final synthetic fusion
// over all hypotheses and the mid-word filter (when some hypothesis ends at a
// word boundary); then the hypotheses ranked by
// (total desc, key asc), each one's words traced back from its best sub-beam,
// rows padded with -1.  Run by a whole workgroup of NT threads; the sort covers
// N >= K entries (N a power of two, N <= NT) in sc / ky / ix; sScan holds
// NT / 64 entries.
template <int NT, int N>
__device__ __forceinline__ void emit_output(const DevParams& P, const DevState& S, int b, const int32_t* lengths,
                                            int32_t Tc, int32_t fin, int32_t* out_hyps, float* out_scores, double* sc,
                                            uint64_t* ky, uint32_t* ix, int32_t* sScan) {
  const int tid = threadIdx.x;
  if (fin && P.fusion_source == 1 && P.fusion_interval > 0) {
    select_fused<N>(P, S, b, 0, sc, ky, ix);
    apply_fused<N>(P, S, b, nullptr, P.eos_count > 0);
  }
  const int n = S.nbeam[b];
  const size_t gb = static_cast<size_t>(b) * P.K;
  // at the end of an utterance, hypotheses inside a word are dropped when at
  // least one hypothesis ends at a word boundary; otherwise all are ranked
  int nroot = 0;
  bool root = false;
  if (fin) {
    root = tid < n && S.node[gb + tid] == kRootNode;
    (void)block_scan<NT>(root ? 1 : 0, sScan, &nroot);
  }
  bool ok = false;
  if (tid < n) {
    ok = !fin || root || nroot == 0;
    sc[tid] = ok ? S.pt[gb + tid] + S.Lw[(gb + tid) * P.O] : kNegInf;
    ky[tid] = ok ? S.key[gb + tid] : ~0ull;
    ix[tid] = tid;
  } else if (tid < N) {
    sc[tid] = kNegInf;
    ky[tid] = ~0ull;
    ix[tid] = 0;
  }
  int m = 0;
  (void)block_scan<NT>(ok ? 1 : 0, sScan, &m);
  if constexpr (N <= 64) {
    // up to 64 entries: each one's position is the number of entries before
    // it in (score desc, key asc, index asc), counted by one wavefront (two
    // barriers instead of the sort's stages)
    double si = kNegInf;
    uint64_t ki = ~0ull;
    int rk = 0;
    if (tid < N) {
      si = sc[tid];
      ki = ky[tid];
      for (int j = 0; j < N; ++j) {
        const double sj = sc[j];
        const uint64_t kj = ky[j];
        rk += (ranks_before(sj, kj, si, ki) || (sj == si && kj == ki && j < tid)) ? 1 : 0;
      }
    }
    __syncthreads();
    if (tid < N) {
      sc[rk] = si;
      ky[rk] = ki;
      ix[rk] = static_cast<uint32_t>(tid);
    }
  } else {
    bitonic_sort<N>(sc, ky, ix);
  }
  if (tid == 0) {
    // the stream's frame counter advances by the frames decoded in this call:
    // a length outside 0..Tc is clamped (the decode did the same) and flagged
    const int32_t len = lengths[b];
    const int32_t adv = len < 0 ? 0 : (len > Tc ? Tc : len);
    if (adv != len) atomicOr(S.flags, kFlagLength);
    S.t0[b] += adv;
  }
  int32_t* const sLen = reinterpret_cast<int32_t*>(ky);  // words written per rank (the keys are read)
  __syncthreads();
  for (int r = tid; r < P.K; r += NT) {
    int32_t* row = out_hyps + (static_cast<size_t>(b) * P.K + r) * P.W;
    int n = 0;
    if (r < m) {
      const size_t bi = gb + ix[r];
      out_scores[static_cast<size_t>(b) * P.K + r] = static_cast<float>(sc[r]);
      const uint32_t h = S.hist[bi * P.O];
      const HistNode top = S.arena[h];
      const int len = static_cast<int>(top.depth);
      // at the end of an utterance with end-of-sentence marks, the best mark follows the words
      int32_t mark = -1;
      if (fin && P.fusion_source == 1 && P.fusion_interval > 0 && P.eos_count > 0) {
        double e;
        mark = best_eos(P, top.word, &e);
      }
      n = len + (mark >= 0 ? 1 : 0);
      if (n > P.W) atomicOr(S.flags, kFlagWords);
      trace_words(S, h, len, row, P.W);
      if (mark >= 0 && len < P.W) row[len] = mark;
    } else {
      out_scores[static_cast<size_t>(b) * P.K + r] = kNegInf;
    }
    sLen[r] = n < P.W ? n : P.W;
  }
  __syncthreads();
  pad_rows<NT>(out_hyps + static_cast<size_t>(b) * P.K * P.W, P.K, P.W, sLen);
}

// The output as a launch of its own (when the call's last decode launch did
// not write it).
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_output(const DevParams P, const DevState S,
                                                  const int32_t* __restrict__ lengths, int32_t Tc, int32_t fin,
                                                  int32_t* __restrict__ out_hyps,
                                                  float* __restrict__ out_scores) {
  __shared__ double sc[BLOCK];
  __shared__ uint64_t ky[BLOCK];
  __shared__ uint32_t ix[BLOCK];
  __shared__ int32_t sScan[BLOCK / 64];
  emit_output<BLOCK, BLOCK>(P, S, blockIdx.x, lengths, Tc, fin, out_hyps, out_scores, sc, ky, ix, sScan);
}

// ------------------------------------------------------------------ gather ceiling

// Reads kGatherPerThread random 64-B lines of a table per thread (line index:
// the multiply-high of splitmix64(seed + i) and the line count, i the global
// gather number), all loads issued before any is used, and writes each thread's
// XOR of what it read so that no load is optimised away: the access pattern of
// the n-gram probes, one 64-B bucket line per probe, as independent threads.
constexpr int kGatherPerThread = 8;
__global__ __launch_bounds__(256) void k_gather_probe(const uint4* __restrict__ table, uint64_t lines, uint64_t n,
                                                      uint64_t seed, uint32_t* __restrict__ out) {
  const uint64_t t = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  uint4 v[kGatherPerThread][4];
#pragma unroll
  for (int g = 0; g < kGatherPerThread; ++g) {
    const uint64_t i = t * kGatherPerThread + g;
    const uint64_t line = i < n ? __umul64hi(splitmix64(seed + i), lines) : 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) v[g][q] = i < n ? table[line * 4 + q] : make_uint4(0, 0, 0, 0);
  }
  uint32_t x = 0;
#pragma unroll
  for (int g = 0; g < kGatherPerThread; ++g)
#pragma unroll
    for (int q = 0; q < 4; ++q) x ^= v[g][q].x ^ v[g][q].y ^ v[g][q].z ^ v[g][q].w;
  if (t * kGatherPerThread < n) out[t] = x;
}

}  // namespace

// ------------------------------------------------------------------ launchers

// Optional start/stop events for the next decode-kernel launch.  They go into
// the kernel's own dispatch (hipExtLaunchKernel), so their elapsed time is the
// kernel's execution without the gaps around it.
namespace {
thread_local hipEvent_t g_ev_start = nullptr;
thread_local hipEvent_t g_ev_stop = nullptr;
}  // namespace

void set_launch_events(hipEvent_t start, hipEvent_t stop) {
  g_ev_start = start;
  g_ev_stop = stop;
}

#define LB_LAUNCH(KERNEL, GRID, BLOCK, ST, ...)                                                  \
  do {                                                                                         \
    hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, 0, ST, g_ev_start, g_ev_stop, 0, __VA_ARGS__);  \
    g_ev_start = g_ev_stop = nullptr;                                                          \
  } while (0)

hipError_t launch_build_order(int order, const int32_t* ids, const float* lp, const float* bo, int64_t count,
                              int32_t vocab, NgramTable t2, NgramTable t3, NgramTable dst, uint32_t* flags,
                              uint32_t* ctx_out, hipStream_t st) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = (count + 255) / 256;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(k_build_order, dim3(grid), dim3(256), 0, st, order, ids, lp, bo, count, vocab, t2, t3,
                     dst, flags, ctx_out);
  return hipGetLastError();
}

uint64_t gather_probe_threads(uint64_t n) { return (n + kGatherPerThread - 1) / kGatherPerThread; }

hipError_t launch_gather_probe(const void* table, uint64_t lines, uint64_t n, uint64_t seed, uint32_t* out,
                               hipStream_t st) {
  const uint64_t threads = gather_probe_threads(n);
  const uint64_t blocks = (threads + 255) / 256;
  if (blocks == 0) return hipSuccess;
  if (blocks > 0x7FFFFFFFull) return hipErrorInvalidValue;
  LB_LAUNCH(k_gather_probe, dim3(static_cast<unsigned>(blocks)), dim3(256), st, static_cast<const uint4*>(table), lines,
            n, seed, out);
  return hipGetLastError();
}

hipError_t launch_begin(const DevParams& P, const DevState& S, int32_t B, hipStream_t st) {
  LB_LAUNCH(k_begin, dim3((B + 255) / 256), dim3(256), st, P, S, B);
  return hipGetLastError();
}

#define LB_DISPATCH_BLOCK(BLK, KERNEL, GRID, ...)                                           \
  do {                                                                                      \
    if ((BLK) == 64)                                                                        \
      LB_LAUNCH(KERNEL<64>, dim3(GRID), dim3(64), st, __VA_ARGS__);                         \
    else if ((BLK) == 128)                                                                  \
      LB_LAUNCH(KERNEL<128>, dim3(GRID), dim3(128), st, __VA_ARGS__);                       \
    else                                                                                    \
      LB_LAUNCH(KERNEL<256>, dim3(GRID), dim3(256), st, __VA_ARGS__);                       \
  } while (0)

// Decode-kernel shapes: (hypotheses per workgroup, lanes per hypothesis).
// Compute units of the current device (queried once).
int cu_count() {
  static int n = 0;
  if (n <= 0) {
    int dev = 0, c = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && c > 0)
      n = c;
    else
      n = 256;
  }
  return n;
}

hipError_t launch_decode(int K, const KArgs* args, const float* logits, const int32_t* lengths, int32_t B,
                         int32_t Tc, int32_t tau0, int32_t tau1, int32_t fin, int32_t* out_hyps, float* out_scores,
                         uint32_t opts, void* scratch, hipStream_t st) {
  unsigned char* const scr = static_cast<unsigned char*>(scratch);
  const KArgs LB_CONST* A = (const KArgs LB_CONST*)args;
  // One workgroup per stream.  A batch that leaves CUs to spare gets more
  // lanes per hypothesis (up to 512 threads per stream, LPB <= 16); a batch
  // with more streams than one round of workgroups holds gets the instances
  // that fit more workgroups per CU: K = 64 with 4 per CU instead of 3 (128
  // registers, some spilling; one in-place LDS beam buffer), K = 256 with 2 per
  // CU (one in-place LDS beam buffer; two lanes per hypothesis, 512 threads,
  // so 128 registers).
  const int cus = cu_count();
  const bool spare = B <= cus;
  // (hash slots per hypothesis: 16 with one workgroup per CU and K <= 64, 8 at
  // K = 256; where workgroups share a CU, 4 with two tables, 8 or 16 with one,
  // as their LDS allows)
#define LB_DECODE(KM, LP, WP, DBUF, HSLOTS, THREADS)                                                         \
  LB_LAUNCH((k_decode<KM, LP, WP, DBUF, HSLOTS>), dim3(B), dim3(THREADS), st, A, logits, lengths, Tc, tau0, tau1, \
            fin, out_hyps, out_scores, opts, scr)
  if (K <= 16 && spare)
    LB_DECODE(16, 16, 1, true, 16, 256);
  else if (K <= 16)
    LB_DECODE(16, 4, 1, true, 4, 64);
  else if (K <= 32 && spare)
    LB_DECODE(32, 16, 1, true, 16, 512);
  else if (K <= 32)
    LB_DECODE(32, 4, 1, true, 4, 128);
  else if (K <= 64 && spare)
    LB_DECODE(64, 8, 1, true, 16, 512);
  else if (K <= 64 && B > 3 * cus)
    LB_DECODE(64, 4, 4, false, 16, 256);
  else if (K <= 64)
    LB_DECODE(64, 4, 1, true, 4, 256);
  else if (K <= 128)
    LB_DECODE(128, 4, 1, true, 4, 512);
  else if (spare)
    LB_DECODE(256, 2, 1, true, 8, 512);
  else
    LB_DECODE(256, 2, 4, false, 8, 512);
#undef LB_DECODE
  return hipGetLastError();
}

hipError_t launch_fuse_select(int block, const DevParams& P, const DevState& S, const int32_t* flag, int32_t B,
                              hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_fuse_select, B, P, S, flag);
  return hipGetLastError();
}

hipError_t launch_fuse_export(int block, const DevParams& P, const DevState& S, int32_t* words, int32_t* n_words,
                              int32_t B, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_fuse_export, B, P, S, words, n_words);
  return hipGetLastError();
}

hipError_t launch_fuse_apply(int block, const DevParams& P, const DevState& S, const float* scores, int32_t B,
                             hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_fuse_apply, B, P, S, scores);
  return hipGetLastError();
}

hipError_t launch_output(int block, const DevParams& P, const DevState& S, const int32_t* lengths, int32_t B,
                         int32_t Tc, int32_t fin, int32_t* out_hyps, float* out_scores, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_output, B, P, S, lengths, Tc, fin, out_hyps, out_scores);
  return hipGetLastError();
}

// ------------------------------------------------------------------ static lookup scratch

// The n-gram lookup scratch of the decode calls that allocate nothing
// (lb_decode_batch_noalloc): one array per device, held until the process
// ends, shared by every such call on that device.  Host code never uses the
// name itself as an address (on the host it stands for the symbol, not for the
// device memory): static_scratch_address() returns the device address, found
// with hipGetSymbolAddress once per device, with that device current.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch_addr[kMaxDevices] = {};

hipError_t static_scratch_address(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

}  // namespace lb
