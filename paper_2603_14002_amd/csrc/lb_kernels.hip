// HIP kernels of the LightBeam gfx950 decoder (wave64, CDNA4).
//
// One frame of Alg. 1 is three launches on the caller's stream:
//   k_frame   one workgroup per stream: fan-out of every hypothesis by blank,
//             repeat and each lexicon-valid symbol (trie child mask), token /
//             word bonuses, recombination of equal prefixes by log-sum-exp,
//             theta pruning, top-K selection (MSD radix select on the ordered
//             score bits and the 64-bit prefix key), beam update and trie-state
//             advance; hypotheses that completed a word are queued.
//   k_ngram   one wavefront per queued hypothesis: every (sub-beam, homophone)
//             pair is scored with the 4-gram backoff LM by probing the HBM hash
//             tables, the top-o survive, lambda pruning, word-history append
//             (Eq. (1), App. E.3).
//   k_fusion  one workgroup per stream, only on fusion frames: top-F selection
//             and replacement of the sub-beam scores by phi * S_fus (Eq. (2)).
// k_output ranks the hypotheses of each stream and writes word ids / scores.
#include <hip/hip_runtime.h>

#include "lb_device.h"
#include "lb_launch.h"

namespace lb {

namespace {

constexpr double kNegInf = -HUGE_VAL;
constexpr int kBins = 1024;         // score bins of the top-K selection
constexpr int kBoundaryCap = 256;   // candidates resolved exactly inside the boundary bin
constexpr int kMaxLevels = 16;      // refinement levels of the top-K selection
#ifndef LB_CAND_UNROLL
#define LB_CAND_UNROLL 64
#endif
#ifndef LB_LPB_LARGE
#define LB_LPB_LARGE 4
#endif

// ------------------------------------------------------------------ block helpers

template <int BLOCK>
__device__ inline double block_max(double v, double* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = red[0];
#pragma unroll
  for (int k = 1; k < BLOCK / 64; ++k) r = fmax(r, red[k]);
  __syncthreads();
  return r;
}

// Block-wide maximum of `mx` and minimum of `mn` in one reduction.
template <int BLOCK>
__device__ inline void block_minmax(double mx, double mn, double* red, double* out_max, double* out_min) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mx = fmax(mx, __shfl_xor(mx, o, 64));
    mn = fmin(mn, __shfl_xor(mn, o, 64));
  }
  constexpr int NW = BLOCK / 64;
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = mx;
    red[NW + (threadIdx.x >> 6)] = mn;
  }
  __syncthreads();
  double a = red[0], c = red[NW];
#pragma unroll
  for (int k = 1; k < NW; ++k) {
    a = fmax(a, red[k]);
    c = fmin(c, red[NW + k]);
  }
  __syncthreads();
  *out_max = a;
  *out_min = c;
}

// Exclusive prefix sum over the block; *total receives the block sum.
template <int BLOCK>
__device__ inline int block_scan(int v, int* red, int* total) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) red[w] = x;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int k = 0; k < BLOCK / 64; ++k) {
    const int t = red[k];
    base += (k < w) ? t : 0;
    tot += t;
  }
  __syncthreads();
  *total = tot;
  return base + x - v;
}

// (score desc, key asc)
__device__ inline bool ranks_before(double sa, uint64_t ka, double sb, uint64_t kb) {
  return sa > sb || (sa == sb && ka < kb);
}

// In-place bitonic sort of BLOCK entries (one per thread) by (score desc, key asc).
template <int BLOCK>
__device__ inline void bitonic_sort(double* sc, uint64_t* ky, uint32_t* val) {
  const int i = threadIdx.x;
  for (int k = 2; k <= BLOCK; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int ixj = i ^ j;
      if (ixj > i) {
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
      __syncthreads();
    }
  }
}

// 8-bit digit of the 128-bit value (hi:lo) starting at bit `pos` (0..120).
__device__ inline uint32_t digit128(uint64_t hi, uint64_t lo, int pos) {
  if (pos >= 64) return static_cast<uint32_t>(hi >> (pos - 64)) & 0xFFu;
  if (pos > 56) return static_cast<uint32_t>((hi << (64 - pos)) | (lo >> pos)) & 0xFFu;
  return static_cast<uint32_t>(lo >> pos) & 0xFFu;
}

// Mask of the bits >= pos of a 128-bit value, split in (hi, lo).
__device__ inline void mask_from(int pos, uint64_t* mhi, uint64_t* mlo) {
  if (pos >= 128) {
    *mhi = 0;
    *mlo = 0;
  } else if (pos >= 64) {
    *mhi = ~0ull << (pos - 64);
    *mlo = 0;
  } else {
    *mhi = ~0ull;
    *mlo = pos == 0 ? ~0ull : (~0ull << pos);
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

__global__ void k_build_order(int order, const int32_t* __restrict__ ids, const float* __restrict__ lp,
                              const float* __restrict__ bo, int64_t count, int32_t vocab, NgramTable t2,
                              NgramTable t3, NgramTable dst, uint32_t* flags) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; e < count; e += stride) {
    const int32_t* r = ids + e * order;
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

// ------------------------------------------------------------------ frame step

// One workgroup per stream.  Hypothesis i is owned by LPB consecutive lanes:
// lane s of it handles the extensions v = 1+s, 1+s+LPB, ... (and lane 0 the
// merged stay), with the hypothesis' scores held in registers.
template <int KMAX, int LPB>
__global__ __launch_bounds__(KMAX * LPB) void k_frame(const DevParams P, const DevState S,
                                                      const float* __restrict__ logits,
                                                      const int32_t* __restrict__ lengths, int32_t Tc,
                                                      int32_t tau) {
  constexpr int BLOCK = KMAX * LPB;
  constexpr int HS = 2 * KMAX;  // LDS hash slots for the current prefix keys
  constexpr int NW = BLOCK / 64;
  constexpr int NC = (kSep + LPB - 1) / LPB;  // extension slots per lane
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  if (b == 0 && tid == 0) S.evq[(tau + 1) & 1] = 0;
  if (tau >= lengths[b]) return;

  __shared__ double sD[kClasses];
  __shared__ uint64_t sKey[KMAX], sPkey[KMAX];
  __shared__ double sAb[KMAX], sP[KMAX], sL[KMAX], sAb2[KMAX], sAnb2[KMAX], sPt2[KMAX], sStay[KMAX];
  __shared__ uint32_t sNode[KMAX], sMeta[KMAX], sFirst[KMAX], sWoff[KMAX], sNwords[KMAX];
  __shared__ uint64_t sMask[KMAX], sTrieMask[KMAX];
  __shared__ double sLw[KMAX * kMaxSub];
  __shared__ uint32_t sHist[KMAX * kMaxSub];
  __shared__ unsigned long long sHKey[HS];
  __shared__ int32_t sHIdx[HS];
  __shared__ uint32_t sHisto[kBins];
  __shared__ double sBScore[kBoundaryCap];
  __shared__ uint64_t sBKey[kBoundaryCap];
  __shared__ double sLvHi[kMaxLevels], sLvInv[kMaxLevels];
  __shared__ int32_t sLvBeta[kMaxLevels], sLvShift[kMaxLevels];
  __shared__ uint32_t sSelSrc[KMAX];
  __shared__ uint32_t sEvQ[KMAX];
  __shared__ double sRed[2 * NW];
  __shared__ int32_t sScan[NW];
  __shared__ int32_t sBucket, sAbove, sBucketCnt, sBCount;
  __shared__ unsigned long long sEvBase;

  const int n = S.nbeam[b];
  const size_t gb = static_cast<size_t>(b) * P.K;

  // ---- load the frame's scaled log-probs and the hypotheses
  for (int v = tid; v < kClasses; v += BLOCK)
    sD[v] = P.alpha * static_cast<double>(logits[(static_cast<size_t>(b) * Tc + tau) * kClasses + v]);
  for (int s = tid; s < HS; s += BLOCK) sHKey[s] = kEmptyKey;
  uint64_t my_key = 0, my_pkey = kNoParent;
  double my_anb = kNegInf;
  uint32_t my_meta = 0;
  if (tid < n) {
    my_key = S.key[gb + tid];
    my_pkey = S.pkey[gb + tid];
    const double ab = S.ab[gb + tid];
    my_anb = S.anb[gb + tid];
    const uint32_t node = S.node[gb + tid];
    my_meta = S.meta[gb + tid];
    const TrieNode tn = S.trie[node];
    sKey[tid] = my_key;
    sPkey[tid] = my_pkey;
    sAb[tid] = ab;
    sP[tid] = S.pt[gb + tid];  // log-sum-exp(ab, anb), kept with the hypothesis
    sNode[tid] = node;
    sMeta[tid] = my_meta;
    const int nsub = (my_meta >> 8) & 0xFF;
    for (int j = 0; j < nsub; ++j) {
      sLw[tid * kMaxSub + j] = S.Lw[(gb + tid) * P.O + j];
      sHist[tid * kMaxSub + j] = S.hist[(gb + tid) * P.O + j];
    }
    sL[tid] = sLw[tid * kMaxSub];
    sMask[tid] = tn.mask;
    sTrieMask[tid] = tn.mask;
    sFirst[tid] = tn.first_child;
    sWoff[tid] = tn.word_off;
    sNwords[tid] = static_cast<uint32_t>(tn.mask >> kWordCountShift);
  }
  __syncthreads();

  // ---- prefix keys into an LDS hash table
  if (tid < n) {
    uint32_t s = static_cast<uint32_t>(my_key) & (HS - 1);
    for (;;) {
      const unsigned long long prev = atomicCAS(&sHKey[s], kEmptyKey, my_key);
      if (prev == kEmptyKey) {
        sHIdx[s] = tid;
        break;
      }
      s = (s + 1) & (HS - 1);
    }
  }
  __syncthreads();

  // ---- recombination: a hypothesis whose parent prefix is also live receives
  // the parent's extension by its last symbol; that extension is removed from
  // the parent's fan-out.
  int par = -1;
  if (tid < n && my_pkey != kNoParent) {
    uint32_t s = static_cast<uint32_t>(my_pkey) & (HS - 1);
    for (int probes = 0; probes < HS; ++probes) {
      const unsigned long long k = sHKey[s];
      if (k == kEmptyKey) break;
      if (k == my_pkey) {
        par = sHIdx[s];
        break;
      }
      s = (s + 1) & (HS - 1);
    }
    if (par >= 0) atomicAnd(reinterpret_cast<unsigned long long*>(&sMask[par]), ~(1ull << (my_meta & 0xFF)));
  }
  __syncthreads();

  // ---- stay candidates (blank-stay, repeat-stay, merged parent extension)
  if (tid < n) {
    const int last = my_meta & 0xFF;
    const double ab2 = sP[tid] + sD[0];
    const double rep = last ? my_anb + sD[last] : kNegInf;
    double ext = kNegInf;
    if (par >= 0) {
      const double base = (last == static_cast<int>(sMeta[par] & 0xFF)) ? sAb[par] : sP[par];
      ext = (base + sD[last]) + (last == kSep ? P.gamma : P.beta);
    }
    const double anb2 = lse2(rep, ext);
    const double pt2 = lse2(ab2, anb2);
    sAb2[tid] = ab2;
    sAnb2[tid] = anb2;
    sPt2[tid] = pt2;
    sStay[tid] = pt2 + sL[tid];
  }
  __syncthreads();

  // ---- this lane's candidates: slot k is the extension by v = 1 + ln + LPB*k,
  // plus the merged stay on lane 0; scores are recomputed in every pass (same
  // operations, same result)
  const int hi_ = tid / LPB;
  const int ln = tid - hi_ * LPB;
  const bool live = hi_ < n;
  uint64_t c_key = 0, c_mask = 0;
  double c_stay = kNegInf, c_ab = 0.0, c_p = 0.0, c_L = 0.0;
  int c_last = 0;
  if (live) {
    c_ab = sAb[hi_];
    c_p = sP[hi_];
    c_L = sL[hi_];
    c_last = sMeta[hi_] & 0xFF;
    c_mask = sMask[hi_];
    c_key = sKey[hi_];
    if (ln == 0) c_stay = sStay[hi_];
  }
  auto score_now = [&](int k) -> double {
    const int v = 1 + ln + LPB * k;
    if (v > kSep || !((c_mask >> v) & 1ull)) return kNegInf;
    const double base = (v == c_last) ? c_ab : c_p;
    return ((base + sD[v]) + (v == kSep ? P.gamma : P.beta)) + c_L;
  };
  auto score_of = score_now;
  auto key_of = [&](int v) -> uint64_t { return v == 0 ? c_key : prefix_step(c_key, v); };
  // f(v, score) for each of this lane's candidates with a finite score
  auto for_cands = [&](auto&& f) {
    if (c_stay != kNegInf) f(0, c_stay);
#pragma unroll LB_CAND_UNROLL
    for (int k = 0; k < NC; ++k) {
      const double s = score_of(k);
      if (s != kNegInf) f(1 + ln + LPB * k, s);
    }
  };

  double mx = kNegInf, mn = HUGE_VAL;
  for_cands([&](int, double s) {
    mx = fmax(mx, s);
    mn = fmin(mn, s);
  });
  double best, lowest;
  block_minmax<BLOCK>(mx, mn, sRed, &best, &lowest);
  const double thr = best - P.theta;

  // ---- top-K.  Level 0 bins (best - score) over [max(thr, lowest), best] into
  // kBins; the map is monotone, so bins above the one holding the K-th
  // candidate are taken whole.  That bin is resolved exactly by rank on
  // (score desc, key asc) when it holds at most kBoundaryCap candidates;
  // otherwise it is re-binned over its own score range (deeper levels), and
  // when its scores are all equal, by the bits of the key (smaller key first).
  const double lo0 = fmax(thr, lowest);
  const double inv0 = best > lo0 ? static_cast<double>(kBins) / (best - lo0) : 0.0;
  const int shift0 = best > lo0 ? -1 : 64 - 10;
  auto bin_score = [&](double hi, double inv, double s) -> int {
    const double x = (hi - s) * inv;
    return x >= static_cast<double>(kBins - 1) ? kBins - 1 : static_cast<int>(x);
  };
  auto bin0 = [&](int v, double s) -> int {
    return shift0 < 0 ? bin_score(best, inv0, s) : static_cast<int>((key_of(v) >> shift0) & (kBins - 1));
  };
  // deeper levels (rare): parameters in LDS
  auto bin_at = [&](int l, int v, double s) -> int {
    const int sh = sLvShift[l];
    if (sh >= 0) return static_cast<int>((key_of(v) >> sh) & (kBins - 1));
    return bin_score(sLvHi[l], sLvInv[l], s);
  };
  // candidates in the boundary bin of levels 0..L-1
  auto member = [&](int L, int v, double s) -> bool {
    if (s < thr || bin0(v, s) != sLvBeta[0]) return false;
    for (int l = 1; l < L; ++l)
      if (bin_at(l, v, s) != sLvBeta[l]) return false;
    return true;
  };
  // the lane's candidates with scores recomputed (no register array): for the rare levels
  auto for_cands_rt = [&](auto&& f) {
    if (c_stay != kNegInf) f(0, c_stay);
#pragma unroll 1
    for (int k = 0; k < NC; ++k) {
      const double s = score_now(k);
      if (s != kNegInf) f(1 + ln + LPB * k, s);
    }
  };
  // finds the bin holding the need-th candidate of sHisto; returns via sBucket/sAbove/sBucketCnt
  auto find_bin = [&](int need_in) -> int {
    constexpr int PER = (kBins + BLOCK - 1) / BLOCK;
    int local = 0;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int d = tid * PER + q;
      local += d < kBins ? static_cast<int>(sHisto[d]) : 0;
    }
    int tot = 0;
    const int before = block_scan<BLOCK>(local, sScan, &tot);
    if (need_in > 0 && before < need_in && before + local >= need_in) {
      int acc = before;
      for (int q = 0; q < PER; ++q) {
        const int d = tid * PER + q;
        const int h = static_cast<int>(sHisto[d]);
        if (acc + h >= need_in) {
          sBucket = d;
          sAbove = acc;
          sBucketCnt = h;
          break;
        }
        acc += h;
      }
    }
    __syncthreads();
    return tot;
  };

  // level-0 bin of each of the lane's candidates, kept packed 16 bits per slot
  // (0xFFFF: no candidate); exact scores are recomputed only inside the boundary bin
  uint32_t binp[(NC + 1) / 2];
  uint32_t bin_stay = 0xFFFFu;
  for (int d = tid; d < kBins; d += BLOCK) sHisto[d] = 0;
  __syncthreads();
  if (c_stay != kNegInf && c_stay >= thr) {
    bin_stay = static_cast<uint32_t>(bin0(0, c_stay));
    atomicAdd(&sHisto[bin_stay], 1u);
  }
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const double s = score_now(k);
    uint32_t bn = 0xFFFFu;
    if (s != kNegInf && s >= thr) {
      bn = static_cast<uint32_t>(bin0(1 + ln + LPB * k, s));
      atomicAdd(&sHisto[bn], 1u);
    }
    if (k & 1)
      binp[k >> 1] |= bn << 16;
    else
      binp[k >> 1] = bn;
  }
  __syncthreads();
  const int nvalid = find_bin(P.K);
  const bool select_all = nvalid <= P.K;
  int beta0 = kBins, nlev = 1, need = P.K, nbc = 0;
  bool all_bin = false;
  if (!select_all) {
    beta0 = sBucket;
    need -= sAbove;
    int cntb = sBucketCnt;
    if (tid == 0) {
      sLvBeta[0] = beta0;
      sLvShift[0] = shift0;
    }
    __syncthreads();
    int key_shift = shift0 >= 0 ? shift0 - 10 : 64 - 10;
    bool key_level = shift0 >= 0;
    while (cntb != need && cntb > kBoundaryCap && !(key_level && sLvShift[nlev - 1] == 0) && nlev < kMaxLevels) {
      // refine: score range of the boundary bin's members, or key bits when it is flat
      const int L = nlev;
      double bmx = kNegInf, bmn = HUGE_VAL;
      for_cands_rt([&](int v, double s) {
        if (member(L, v, s)) {
          bmx = fmax(bmx, s);
          bmn = fmin(bmn, s);
        }
      });
      double lv_hi, lv_lo;
      block_minmax<BLOCK>(bmx, bmn, sRed, &lv_hi, &lv_lo);
      if (tid == 0) {
        sLvHi[L] = lv_hi;
        sLvInv[L] = lv_hi > lv_lo ? static_cast<double>(kBins) / (lv_hi - lv_lo) : 0.0;
        sLvShift[L] = lv_hi > lv_lo ? -1 : (key_shift > 0 ? key_shift : 0);
      }
      for (int d = tid; d < kBins; d += BLOCK) sHisto[d] = 0;
      __syncthreads();
      key_level = sLvShift[L] >= 0;
      if (key_level) key_shift -= 10;
      for_cands_rt([&](int v, double s) {
        if (member(L, v, s)) atomicAdd(&sHisto[bin_at(L, v, s)], 1u);
      });
      __syncthreads();
      (void)find_bin(need);
      if (tid == 0) sLvBeta[L] = sBucket;
      need -= sAbove;
      cntb = sBucketCnt;
      nlev = L + 1;
      __syncthreads();
    }
    if (cntb == need) {
      all_bin = true;
    } else {
      // exact rank inside the boundary bin (a flat key level of shift 0 holds one key)
      if (tid == 0) sBCount = 0;
      __syncthreads();
      const int L = nlev;
      for_cands_rt([&](int v, double s) {
        if (!member(L, v, s)) return;
        const int slot = atomicAdd(&sBCount, 1);
        if (slot < kBoundaryCap) {
          sBScore[slot] = s;
          sBKey[slot] = key_of(v);
        }
      });
      __syncthreads();
      nbc = sBCount < kBoundaryCap ? sBCount : kBoundaryCap;
      if (sBCount > kBoundaryCap && tid == 0) atomicOr(S.flags, kFlagSelect);
    }
  }
  // selection of a candidate from its level-0 bin; the exact score (score_fn)
  // is needed only inside the boundary bin
  auto selected = [&](uint32_t bn, int v, auto&& score_fn) -> bool {
    if (bn == 0xFFFFu) return false;
    if (select_all) return true;
    if (static_cast<int>(bn) != beta0) return static_cast<int>(bn) < beta0;
    const double s = score_fn();
    for (int l = 1; l < nlev; ++l) {
      const int bl = bin_at(l, v, s);
      if (bl != sLvBeta[l]) return bl < sLvBeta[l];
    }
    if (all_bin) return true;
    // rank inside the boundary bin by (score desc, key asc)
    const uint64_t k = key_of(v);
    int rank = 0;
    for (int u = 0; u < nbc; ++u) rank += ranks_before(sBScore[u], sBKey[u], s, k);
    return rank < need;
  };

  // ---- selection bits (bit 0: the stay, bit k+1: slot k), then a
  // deterministic gather of the sources in lane order
  uint64_t sel_bits = 0;
  if (selected(bin_stay, 0, [&] { return c_stay; })) sel_bits |= 1ull;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const uint32_t bn = (binp[k >> 1] >> ((k & 1) * 16)) & 0xFFFFu;
    if (selected(bn, 1 + ln + LPB * k, [&] { return score_now(k); })) sel_bits |= 2ull << k;
  }
  int nsel = 0;
  int wpos = block_scan<BLOCK>(__popcll(sel_bits), sScan, &nsel);
  if (nsel > P.K) {  // cannot happen when the selection is exact; never write past K entries
    nsel = P.K;
    if (tid == 0) atomicOr(S.flags, kFlagSelect);
  }
  if ((sel_bits & 1ull) && wpos < nsel) sSelSrc[wpos++] = static_cast<uint32_t>(hi_);
#pragma unroll LB_CAND_UNROLL
  for (int k = 0; k < NC; ++k)
    if (((sel_bits >> (k + 1)) & 1ull) && wpos < nsel)
      sSelSrc[wpos++] = static_cast<uint32_t>(hi_) | (static_cast<uint32_t>(1 + ln + LPB * k) << 16);
  __syncthreads();

  // ---- write the new hypotheses (in place: every old value is in LDS)
  const int r = tid;
  int is_event = 0, my_nq = 0, ev_src = 0;
  uint32_t ev_pnode = 0, ev_woff = 0, ev_H = 0, ev_nsub = 0;
  if (r < nsel) {
    const uint32_t src = sSelSrc[r];
    const int i = src & 0xFFFF;
    const int v = src >> 16;
    const size_t o = gb + r;
    const uint32_t meta_i = sMeta[i];
    const int nsub = (meta_i >> 8) & 0xFF;
    if (v == 0) {
      S.key[o] = sKey[i];
      S.pkey[o] = sPkey[i];
      S.ab[o] = sAb2[i];
      S.anb[o] = sAnb2[i];
      S.pt[o] = sPt2[i];
      S.node[o] = sNode[i];
      S.meta[o] = meta_i;
    } else {
      const int last = meta_i & 0xFF;
      const double base = (v == last) ? sAb[i] : sP[i];
      const double anb = (base + sD[v]) + (v == kSep ? P.gamma : P.beta);
      S.key[o] = prefix_step(sKey[i], v);
      S.pkey[o] = sKey[i];
      S.ab[o] = kNegInf;
      S.anb[o] = anb;
      S.pt[o] = lse2(kNegInf, anb);
      uint32_t child = kRootNode;
      if (v != kSep) child = sFirst[i] + __popcll(sTrieMask[i] & ((1ull << v) - 1ull));
      S.node[o] = child;
      S.meta[o] = static_cast<uint32_t>(v) | (meta_i & 0xFF00u);
      if (v == kSep) {
        is_event = 1;
        ev_pnode = sNode[i];
        ev_woff = sWoff[i];
        ev_H = sNwords[i];
        ev_nsub = static_cast<uint32_t>(nsub);
        my_nq = static_cast<int>(ev_nsub * ev_H);
        ev_src = i;
      }
    }
    for (int j = 0; j < nsub; ++j) {
      S.Lw[o * P.O + j] = sLw[i * kMaxSub + j];
      S.hist[o * P.O + j] = sHist[i * kMaxSub + j];
    }
  }
  int nev = 0, nq_blk = 0;
  const int erank = block_scan<BLOCK>(is_event, sScan, &nev);
  const int qpos = block_scan<BLOCK>(my_nq, sScan, &nq_blk);
  if (tid == 0) {
    S.nbeam[b] = nsel;
    sEvBase = nev ? atomicAdd(&S.evq[tau & 1], (static_cast<unsigned long long>(nev) << 32) |
                                                   static_cast<unsigned long long>(nq_blk))
                  : 0ull;
    unsigned long long* cn = S.counters + static_cast<size_t>(b) * kNumCounters;
    cn[kCntExpansions] += static_cast<unsigned long long>(n) * kClasses;
    cn[kCntFrames] += 1;
  }
  if (is_event) sEvQ[erank] = static_cast<uint32_t>(qpos);
  __syncthreads();
  const uint32_t ev0 = static_cast<uint32_t>(sEvBase >> 32);
  const uint32_t q0 = static_cast<uint32_t>(sEvBase);
  if (is_event) {
    Event e;
    e.stream = b;
    e.beam = r;
    e.pnode = ev_pnode;
    e.woff = ev_woff;
    e.H = ev_H;
    e.nsub = ev_nsub;
    e.qoff = q0 + qpos;
    e.pad = 0;
#pragma unroll
    for (int j = 0; j < kMaxSub; ++j) e.hist[j] = j < static_cast<int>(ev_nsub) ? sHist[ev_src * kMaxSub + j] : 0u;
    S.events[ev0 + erank] = e;
  }
  // query -> event map of this block's queries (events are contiguous, in order)
  for (int k = tid; k < nq_blk; k += BLOCK) {
    int lo = 0, hi = nev - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (sEvQ[mid] <= static_cast<uint32_t>(k)) lo = mid; else hi = mid - 1;
    }
    S.qmap[q0 + k] = ev0 + lo;
  }
}

// ------------------------------------------------------------------ n-gram shallow fusion

// One 64-B bucket: four 16-B slots {key lo, key hi, log10 p, backoff}.
struct Bucket {
  uint4 s0, s1, s2, s3;
};

__device__ __forceinline__ Bucket load_bucket(const NgramTable& t, uint64_t bk) {
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

// Scans a bucket for `key`: 1 found (slot index and values set), 0 absent, -1 bucket full.
__device__ __forceinline__ int scan_bucket(const Bucket& q, uint64_t key, uint64_t bk, uint32_t* slot, float* lp,
                                           float* bo) {
#define LB_SCAN_SLOT(V, K)                              \
  {                                                     \
    const uint64_t kk = slot_key(V);                    \
    if (kk == key) {                                    \
      *slot = static_cast<uint32_t>(bk * 4 + (K));      \
      *lp = __uint_as_float((V).z);                     \
      *bo = __uint_as_float((V).w);                     \
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
__device__ __forceinline__ bool resolve(const NgramTable& t, uint64_t key, uint64_t bk, const Bucket& first,
                                        uint32_t* slot, float* lp, float* bo, uint32_t* lines) {
  int r = scan_bucket(first, key, bk, slot, lp, bo);
  for (uint64_t it = 1; r < 0 && it < t.nbuckets; ++it) {
    bk = (bk + 1 == t.nbuckets) ? 0 : bk + 1;
    ++*lines;
    r = scan_bucket(load_bucket(t, bk), key, bk, slot, lp, bo);
  }
  return r == 1;
}

__device__ __forceinline__ uint32_t hist_of(const Event& ev, uint32_t j) {
  return j == 0 ? ev.hist[0] : (j == 1 ? ev.hist[1] : (j == 2 ? ev.hist[2] : ev.hist[3]));
}

// The LM lookup phase: one thread per (completed word, parent sub-beam,
// homophone) query of the frame, over every stream.  The three bucket lines
// (orders 2, 3, 4) and the unigram are loaded together, then resolved.
__global__ __launch_bounds__(256) void k_lmquery(const DevParams P, const DevState S, int32_t tau) {
  const uint32_t nq = static_cast<uint32_t>(S.evq[tau & 1]);
  uint32_t lines = 0;
  const uint32_t stride = gridDim.x * blockDim.x;
  for (uint32_t q = blockIdx.x * blockDim.x + threadIdx.x; q < nq; q += stride) {
    const Event ev = S.events[S.qmap[q]];
    const uint32_t loc = q - ev.qoff;
    const uint32_t j = loc / ev.H;
    const uint32_t h = loc - j * ev.H;
    const int w = S.trie_words[ev.woff + h];
    const uint32_t ph = hist_of(ev, j);
    const HistNode ctx = S.arena[ph];
    const double Lw = S.Lw[(static_cast<size_t>(ev.stream) * P.K + ev.beam) * P.O + j];
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
    lines += 1u + (has3 ? 1u : 0u) + (has4 ? 1u : 0u);
    uint32_t s2 = kNone, s3 = kNone, s4 = kNone;
    float p2 = 0.f, bb2 = 0.f, p3 = 0.f, bb3 = 0.f, p4 = 0.f, bb4 = 0.f;
    const bool f2 = resolve(S.t2, k2, b2, q2, &s2, &p2, &bb2, &lines);
    const bool f3 = has3 && resolve(S.t3, k3, b3, q3, &s3, &p3, &bb3, &lines);
    const bool f4 = has4 && resolve(S.t4, k4, b4, q4, &s4, &p4, &bb4, &lines);
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
    S.qL[q] = Lw + P.comega * lp;
    QState st;
    st.c2 = f2 ? s2 : kNone;
    st.c3 = f3 ? s3 : kNone;
    st.bo2 = f2 ? bb2 : 0.0f;
    st.bo3 = f3 ? bb3 : 0.0f;
    S.qS[q] = st;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) lines += __shfl_xor(lines, o, 64);
  if ((threadIdx.x & 63) == 0 && lines) {
    const uint32_t slot = ((blockIdx.x * blockDim.x + threadIdx.x) >> 6) & (kSpread - 1);
    atomicAdd(&S.lines[slot * kSpreadStride], static_cast<unsigned long long>(lines));
  }
}

// Homophone top-o (Eq. (1), App. E.3): one wavefront per completed word ranks
// its queries by (score desc, (sub-beam, homophone) index asc), keeps o, drops
// those more than lambda below the best, and appends word-history nodes.
__global__ __launch_bounds__(256) void k_lmselect(const DevParams P, const DevState S, int32_t tau) {
  const uint32_t nev = static_cast<uint32_t>(S.evq[tau & 1] >> 32);
  const int lane = threadIdx.x & 63;
  const uint32_t wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const uint32_t nwaves = (gridDim.x * blockDim.x) >> 6;
  const bool synth = P.fusion_source == 1;
  for (uint32_t e = wave; e < nev; e += nwaves) {
    const Event ev = S.events[e];
    const size_t bi = static_cast<size_t>(ev.stream) * P.K + ev.beam;
    const int nq = static_cast<int>(ev.nsub * ev.H);
    double tL[kMaxSub];
    int tq[kMaxSub];
#pragma unroll
    for (int k = 0; k < kMaxSub; ++k) {
      tL[k] = kNegInf;
      tq[k] = 0x7FFFFFFF;
    }
    auto insert = [&](double L, int qq) {
#pragma unroll
      for (int k = 0; k < kMaxSub; ++k) {
        if (k < P.O && (L > tL[k] || (L == tL[k] && qq < tq[k]))) {
          const double t = tL[k];
          const int u = tq[k];
          tL[k] = L;
          tq[k] = qq;
          L = t;
          qq = u;
        }
      }
    };
    // four independent loads in flight per lane, then the insertions
    const double* ql = S.qL + ev.qoff;
    int q = lane;
    for (; q + 192 < nq; q += 256) {
      const double a0 = ql[q], a1 = ql[q + 64], a2 = ql[q + 128], a3 = ql[q + 192];
      insert(a0, q);
      insert(a1, q + 64);
      insert(a2, q + 128);
      insert(a3, q + 192);
    }
    for (; q < nq; q += 64) insert(ql[q], q);
    uint32_t abase = 0;
    if (lane == 0) abase = atomicAdd(&S.arena_n[ev.stream], static_cast<uint32_t>(P.O));
    abase = __shfl(abase, 0, 64);
    const bool room = static_cast<uint64_t>(abase) + P.O <= S.arena_cap;
    if (!room && lane == 0) atomicOr(S.flags, kFlagArena);
    const uint32_t node0 = 1u + static_cast<uint32_t>(static_cast<uint64_t>(ev.stream) * S.arena_cap) + abase;
    double bestL = kNegInf;
    int kept = 0;
#pragma unroll
    for (int k = 0; k < kMaxSub; ++k) {
      if (k >= P.O) break;
      double bL = tL[0];
      int bq = tq[0];
      int bl = lane;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const double oL = __shfl_xor(bL, o, 64);
        const int oq = __shfl_xor(bq, o, 64);
        const int ol = __shfl_xor(bl, o, 64);
        if (oL > bL || (oL == bL && (oq < bq || (oq == bq && ol < bl)))) {
          bL = oL;
          bq = oq;
          bl = ol;
        }
      }
      if (bL == kNegInf) break;
      if (k == 0) bestL = bL;
      if (bL < bestL - P.lam) break;
      if (lane == bl) {
        if (room) {
          const uint32_t j = static_cast<uint32_t>(bq) / ev.H;
          const uint32_t h = static_cast<uint32_t>(bq) - j * ev.H;
          const int w = S.trie_words[ev.woff + h];
          const uint32_t ph = hist_of(ev, j);
          const QState st = S.qS[ev.qoff + bq];
          HistNode hn;
          hn.parent = ph;
          hn.word = w;
          hn.c2 = st.c2;
          hn.c3 = st.c3;
          hn.bo1 = S.uni[w].bo;
          hn.bo2 = st.bo2;
          hn.bo3 = st.bo3;
          hn.pad = 0;
          if (synth) {
            const HistNode ctx = S.arena[ph];
            hn.sfus = ctx.sfus + bigram_score(P, ctx.word, w);
          } else {
            hn.sfus = 0.0;
          }
          S.arena[node0 + k] = hn;
          S.Lw[bi * P.O + k] = bL;
          S.hist[bi * P.O + k] = node0 + k;
        }
#pragma unroll
        for (int m = 0; m + 1 < kMaxSub; ++m) {
          tL[m] = tL[m + 1];
          tq[m] = tq[m + 1];
        }
        tL[kMaxSub - 1] = kNegInf;
        tq[kMaxSub - 1] = 0x7FFFFFFF;
      }
      kept = k + 1;
    }
    if (lane == 0) {
      if (room) S.meta[bi] = (S.meta[bi] & 0xFFu) | (static_cast<uint32_t>(kept) << 8);
      unsigned long long* cn = S.counters + static_cast<size_t>(ev.stream) * kNumCounters;
      atomicAdd(&cn[kCntWordEvents], 1ull);
      atomicAdd(&cn[kCntLmQueries], static_cast<unsigned long long>(nq));
    }
  }
}

// ------------------------------------------------------------------ delayed fusion

// Selects the top-F hypotheses of stream b by (total desc, key asc) into
// S.fsel[b][0..F) and S.fsel_n[b] (F = all hypotheses when top_f <= 0).
template <int BLOCK>
__device__ void select_fused(const DevParams& P, const DevState& S, int b, int top_f, double* sc, uint64_t* ky,
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
    } else {
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
template <int BLOCK>
__device__ void apply_fused(const DevParams& P, const DevState& S, int b, const float* ext) {
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
        const double f = ext ? static_cast<double>(ext[(gb + tid) * P.O + j]) : S.arena[h[j]].sfus;
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

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fusion(const DevParams P, const DevState S,
                                                  const int32_t* __restrict__ lengths, int32_t tau) {
  const int b = blockIdx.x;
  if (tau >= lengths[b]) return;
  const int64_t t = S.t0[b] + tau;
  if (t == 0 || t % P.fusion_interval != 0) return;
  __shared__ double sc[BLOCK];
  __shared__ uint64_t ky[BLOCK];
  __shared__ uint32_t ix[BLOCK];
  select_fused<BLOCK>(P, S, b, P.fusion_top_f, sc, ky, ix);
  apply_fused<BLOCK>(P, S, b, nullptr);
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
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fuse_export(const DevParams P, const DevState S,
                                                       int32_t* __restrict__ words, int32_t* __restrict__ n_words) {
  const int b = blockIdx.x;
  const size_t gb = static_cast<size_t>(b) * P.K;
  const int F = S.fsel_n[b];
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
        len = 0;
        for (uint32_t x = h; x != kRootHist && static_cast<uint64_t>(len) <= S.arena_cap; x = S.arena[x].parent) ++len;
        if (len > P.W) atomicOr(S.flags, kFlagWords);
        int k = len - 1;
        for (uint32_t x = h; x != kRootHist && k >= 0; x = S.arena[x].parent, --k)
          if (k < P.W) row[k] = S.arena[x].word;
        for (int k2 = len; k2 < P.W; ++k2) row[k2] = -1;
        if (len > P.W) len = P.W;
      }
    }
    if (len < 0)
      for (int k2 = 0; k2 < P.W; ++k2) row[k2] = -1;
    n_words[slot] = len;
  }
}

// External scorer, step 3: apply the caller's scores [B][K][O] to the selection.
template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_fuse_apply(const DevParams P, const DevState S,
                                                      const float* __restrict__ scores) {
  apply_fused<BLOCK>(P, S, blockIdx.x, scores);
}

// ------------------------------------------------------------------ output

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_output(const DevParams P, const DevState S,
                                                  const int32_t* __restrict__ lengths, int32_t fin,
                                                  int32_t* __restrict__ out_hyps,
                                                  float* __restrict__ out_scores) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ double sc[BLOCK];
  __shared__ uint64_t ky[BLOCK];
  __shared__ uint32_t ix[BLOCK];
  __shared__ int32_t sScan[BLOCK / 64];
  if (b == 0 && tid == 0) {
    S.evq[0] = 0;
    S.evq[1] = 0;
  }
  if (fin && P.fusion_source == 1 && P.fusion_interval > 0) {
    select_fused<BLOCK>(P, S, b, 0, sc, ky, ix);
    apply_fused<BLOCK>(P, S, b, nullptr);
  }
  const int n = S.nbeam[b];
  const size_t gb = static_cast<size_t>(b) * P.K;
  bool ok = false;
  if (tid < n) {
    ok = !fin || S.node[gb + tid] == kRootNode;
    sc[tid] = ok ? S.pt[gb + tid] + S.Lw[(gb + tid) * P.O] : kNegInf;
    ky[tid] = ok ? S.key[gb + tid] : ~0ull;
    ix[tid] = tid;
  } else {
    sc[tid] = kNegInf;
    ky[tid] = ~0ull;
    ix[tid] = 0;
  }
  int m = 0;
  (void)block_scan<BLOCK>(ok ? 1 : 0, sScan, &m);
  bitonic_sort<BLOCK>(sc, ky, ix);
  if (tid == 0) S.t0[b] += lengths[b];
  for (int r = tid; r < P.K; r += BLOCK) {
    int32_t* row = out_hyps + (static_cast<size_t>(b) * P.K + r) * P.W;
    if (r < m) {
      const size_t bi = gb + ix[r];
      out_scores[static_cast<size_t>(b) * P.K + r] = static_cast<float>(sc[r]);
      uint32_t h = S.hist[bi * P.O];
      int len = 0;
      for (uint32_t x = h; x != kRootHist && static_cast<uint64_t>(len) <= S.arena_cap; x = S.arena[x].parent)
        ++len;
      if (len > P.W) atomicOr(S.flags, kFlagWords);
      int k = len - 1;
      for (uint32_t x = h; x != kRootHist && k >= 0; x = S.arena[x].parent, --k)
        if (k < P.W) row[k] = S.arena[x].word;
      for (int k2 = len; k2 < P.W; ++k2) row[k2] = -1;
    } else {
      out_scores[static_cast<size_t>(b) * P.K + r] = kNegInf;
      for (int k2 = 0; k2 < P.W; ++k2) row[k2] = -1;
    }
  }
}

}  // namespace

// ------------------------------------------------------------------ launchers

hipError_t launch_build_order(int order, const int32_t* ids, const float* lp, const float* bo, int64_t count,
                              int32_t vocab, NgramTable t2, NgramTable t3, NgramTable dst, uint32_t* flags,
                              hipStream_t st) {
  if (count <= 0) return hipSuccess;
  const int64_t blocks = (count + 255) / 256;
  const int grid = static_cast<int>(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(k_build_order, dim3(grid), dim3(256), 0, st, order, ids, lp, bo, count, vocab, t2, t3,
                     dst, flags);
  return hipGetLastError();
}

hipError_t launch_begin(const DevParams& P, const DevState& S, int32_t B, hipStream_t st) {
  hipLaunchKernelGGL(k_begin, dim3((B + 255) / 256), dim3(256), 0, st, P, S, B);
  return hipGetLastError();
}

#define LB_DISPATCH_BLOCK(BLK, KERNEL, GRID, ...)                                           \
  do {                                                                                      \
    if ((BLK) == 64)                                                                        \
      hipLaunchKernelGGL(KERNEL<64>, dim3(GRID), dim3(64), 0, st, __VA_ARGS__);             \
    else if ((BLK) == 128)                                                                  \
      hipLaunchKernelGGL(KERNEL<128>, dim3(GRID), dim3(128), 0, st, __VA_ARGS__);           \
    else                                                                                    \
      hipLaunchKernelGGL(KERNEL<256>, dim3(GRID), dim3(256), 0, st, __VA_ARGS__);           \
  } while (0)

// Frame-kernel shapes: (hypotheses per workgroup, lanes per hypothesis).
hipError_t launch_frame(int K, const DevParams& P, const DevState& S, const float* logits,
                        const int32_t* lengths, int32_t B, int32_t Tc, int32_t tau, hipStream_t st) {
  if (K <= 16)
    hipLaunchKernelGGL((k_frame<16, 4>), dim3(B), dim3(64), 0, st, P, S, logits, lengths, Tc, tau);
  else if (K <= 32)
    hipLaunchKernelGGL((k_frame<32, 4>), dim3(B), dim3(128), 0, st, P, S, logits, lengths, Tc, tau);
  else if (K <= 64)
    hipLaunchKernelGGL((k_frame<64, 4>), dim3(B), dim3(256), 0, st, P, S, logits, lengths, Tc, tau);
  else if (K <= 128)
    hipLaunchKernelGGL((k_frame<128, LB_LPB_LARGE>), dim3(B), dim3(128 * LB_LPB_LARGE), 0, st, P, S, logits, lengths,
                       Tc, tau);
  else
    hipLaunchKernelGGL((k_frame<256, LB_LPB_LARGE>), dim3(B), dim3(256 * LB_LPB_LARGE), 0, st, P, S, logits, lengths,
                       Tc, tau);
  return hipGetLastError();
}

hipError_t launch_lmquery(int grid, const DevParams& P, const DevState& S, int32_t tau, hipStream_t st) {
  hipLaunchKernelGGL(k_lmquery, dim3(grid), dim3(256), 0, st, P, S, tau);
  return hipGetLastError();
}

hipError_t launch_lmselect(int grid, const DevParams& P, const DevState& S, int32_t tau, hipStream_t st) {
  hipLaunchKernelGGL(k_lmselect, dim3(grid), dim3(256), 0, st, P, S, tau);
  return hipGetLastError();
}

hipError_t launch_fusion(int block, const DevParams& P, const DevState& S, const int32_t* lengths, int32_t B,
                         int32_t tau, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_fusion, B, P, S, lengths, tau);
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
                         int32_t fin, int32_t* out_hyps, float* out_scores, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_output, B, P, S, lengths, fin, out_hyps, out_scores);
  return hipGetLastError();
}

}  // namespace lb
