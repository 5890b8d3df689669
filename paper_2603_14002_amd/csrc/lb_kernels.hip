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
  S.node[i] = kRootNode;
  S.meta[i] = 1u << 8;  // no last symbol, one sub-beam
  S.Lw[i * P.O] = 0.0;
  S.hist[i * P.O] = kRootHist;
  S.t0[b] = 0;
  S.arena_n[b] = 0;
}

// ------------------------------------------------------------------ frame step

template <int BLOCK>
__global__ __launch_bounds__(BLOCK) void k_frame(const DevParams P, const DevState S,
                                                 const float* __restrict__ logits,
                                                 const int32_t* __restrict__ lengths, int32_t Tc,
                                                 int32_t tau) {
  constexpr int HS = 2 * BLOCK;  // LDS hash slots for the current prefix keys
  constexpr int NW = BLOCK / 64;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  if (b == 0 && tid == 0) S.ev_count[(tau + 1) & 1] = 0;
  if (tau >= lengths[b]) return;

  __shared__ double sD[kClasses];
  __shared__ uint64_t sKey[BLOCK], sPkey[BLOCK];
  __shared__ double sAb[BLOCK], sP[BLOCK], sL[BLOCK], sAb2[BLOCK], sAnb2[BLOCK], sStay[BLOCK];
  __shared__ uint32_t sNode[BLOCK], sMeta[BLOCK], sFirst[BLOCK];
  __shared__ uint64_t sMask[BLOCK], sTrieMask[BLOCK];
  __shared__ double sLw[BLOCK * kMaxSub];
  __shared__ uint32_t sHist[BLOCK * kMaxSub];
  __shared__ unsigned long long sHKey[HS];
  __shared__ int32_t sHIdx[HS];
  __shared__ uint32_t sHisto[256];
  __shared__ double sSelScore[BLOCK];
  __shared__ uint64_t sSelKey[BLOCK];
  __shared__ uint32_t sSelSrc[BLOCK];
  __shared__ double sRed[NW];
  __shared__ int32_t sScan[NW];
  __shared__ int32_t sBucket, sAbove, sBucketCnt, sEvBase;

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
    sKey[tid] = my_key;
    sPkey[tid] = my_pkey;
    sAb[tid] = ab;
    sP[tid] = lse2(ab, my_anb);
    sNode[tid] = node;
    sMeta[tid] = my_meta;
    const int nsub = (my_meta >> 8) & 0xFF;
    for (int j = 0; j < nsub; ++j) {
      sLw[tid * kMaxSub + j] = S.Lw[(gb + tid) * P.O + j];
      sHist[tid * kMaxSub + j] = S.hist[(gb + tid) * P.O + j];
    }
    sL[tid] = sLw[tid * kMaxSub];
    const TrieNode tn = S.trie[node];
    sMask[tid] = tn.mask;
    sTrieMask[tid] = tn.mask;
    sFirst[tid] = tn.first_child;
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
    sAb2[tid] = ab2;
    sAnb2[tid] = anb2;
    sStay[tid] = lse2(ab2, anb2) + sL[tid];
  }
  __syncthreads();

  // candidate c = i*41 + v: v = 0 is hypothesis i's stay, v >= 1 its extension by v
  auto cand = [&](int c, double* score) -> bool {
    const int i = c / kClasses;
    const int v = c - i * kClasses;
    double s;
    if (v == 0) {
      s = sStay[i];
    } else {
      if (!((sMask[i] >> v) & 1ull)) return false;
      const int last = sMeta[i] & 0xFF;
      const double base = (v == last) ? sAb[i] : sP[i];
      s = ((base + sD[v]) + (v == kSep ? P.gamma : P.beta)) + sL[i];
    }
    *score = s;
    return s != kNegInf;
  };
  auto cand_key = [&](int c) -> uint64_t {
    const int i = c / kClasses;
    const int v = c - i * kClasses;
    return v == 0 ? sKey[i] : prefix_step(sKey[i], v);
  };

  const int nc = n * kClasses;
  double mx = kNegInf;
  for (int c = tid; c < nc; c += BLOCK) {
    double s;
    if (cand(c, &s)) mx = fmax(mx, s);
  }
  const double best = block_max<BLOCK>(mx, sRed);
  const double thr = best - P.theta;

  int cnt = 0;
  for (int c = tid; c < nc; c += BLOCK) {
    double s;
    if (cand(c, &s) && s >= thr) ++cnt;
  }
  int nvalid = 0;
  (void)block_scan<BLOCK>(cnt, sScan, &nvalid);

  // ---- top-K: MSD radix select over (ordered score bits, ~key), 8 bits a pass
  uint64_t pre_hi = 0, pre_lo = 0, m_hi = 0, m_lo = 0;
  const bool select_all = nvalid <= P.K;
  if (!select_all) {
    const uint64_t ob_best = order_bits(best), ob_thr = order_bits(thr);
    const int common = (ob_best == ob_thr) ? 64 : __clzll(static_cast<long long>(ob_best ^ ob_thr));
    int pos = ((127 - common) / 8) * 8;
    mask_from(pos + 8, &m_hi, &m_lo);
    pre_hi = ob_best & m_hi;
    pre_lo = 0;
    int need = P.K;
    for (;;) {
      for (int d = tid; d < 256; d += BLOCK) sHisto[d] = 0;
      __syncthreads();
      const bool want_key = pos < 64;
      for (int c = tid; c < nc; c += BLOCK) {
        double s;
        if (!cand(c, &s) || s < thr) continue;
        const uint64_t hi = order_bits(s);
        if ((hi & m_hi) != pre_hi) continue;
        const uint64_t lo = want_key ? ~cand_key(c) : 0;
        if ((lo & m_lo) != pre_lo) continue;
        atomicAdd(&sHisto[digit128(hi, lo, pos)], 1u);
      }
      __syncthreads();
      if (tid < 64) {
        // lane l owns bins 4l..4l+3; find the bin holding the need-th largest
        const int l = tid;
        const uint32_t h0 = sHisto[4 * l], h1 = sHisto[4 * l + 1], h2 = sHisto[4 * l + 2],
                       h3 = sHisto[4 * l + 3];
        const int mine = static_cast<int>(h0 + h1 + h2 + h3);
        int suf = mine;  // inclusive suffix sum over lanes >= l
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int y = __shfl_down(suf, o, 64);
          if (l + o < 64) suf += y;
        }
        const int above_lane = suf - mine;
        if (above_lane < need && suf >= need) {
          int acc = above_lane;
          const uint32_t hh[4] = {h0, h1, h2, h3};
          for (int q = 3; q >= 0; --q) {
            if (acc + static_cast<int>(hh[q]) >= need) {
              sBucket = 4 * l + q;
              sAbove = acc;
              sBucketCnt = static_cast<int>(hh[q]);
              break;
            }
            acc += static_cast<int>(hh[q]);
          }
        }
      }
      __syncthreads();
      const int bucket = sBucket;
      need -= sAbove;
      const int bcnt = sBucketCnt;
      __syncthreads();
      if (pos >= 64) {
        pre_hi |= static_cast<uint64_t>(bucket) << (pos - 64);
      } else if (pos > 56) {
        pre_hi |= static_cast<uint64_t>(bucket) >> (64 - pos);
        pre_lo |= static_cast<uint64_t>(bucket) << pos;
      } else {
        pre_lo |= static_cast<uint64_t>(bucket) << pos;
      }
      mask_from(pos, &m_hi, &m_lo);
      if (bcnt == need || pos == 0) break;
      pos -= 8;
    }
  }

  // ---- gather the selected candidates (prefix-sum order), then sort them
  int mysel = 0;
  for (int c = tid; c < nc; c += BLOCK) {
    double s;
    if (!cand(c, &s) || s < thr) continue;
    if (!select_all) {
      const uint64_t hi = order_bits(s);
      if (hi < pre_hi || (hi == pre_hi && ~cand_key(c) < pre_lo)) continue;
    }
    ++mysel;
  }
  int nsel = 0;
  int wpos = block_scan<BLOCK>(mysel, sScan, &nsel);
  if (nsel > P.K) {  // cannot happen when the selection is exact; never write past K entries
    nsel = P.K;
    if (tid == 0) atomicOr(S.flags, kFlagSelect);
  }
  for (int c = tid; c < nc; c += BLOCK) {
    double s;
    if (!cand(c, &s) || s < thr) continue;
    const uint64_t hi = order_bits(s);
    if (!select_all && hi < pre_hi) continue;
    const uint64_t k = cand_key(c);
    if (!select_all && hi == pre_hi && ~k < pre_lo) continue;
    if (wpos >= nsel) break;
    const int i = c / kClasses;
    sSelScore[wpos] = s;
    sSelKey[wpos] = k;
    sSelSrc[wpos] = static_cast<uint32_t>(i) | (static_cast<uint32_t>(c - i * kClasses) << 16);
    ++wpos;
  }
  __syncthreads();
  if (tid >= nsel) {
    sSelScore[tid] = kNegInf;
    sSelKey[tid] = ~0ull;
    sSelSrc[tid] = 0;
  }
  __syncthreads();
  bitonic_sort<BLOCK>(sSelScore, sSelKey, sSelSrc);

  // ---- write the new hypotheses (in place: every old value is in LDS)
  const int r = tid;
  int is_event = 0;
  uint32_t ev_pnode = 0;
  if (r < nsel) {
    const uint32_t src = sSelSrc[r];
    const int i = src & 0xFFFF;
    const int v = src >> 16;
    const size_t o = gb + r;
    const uint32_t meta_i = sMeta[i];
    if (v == 0) {
      S.key[o] = sKey[i];
      S.pkey[o] = sPkey[i];
      S.ab[o] = sAb2[i];
      S.anb[o] = sAnb2[i];
      S.node[o] = sNode[i];
      S.meta[o] = meta_i;
    } else {
      const int last = meta_i & 0xFF;
      const double base = (v == last) ? sAb[i] : sP[i];
      S.key[o] = sSelKey[r];
      S.pkey[o] = sKey[i];
      S.ab[o] = kNegInf;
      S.anb[o] = (base + sD[v]) + (v == kSep ? P.gamma : P.beta);
      uint32_t child = kRootNode;
      if (v != kSep) child = sFirst[i] + __popcll(sTrieMask[i] & ((1ull << v) - 1ull));
      S.node[o] = child;
      S.meta[o] = static_cast<uint32_t>(v) | (meta_i & 0xFF00u);
      if (v == kSep) {
        is_event = 1;
        ev_pnode = sNode[i];
      }
    }
    const int nsub = (meta_i >> 8) & 0xFF;
    for (int j = 0; j < nsub; ++j) {
      S.Lw[o * P.O + j] = sLw[i * kMaxSub + j];
      S.hist[o * P.O + j] = sHist[i * kMaxSub + j];
    }
  }
  int nev = 0;
  const int epos = block_scan<BLOCK>(is_event, sScan, &nev);
  if (tid == 0) {
    S.nbeam[b] = nsel;
    sEvBase = nev ? static_cast<int>(atomicAdd(&S.ev_count[tau & 1], static_cast<uint32_t>(nev))) : 0;
    unsigned long long* cn = S.counters + static_cast<size_t>(b) * kNumCounters;
    cn[kCntExpansions] += static_cast<unsigned long long>(n) * kClasses;
    cn[kCntFrames] += 1;
  }
  __syncthreads();
  if (is_event) {
    Event e;
    e.stream = b;
    e.beam = r;
    e.pnode = ev_pnode;
    e.pad = 0;
    S.events[sEvBase + epos] = e;
  }
}

// ------------------------------------------------------------------ n-gram shallow fusion

struct SubCand {
  double L;
  int32_t q;       // (parent sub-beam, homophone) index: ties break on it ascending
  int32_t w;
  uint32_t ph;     // parent history node
  uint32_t c2, c3;
  float bo1, bo2, bo3;
  double sf;
};

__device__ inline bool sub_before(const SubCand& a, const SubCand& b) {
  return a.L > b.L || (a.L == b.L && a.q < b.q);
}

__global__ __launch_bounds__(256) void k_ngram(const DevParams P, const DevState S, int32_t tau) {
  const uint32_t count = S.ev_count[tau & 1];
  const int lane = threadIdx.x & 63;
  const uint32_t wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const uint32_t nwaves = (gridDim.x * blockDim.x) >> 6;
  const bool synth = P.fusion_source == 1;
  for (uint32_t e = wave; e < count; e += nwaves) {
    const Event ev = S.events[e];
    const size_t bi = static_cast<size_t>(ev.stream) * P.K + ev.beam;
    const uint32_t meta = S.meta[bi];
    const int nsub = (meta >> 8) & 0xFF;
    const uint32_t woff = S.trie[ev.pnode].word_off;
    const int H = static_cast<int>(S.trie[ev.pnode + 1].word_off - woff);
    const int nq = nsub * H;

    uint32_t lines = 0;
    SubCand top[kMaxSub];
#pragma unroll
    for (int k = 0; k < kMaxSub; ++k) {
      top[k].L = kNegInf;
      top[k].q = 0x7FFFFFFF;
    }
    for (int q = lane; q < nq; q += 64) {
      const int j = q / H;
      const int h = q - j * H;
      const int w = S.trie_words[woff + h];
      const uint32_t ph = S.hist[bi * P.O + j];
      const double Lw = S.Lw[bi * P.O + j];
      const HistNode ctx = S.arena[ph];
      uint32_t s2 = kNone, s3 = kNone, s4;
      float p2 = 0.f, b2 = 0.f, p3 = 0.f, b3 = 0.f, p4 = 0.f, b4;
      const bool f2 = probe(S.t2, (static_cast<uint64_t>(static_cast<uint32_t>(ctx.word)) << 32) |
                                      static_cast<uint32_t>(w), &s2, &p2, &b2, &lines);
      const bool f3 = ctx.c2 != kNone &&
                      probe(S.t3, (static_cast<uint64_t>(ctx.c2) << 32) | static_cast<uint32_t>(w), &s3, &p3, &b3, &lines);
      const bool f4 = ctx.c3 != kNone &&
                      probe(S.t4, (static_cast<uint64_t>(ctx.c3) << 32) | static_cast<uint32_t>(w), &s4, &p4, &b4, &lines);
      const Unigram u = S.uni[w];
      // log10 P(w | context) by backoff, innermost order first
      double lp;
      if (f4) {
        lp = static_cast<double>(p4);
      } else {
        double l3;
        if (f3) {
          l3 = static_cast<double>(p3);
        } else {
          const double l2 = f2 ? static_cast<double>(p2)
                               : static_cast<double>(ctx.bo1) + static_cast<double>(u.logp);
          l3 = static_cast<double>(ctx.bo2) + l2;
        }
        lp = static_cast<double>(ctx.bo3) + l3;
      }
      SubCand c;
      c.L = Lw + P.comega * lp;
      c.q = q;
      c.w = w;
      c.ph = ph;
      c.c2 = f2 ? s2 : kNone;
      c.c3 = f3 ? s3 : kNone;
      c.bo1 = u.bo;
      c.bo2 = f2 ? b2 : 0.0f;
      c.bo3 = f3 ? b3 : 0.0f;
      c.sf = synth ? ctx.sfus + bigram_score(P, ctx.word, w) : 0.0;
#pragma unroll
      for (int k = 0; k < kMaxSub; ++k) {
        if (k < P.O && sub_before(c, top[k])) {
          const SubCand t = top[k];
          top[k] = c;
          c = t;
        }
      }
    }

#pragma unroll
    for (int o = 32; o > 0; o >>= 1) lines += __shfl_xor(lines, o, 64);
    // merge the per-lane lists: O rounds of a wave arg-max on (L desc, q asc)
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
      double bL = top[0].L;
      int bq = top[0].q;
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
          HistNode hn;
          hn.parent = top[0].ph;
          hn.word = top[0].w;
          hn.c2 = top[0].c2;
          hn.c3 = top[0].c3;
          hn.bo1 = top[0].bo1;
          hn.bo2 = top[0].bo2;
          hn.bo3 = top[0].bo3;
          hn.pad = 0;
          hn.sfus = top[0].sf;
          S.arena[node0 + k] = hn;
          S.Lw[bi * P.O + k] = top[0].L;
          S.hist[bi * P.O + k] = node0 + k;
        }
#pragma unroll
        for (int m = 0; m + 1 < kMaxSub; ++m) top[m] = top[m + 1];
        top[kMaxSub - 1].L = kNegInf;
        top[kMaxSub - 1].q = 0x7FFFFFFF;
      }
      kept = k + 1;
    }
    if (lane == 0) {
      if (room) S.meta[bi] = (meta & 0xFFu) | (static_cast<uint32_t>(kept) << 8);
      unsigned long long* cn = S.counters + static_cast<size_t>(ev.stream) * kNumCounters;
      atomicAdd(&cn[kCntWordEvents], 1ull);
      atomicAdd(&cn[kCntLmQueries], static_cast<unsigned long long>(nq));
      atomicAdd(&cn[kCntProbeLines], static_cast<unsigned long long>(lines));
    }
  }
}

// ------------------------------------------------------------------ delayed fusion

// Replaces the sub-beam scores of the top-F hypotheses of stream b by
// phi * fusion score and re-ranks the sub-beams (stable).  `ext` (optional)
// holds caller scores [K][O] by fusion rank; otherwise the synthetic score of
// the history node is used.  Also records the selection in fsel.
template <int BLOCK>
__device__ void fuse_stream(const DevParams& P, const DevState& S, int b, int top_f, const float* ext,
                            double* sc, uint64_t* ky, uint32_t* ix) {
  const int tid = threadIdx.x;
  const int n = S.nbeam[b];
  const size_t gb = static_cast<size_t>(b) * P.K;
  const int F = (top_f <= 0 || top_f >= n) ? n : top_f;
  if (F < n) {
    if (tid < n) {
      sc[tid] = lse2(S.ab[gb + tid], S.anb[gb + tid]) + S.Lw[(gb + tid) * P.O];
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
  if (tid < F) {
    const int i = (F < n) ? static_cast<int>(ix[tid]) : tid;
    const size_t bi = gb + i;
    const uint32_t meta = S.meta[bi];
    const int nsub = (meta >> 8) & 0xFF;
    double L[kMaxSub];
    uint32_t h[kMaxSub];
#pragma unroll
    for (int j = 0; j < kMaxSub; ++j) {
      if (j < nsub) {
        h[j] = S.hist[bi * P.O + j];
        const double f = ext ? static_cast<double>(ext[static_cast<size_t>(tid) * P.O + j]) : S.arena[h[j]].sfus;
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
  fuse_stream<BLOCK>(P, S, b, P.fusion_top_f, nullptr, sc, ky, ix);
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
    S.ev_count[0] = 0;
    S.ev_count[1] = 0;
  }
  if (fin && P.fusion_source == 1 && P.fusion_interval > 0) fuse_stream<BLOCK>(P, S, b, 0, nullptr, sc, ky, ix);
  const int n = S.nbeam[b];
  const size_t gb = static_cast<size_t>(b) * P.K;
  bool ok = false;
  if (tid < n) {
    ok = !fin || S.node[gb + tid] == kRootNode;
    sc[tid] = ok ? lse2(S.ab[gb + tid], S.anb[gb + tid]) + S.Lw[(gb + tid) * P.O] : kNegInf;
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

hipError_t launch_frame(int block, const DevParams& P, const DevState& S, const float* logits,
                        const int32_t* lengths, int32_t B, int32_t Tc, int32_t tau, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_frame, B, P, S, logits, lengths, Tc, tau);
  return hipGetLastError();
}

hipError_t launch_ngram(int grid, const DevParams& P, const DevState& S, int32_t tau, hipStream_t st) {
  hipLaunchKernelGGL(k_ngram, dim3(grid), dim3(256), 0, st, P, S, tau);
  return hipGetLastError();
}

hipError_t launch_fusion(int block, const DevParams& P, const DevState& S, const int32_t* lengths, int32_t B,
                         int32_t tau, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_fusion, B, P, S, lengths, tau);
  return hipGetLastError();
}

hipError_t launch_output(int block, const DevParams& P, const DevState& S, const int32_t* lengths, int32_t B,
                         int32_t fin, int32_t* out_hyps, float* out_scores, hipStream_t st) {
  LB_DISPATCH_BLOCK(block, k_output, B, P, S, lengths, fin, out_hyps, out_scores);
  return hipGetLastError();
}

}  // namespace lb
