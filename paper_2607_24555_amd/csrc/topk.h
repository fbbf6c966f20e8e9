// Wave- and block-level top-k machinery shared by the selection kernels and the
// attention kernel that derives its page table in its prologue.
//
// Keys are uint32 order keys (larger key = larger share-averaged page mass);
// key 0 marks an empty slot.  A cut (T, take_eq) keeps every key > T and the
// first take_eq keys == T in position order, so ties go to the lower position.
#pragma once

#include "locks_internal.h"

namespace locks {

constexpr int kFastK = 128;  // largest k - 2 of the fast selection path


template <int C>
__device__ __forceinline__ int dpp(int v) {
  return __builtin_amdgcn_update_dpp(0, v, C, 0xF, 0xF, false);
}
// All-lane sums / extrema over the wave: quad xor, half-row and row mirrors,
// then the 16- and 32-lane swaps.
__device__ __forceinline__ int wave_sum_i(int v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = (int)p[0] + (int)p[1];
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __builtin_amdgcn_readfirstlane((int)r[0] + (int)r[1]);
}
__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
  v = max(v, (uint32_t)dpp<0xB1>((int)v));
  v = max(v, (uint32_t)dpp<0x4E>((int)v));
  v = max(v, (uint32_t)dpp<0x141>((int)v));
  v = max(v, (uint32_t)dpp<0x140>((int)v));
  auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = max((uint32_t)p[0], (uint32_t)p[1]);
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __builtin_amdgcn_readfirstlane(max((uint32_t)r[0], (uint32_t)r[1]));
}
__device__ __forceinline__ uint32_t wave_min_u(uint32_t v) {
  v = min(v, (uint32_t)dpp<0xB1>((int)v));
  v = min(v, (uint32_t)dpp<0x4E>((int)v));
  v = min(v, (uint32_t)dpp<0x141>((int)v));
  v = min(v, (uint32_t)dpp<0x140>((int)v));
  auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  v = min((uint32_t)p[0], (uint32_t)p[1]);
  auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __builtin_amdgcn_readfirstlane(min((uint32_t)r[0], (uint32_t)r[1]));
}
// Inclusive prefix sum over the wave: shifts inside 16-lane rows, then the
// last lane of row 0 / row 2 is added to row 1 / row 3 and lane 31 to rows 2-3.
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += dpp<0x111>(x);
  x += dpp<0x112>(x);
  x += dpp<0x114>(x);
  x += dpp<0x118>(x);
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);
  return x;
}

__device__ __forceinline__ uint64_t lanes_below() {
  const int l = threadIdx.x & 63;
  return l ? (~0ull >> (64 - l)) : 0ull;
}

// Cut of a top K: keep keys > T, and the first take_eq keys == T in position
// order.  Key 0 marks an empty slot.  lo_hint must satisfy
// count(key >= lo_hint) >= K (1 is always valid).  The bisection stops as soon
// as some threshold has exactly K keys at or above it.
struct WaveCut {
  uint32_t T;
  int take_eq;
};

// An empty asm that consumes v: the load producing v can no longer be moved
// under a branch, where it would be waited for before the next one is issued.
template <typename T>
__device__ __forceinline__ void pin(T& v) {
  asm volatile("" : "+v"(v));
}

// Block-cooperative cut over NW waves holding NK keys per lane.  Every wave
// takes the same decisions from per-wave ballot counts exchanged through LDS,
// one barrier per bisection step (the count slots are double-buffered).
template <int NW>
struct CutLds {
  int cnt[2][NW];
  uint32_t mn[NW], mx[NW];
  int eq[NW], gt[NW];
};

template <int NK>
__device__ __forceinline__ int wave_count_ge(const uint32_t (&key)[NK], uint32_t t) {
  int c = 0;
#pragma unroll
  for (int u = 0; u < NK; ++u) c += __popcll(__ballot(key[u] >= t));
  return c;
}

template <int NK, int NW>
__device__ __forceinline__ WaveCut block_cut(const uint32_t (&key)[NK], int K, uint32_t lo_hint,
                                             CutLds<NW>& L) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint32_t kmx = 0u, kmn = 0xffffffffu;
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    kmx = max(kmx, key[u]);
    kmn = min(kmn, key[u] ? key[u] : 0xffffffffu);
  }
  const int nz = wave_count_ge(key, 1u);
  kmx = wave_max_u(kmx);
  kmn = wave_min_u(kmn);
  if (lane == 0) { L.cnt[0][wave] = nz; L.mn[wave] = kmn; L.mx[wave] = kmx; }
  __syncthreads();
  int total = 0;
  uint32_t lo = 0xffffffffu, hi = 0u;
#pragma unroll
  for (int w = 0; w < NW; ++w) { total += L.cnt[0][w]; lo = min(lo, L.mn[w]); hi = max(hi, L.mx[w]); }
  if (total <= K) return WaveCut{1u, 1 << 30};
  lo = max(lo, lo_hint);
  int par = 1;
  while (lo < hi) {
    const uint32_t mid = lo + (uint32_t)((((uint64_t)hi - lo) + 1) >> 1);
    const int cw = wave_count_ge(key, mid);
    if (lane == 0) L.cnt[par][wave] = cw;
    __syncthreads();
    int c = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) c += L.cnt[par][w];
    par ^= 1;
    if (c == K) { lo = mid; break; }
    if (c > K) lo = mid; else hi = mid - 1;
  }
  const int gw = lo == 0xffffffffu ? 0 : wave_count_ge(key, lo + 1);
  if (lane == 0) L.cnt[par][wave] = gw;
  __syncthreads();
  int c = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) c += L.cnt[par][w];
  return WaveCut{lo, K - c};
}

// Calls f(u, slot) for every kept element (slot = rank in block position
// order); returns the number kept.  Contains one barrier.
template <int NK, int NW, typename F>
__device__ __forceinline__ int block_emit(const uint32_t (&key)[NK], WaveCut cut, CutLds<NW>& L,
                                          F f) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int eq_w = 0, gt_w = 0;
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    eq_w += __popcll(__ballot(key[u] != 0u && key[u] == cut.T));
    gt_w += __popcll(__ballot(key[u] != 0u && key[u] > cut.T));
  }
  if (lane == 0) { L.eq[wave] = eq_w; L.gt[wave] = gt_w; }
  __syncthreads();
  int eq_base = 0, base = 0, total = 0;
  // kept by each wave: its keys > T plus its share of the first take_eq keys == T
  int eq_seen = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int e = L.eq[w];
    const int kept = L.gt[w] + min(max(cut.take_eq - eq_seen, 0), e);
    if (w < wave) { base += kept; eq_base += e; }
    total += kept;
    eq_seen += e;
  }
  const uint64_t lt = lanes_below();
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    const bool nz = key[u] != 0u;
    const bool eq = nz && key[u] == cut.T;
    const uint64_t em = __ballot(eq);
    const int er = eq_base + __popcll(em & lt);
    eq_base += __popcll(em);
    const bool keep = (nz && key[u] > cut.T) || (eq && er < cut.take_eq);
    const uint64_t km = __ballot(keep);
    if (keep) f(u, base + __popcll(km & lt));
    base += __popcll(km);
  }
  return total;
}

// Histogram cut.  Bins measure how far a key lies below the block maximum M,
// in 1/32 of a log2 unit (bin 0 holds M; the last bin also takes everything
// further down).  The prefix over bins locates the boundary bin b*: every key
// in a lower bin is kept, and only the few keys of b* are ranked exactly.  When
// b* holds more than kBoundaryMax keys, bisection over b*'s key range decides.
constexpr int kBins = 1024;
constexpr float kBinsPerUnit = 32.0f;
constexpr int kBoundaryMax = 64;

template <int NW>
struct HistLds {
  int hist[kBins];
  uint32_t mx[NW];
  int wtot[NW];
  int nb;                      // keys in the boundary bin
  uint32_t bmin;               // smallest key in the boundary bin
  int bstar, need;             // boundary bin, keys to take from it
  uint32_t bkey[kBoundaryMax];
  int bpos[kBoundaryMax];
  WaveCut cut;
};

__device__ __forceinline__ int key_bin(uint32_t key, float Mf) {
  const float d = (Mf - order_key_f32(key)) * kBinsPerUnit;
  return (int)fminf(fmaxf(d, 0.0f), (float)(kBins - 1));
}

template <int NK, int NW>
__device__ __forceinline__ WaveCut block_hist_cut(const uint32_t (&key)[NK], int K, HistLds<NW>& H,
                                                  CutLds<NW>& L) {
  constexpr int kT = 64 * NW, kPer = kBins / kT;
  static_assert(kBins % kT == 0, "bins per thread");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // 1. block maximum and candidate count; clear the histogram
#pragma unroll
  for (int b = 0; b < kPer; ++b) H.hist[tid * kPer + b] = 0;
  if (tid == 0) { H.nb = 0; H.bmin = 0xffffffffu; H.bstar = kBins - 1; H.need = 1; }
  uint32_t kmx = 0u;
#pragma unroll
  for (int u = 0; u < NK; ++u) kmx = max(kmx, key[u]);
  const int nz = wave_count_ge(key, 1u);
  kmx = wave_max_u(kmx);
  if (lane == 0) { H.mx[wave] = kmx; H.wtot[wave] = nz; }
  __syncthreads();
  uint32_t M = 0u;
  int total = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) { M = max(M, H.mx[w]); total += H.wtot[w]; }
  if (total <= K) return WaveCut{1u, 1 << 30};
  const float Mf = order_key_f32(M);
  // 2. histogram
  int bin[NK];
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    bin[u] = key[u] ? key_bin(key[u], Mf) : -1;
    if (key[u]) atomicAdd(&H.hist[bin[u]], 1);
  }
  __syncthreads();
  // 3. boundary bin: first bin where the running count reaches K
  int c = 0;
#pragma unroll
  for (int b = 0; b < kPer; ++b) c += H.hist[tid * kPer + b];
  int incl = wave_incl_scan(c);
  if (lane == 63) H.wtot[wave] = incl;
  __syncthreads();
  int before = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) before += w < wave ? H.wtot[w] : 0;
  incl += before;
  if (incl >= K && incl - c < K) {
    int run = incl - c, b = 0;
    while (b < kPer - 1 && run + H.hist[tid * kPer + b] < K) run += H.hist[tid * kPer + b++];
    H.bstar = tid * kPer + b;
    H.need = K - run;
  }
  __syncthreads();
  // 4. collect the boundary bin (position order is rebuilt by ranking)
  const int bstar = H.bstar;
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    if (bin[u] == bstar) {
      const int slot = atomicAdd(&H.nb, 1);
      atomicMin(&H.bmin, key[u]);
      if (slot < kBoundaryMax) {
        H.bkey[slot] = key[u];
        H.bpos[slot] = (wave * NK + u) * 64 + lane;
      }
    }
  }
  __syncthreads();
  const int nb = H.nb;
  if (nb > kBoundaryMax) return block_cut<NK, NW>(key, K, H.bmin, L);
  // 5. wave 0 ranks the boundary keys: (key desc, position asc)
  if (wave == 0) {
    const bool have = lane < nb;
    const uint32_t mk = have ? H.bkey[lane] : 0u;
    const int mp_ = have ? H.bpos[lane] : 0x7fffffff;
    int rank = 0;
    for (int j = 0; j < nb; ++j) {
      const uint32_t kj = (uint32_t)__builtin_amdgcn_readlane((int)mk, j);
      const int pj = __builtin_amdgcn_readlane(mp_, j);
      rank += (kj > mk) || (kj == mk && pj < mp_);
    }
    const int need = H.need;
    const uint64_t at = __ballot(have && rank == need - 1);
    const uint32_t T = __shfl(mk, (int)__builtin_ctzll(at), 64);
    const int gt = __popcll(__ballot(have && mk > T));
    if (lane == 0) H.cut = WaveCut{T, need - gt};
  }
  __syncthreads();
  return H.cut;
}

// Survivors compacted in position order for a cheap final cut.
constexpr int kCompactNK = 2;  // keys per lane after compaction (512 per 4-wave block)

template <int NW>
struct MergeLds {
  CutLds<NW> L;
  HistLds<NW> H;
  uint32_t lo;
  int wcnt[NW];
  uint32_t ck[64 * NW * kCompactNK];
  int32_t ci[64 * NW * kCompactNK];
};

// Page table of one (sequence, KV head) from its chunk survivors: s_tab[0] = 0
// (sink), s_tab[1 .. k-2] = the k - 2 best candidates ascending, s_tab[k-1] = n-1
// (recent); with n <= k every page, then -1.  ck / ci hold `used` rows of K
// survivors (page order inside a row, rows in page order); thr[c] is a lower
// bound of the sequence-wide cut.  Survivors at or above the best lower bound
// are compacted (in order) and cut there; if more than 64 * NW * kCompactNK
// remain, the cut runs over all of them in registers.  Called by every thread
// of an NW-wave block; requires used * K <= 64 * NW * NK; ends with a barrier.
template <int NK, int NW>
__device__ __forceinline__ void merge_table(int k, int n, int used, const uint32_t* __restrict__ ck,
                                            const int32_t* __restrict__ ci,
                                            const uint32_t* __restrict__ thr, int32_t* s_tab,
                                            MergeLds<NW>& M) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int K = k - 2;
  if (n <= k) {
    for (int t = tid; t < k; t += 64 * NW) s_tab[t] = t < n ? t : -1;
  } else {
    if (K > 0) {
      const int N = used * K;
      const int e0 = wave * (64 * NK) + lane;
      uint32_t key[NK];
      int32_t idx[NK];
#pragma unroll
      for (int u = 0; u < NK; ++u) {
        const int e = min(e0 + u * 64, N - 1);
        key[u] = ck[e];
        idx[u] = ci[e];
      }
      if (wave == 0) {
        uint32_t lo = 1u;
        for (int c = lane; c < used; c += 64) lo = max(lo, thr[c]);
        lo = wave_max_u(lo);
        if (lane == 0) M.lo = lo;
      }
#pragma unroll
      for (int u = 0; u < NK; ++u) pin(key[u]);
      __syncthreads();
      // keys below the best chunk cut cannot reach the sequence-wide top K
      const uint32_t lo = M.lo;
#pragma unroll
      for (int u = 0; u < NK; ++u) key[u] = (e0 + u * 64 < N && key[u] >= lo) ? key[u] : 0u;
      const int live = wave_count_ge(key, 1u);
      if (lane == 0) M.wcnt[wave] = live;
      __syncthreads();
      int off = 0, total = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        off += w < wave ? M.wcnt[w] : 0;
        total += M.wcnt[w];
      }
      constexpr int kCap = 64 * NW * kCompactNK;
      if (total <= kCap) {
        const uint64_t lt = lanes_below();
#pragma unroll
        for (int u = 0; u < NK; ++u) {
          const uint64_t m = __ballot(key[u] != 0u);
          if (key[u]) {
            const int slot = off + __popcll(m & lt);
            M.ck[slot] = key[u];
            M.ci[slot] = idx[u];
          }
          off += __popcll(m);
        }
        __syncthreads();
        uint32_t k2[kCompactNK];
        int e2[kCompactNK];
#pragma unroll
        for (int u = 0; u < kCompactNK; ++u) {
          e2[u] = (wave * kCompactNK + u) * 64 + lane;
          k2[u] = e2[u] < total ? M.ck[e2[u]] : 0u;
        }
        const WaveCut cut = block_hist_cut<kCompactNK, NW>(k2, K, M.H, M.L);
        block_emit<kCompactNK, NW>(k2, cut, M.L, [&](int u, int slot) { s_tab[1 + slot] = M.ci[e2[u]]; });
      } else {
        const WaveCut cut = block_hist_cut<NK, NW>(key, K, M.H, M.L);
        block_emit<NK, NW>(key, cut, M.L, [&](int u, int slot) { s_tab[1 + slot] = idx[u]; });
      }
    }
    if (tid == 0) {
      s_tab[0] = 0;
      s_tab[k - 1] = n - 1;
    }
  }
  __syncthreads();
}

}  // namespace locks
