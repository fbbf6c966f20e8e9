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

// Block-wide sum and exclusive scan of per-thread ints through double-buffered
// per-wave slots (par alternates between consecutive calls).
template <int NW>
struct BlockLds {
  int v[2][NW];
  uint32_t mx[NW];
};

template <int NW>
__device__ __forceinline__ int block_total(int v, BlockLds<NW>& B, int par) {
  const int w = wave_sum_i(v);
  if ((threadIdx.x & 63) == 0) B.v[par][threadIdx.x >> 6] = w;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) t += B.v[par][i];
  return t;
}

template <int NW>
__device__ __forceinline__ int block_excl(int v, BlockLds<NW>& B, int par) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int incl = wave_incl_scan(v);
  if (lane == 63) B.v[par][wave] = incl;
  __syncthreads();
  int before = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) before += i < wave ? B.v[par][i] : 0;
  return before + incl - v;
}

// Exact top K of keys[0 .. N) in global memory (0 = no candidate), ties to the
// lower position; the kept positions go to out[0 .. K) in ascending order.
// lo_hint must not exceed the K-th largest key.  Each thread owns a contiguous
// run of keys and re-reads it in every bisection step, so this is the slow,
// general path.  Called by every thread; ends with a barrier.
template <int NW>
__device__ void exact_cut_global(const uint32_t* __restrict__ keys, int N, int K,
                                 uint32_t lo_hint, int32_t* out, BlockLds<NW>& B) {
  constexpr int kT = 64 * NW;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int P = (N + kT - 1) / kT;
  const int e0 = min(N, tid * P), e1 = min(N, e0 + P);
  uint32_t kmx = 0u;
  int nz = 0;
  for (int e = e0; e < e1; ++e) {
    const uint32_t v = keys[e];
    kmx = max(kmx, v);
    nz += v != 0u;
  }
  kmx = wave_max_u(kmx);
  if (lane == 0) B.mx[wave] = kmx;
  int par = 0;
  const int total = block_total<NW>(nz, B, par);
  par ^= 1;
  uint32_t hi = 0u;
#pragma unroll
  for (int w = 0; w < NW; ++w) hi = max(hi, B.mx[w]);
  uint32_t T = 1u;
  int take_eq = 1 << 30;
  if (total > K) {
    uint32_t lo = max(lo_hint, 1u);  // invariant: count(key >= lo) >= K
    while (lo < hi) {
      const uint32_t mid = lo + (uint32_t)((((uint64_t)hi - lo) + 1) >> 1);
      int c = 0;
      for (int e = e0; e < e1; ++e) c += keys[e] >= mid;
      if (block_total<NW>(c, B, par) >= K) lo = mid; else hi = mid - 1;
      par ^= 1;
    }
    T = lo;
    int c = 0;
    for (int e = e0; e < e1; ++e) c += keys[e] > T;
    take_eq = K - block_total<NW>(c, B, par);
    par ^= 1;
  }
  int eq = 0;
  for (int e = e0; e < e1; ++e) {
    const uint32_t v = keys[e];
    eq += v != 0u && v == T;
  }
  const int eq_before = block_excl<NW>(eq, B, par);
  par ^= 1;
  int kept = 0;
  {
    int r = eq_before;
    for (int e = e0; e < e1; ++e) {
      const uint32_t v = keys[e];
      const bool is_eq = v != 0u && v == T;
      kept += (v != 0u && v > T) || (is_eq && r < take_eq);
      r += is_eq;
    }
  }
  int pos = block_excl<NW>(kept, B, par);
  {
    int r = eq_before;
    for (int e = e0; e < e1; ++e) {
      const uint32_t v = keys[e];
      const bool is_eq = v != 0u && v == T;
      if ((v != 0u && v > T) || (is_eq && r < take_eq)) out[pos++] = e;
      r += is_eq;
    }
  }
  __syncthreads();
}

template <int NW>
struct UnionLds {
  CutLds<NW> L;
  HistLds<NW> H;
  BlockLds<NW> B;
  int fallback;
};

// The survivor registers of the union, loaded before the sequence length is known
// (rows x width entries of which the first used x width are valid).
template <int NK>
struct UnionRegs {
  uint32_t key[NK];
  int32_t idx[NK], blk[NK];
  uint32_t tr[4];
};

template <int NK, int NW>
__device__ __forceinline__ void union_load(UnionRegs<NK>& R, int rows, int width,
                                           const uint32_t* __restrict__ ck,
                                           const int32_t* __restrict__ ci,
                                           const int32_t* __restrict__ cb,
                                           const uint32_t* __restrict__ sat) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int N = rows * width;
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    const int e = (wave * NK + u) * 64 + lane;
    const int ec = e < N ? e : N - 1;
    R.key[u] = ck[ec];
    R.idx[u] = ci[ec];
    R.blk[u] = cb[ec];
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) R.tr[u] = sat[min(lane + 64 * u, rows - 1)];
}

// Page table of one (sequence, KV head) with n pages and budget k:
// s_tab[0] = 0 (sink), s_tab[1 .. k-2] = the k - 2 candidates of largest key in
// ascending page order, s_tab[k-1] = n - 1 (recent); with n <= k every page,
// then -1.  s_blk[t] is the physical block of entry t (-1 for padding).
// Inputs: `used` rows of `width` chunk survivors (key, page, block; page order
// inside a row, rows in page order, key 0 = empty slot); sat[c] = the key at
// which chunk c was truncated (0 if it kept every candidate); keys = every
// page's key for pages 0 .. n - 2 (0 for the sink).  The cut over the
// survivors is exact unless some chunk was
// truncated at or above it; then the whole sequence is cut again from keys.
// Requires used * width <= 64 * NW * NK and used <= 256.  Called by every
// thread of an NW-wave block, with R from union_load; ends with a barrier.
template <int NK, int NW>
__device__ __forceinline__ void union_table_from(UnionRegs<NK>& R, int k, int n, int used,
                                                 int width, const uint32_t* __restrict__ keys,
                                                 const int32_t* __restrict__ pt_row,
                                                 int32_t* s_tab, int32_t* s_blk,
                                                 UnionLds<NW>& U) {
  constexpr int kT = 64 * NW;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int K = k - 2;
  if (n <= k) {
    for (int t = tid; t < k; t += kT) {
      s_tab[t] = t < n ? t : -1;
      s_blk[t] = t < n ? pt_row[t] : -1;
    }
    __syncthreads();
    return;
  }
  if (tid == 0) {
    s_tab[0] = 0;
    s_blk[0] = pt_row[0];
    s_tab[k - 1] = n - 1;
    s_blk[k - 1] = pt_row[n - 1];
  }
  if (K > 0) {
    const int N = used * width;
#pragma unroll
    for (int u = 0; u < NK; ++u) R.key[u] = (wave * NK + u) * 64 + lane < N ? R.key[u] : 0u;
    const WaveCut cut = block_hist_cut<NK, NW>(R.key, K, U.H, U.L);
    if (wave == 0) {
      bool bad = false;
#pragma unroll
      for (int u = 0; u < 4; ++u) bad |= lane + 64 * u < used && R.tr[u] != 0u && R.tr[u] >= cut.T;
      const bool any = __ballot(bad) != 0ull;
      if (lane == 0) U.fallback = any;
    }
    __syncthreads();
    if (!U.fallback) {
      block_emit<NK, NW>(R.key, cut, U.L, [&](int u, int slot) {
        s_tab[1 + slot] = R.idx[u];
        s_blk[1 + slot] = R.blk[u];
      });
    } else {
      exact_cut_global<NW>(keys, n - 1, K, cut.T, s_tab + 1, U.B);  // pages 0 .. n - 2
      for (int t = 1 + tid; t <= K; t += kT) s_blk[t] = pt_row[s_tab[t]];
    }
  }
  __syncthreads();
}

// union_load and union_table_from in one call.
template <int NK, int NW>
__device__ __forceinline__ void union_table(int k, int n, int used, int width, const uint32_t* __restrict__ ck,
                            const int32_t* __restrict__ ci, const int32_t* __restrict__ cb,
                            const uint32_t* __restrict__ sat, const uint32_t* __restrict__ keys,
                            const int32_t* __restrict__ pt_row, int32_t* s_tab, int32_t* s_blk,
                            UnionLds<NW>& U) {
  UnionRegs<NK> R;
  if (n > k && used > 0) union_load<NK, NW>(R, used, width, ck, ci, cb, sat);
  union_table_from<NK, NW>(R, k, n, used, width, keys, pt_row, s_tab, s_blk, U);
}

}  // namespace locks
