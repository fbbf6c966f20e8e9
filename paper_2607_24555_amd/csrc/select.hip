// Share-average combine and shared top-k table (Sec. 4 "Score"; Cor.
// "Group-shared selection"; App. E "union table").
//
// Two kernels:
//  select_chunk_kernel, grid (chunk of kSelChunk pages, KV head, sequence):
//   * reduces the scan blocks' partials into lz2_g = log2 Z_g;
//   * scores the candidate pages of its chunk (neither page 0 nor the most recent
//     page):  log2 mbar_j + log2 G = log2 sum_g 2^(s2_j(q_g) - lz2_g), as an
//     order-preserving uint32 key (key 0 marks "no candidate");
//   * keeps the chunk's top (k-2) keys: a bisection over the key space finds T,
//     the (k-2)-th largest key; an ordered compaction keeps every key above T and
//     the lowest-index keys equal to T (ties go to the lower page index), so the
//     survivors come out in ascending page order.
//  select_merge_kernel, one block per (sequence, KV head): the same selection over
//   all chunks' survivors, plus page 0 and the most recent page, written as the
//   ascending table, and the selected pages' hat s gathered for every head.
// Each thread owns a contiguous run of pages (or survivors) held in registers;
// block counts use wave ballots and the ordered compaction two exclusive scans.
#include "locks_internal.h"
#include "topk.h"

namespace locks {
namespace {

constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kPerThread = kSelChunk / kSelThreads;  // contiguous pages per thread
constexpr int kMergeRegs = 32;                       // survivors per thread in registers
constexpr float kLog2e = 1.4426950408889634f;

struct Red {
  int v[2][kSelWaves];
  int sc[2][kSelWaves];
  uint32_t mx[kSelWaves], mn[kSelWaves];
};

// Block sum of small non-negative per-thread counts (< 2^bits), via wave ballots.
__device__ __forceinline__ int block_count(int v, int bits, Red& r, int par) {
  int w = 0;
  for (int b = 0; b < bits; ++b) w += __popcll(__ballot((v >> b) & 1)) << b;
  if ((threadIdx.x & 63) == 0) r.v[par][threadIdx.x >> 6] = w;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int i = 0; i < kSelWaves; ++i) t += r.v[par][i];
  return t;
}

// Exclusive block scan of per-thread ints in thread order, and the total.
__device__ __forceinline__ int block_excl_scan(int v, Red& r, int par, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) r.sc[par][wave] = x;
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kSelWaves; ++i) {
    before += i < wave ? r.sc[par][i] : 0;
    tot += r.sc[par][i];
  }
  *total = tot;
  return before + x - v;
}

__device__ __forceinline__ void block_minmax(uint32_t& mn, uint32_t& mx, Red& r) {
  for (int o = 32; o > 0; o >>= 1) {
    mx = max(mx, (uint32_t)__shfl_xor((int)mx, o, 64));
    mn = min(mn, (uint32_t)__shfl_xor((int)mn, o, 64));
  }
  if ((threadIdx.x & 63) == 0) { r.mx[threadIdx.x >> 6] = mx; r.mn[threadIdx.x >> 6] = mn; }
  __syncthreads();
  mx = 0u;
  mn = 0xffffffffu;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) { mx = max(mx, r.mx[w]); mn = min(mn, r.mn[w]); }
  __syncthreads();
}

__device__ __forceinline__ int bit_length(int x) { return x > 0 ? 32 - __clz(x) : 0; }

// Flags in sel[] the K largest of the keys held by the block (NK per thread,
// key 0 = empty, thread-major order = ascending page order).  Ties at the
// threshold keep the lowest positions.  Returns this thread's kept count.
template <int NK>
__device__ __forceinline__ int select_top(const uint32_t (&key)[NK], int K, bool (&sel)[NK],
                                          Red& red) {
  int local = 0;
  uint32_t kmx = 0u, kmn = 0xffffffffu;
#pragma unroll
  for (int u = 0; u < NK; ++u)
    if (key[u]) { ++local; kmx = max(kmx, key[u]); kmn = min(kmn, key[u]); }
  const int bits = bit_length(NK);
  int par = 0;
  const int n_cand = block_count(local, bits, red, par);
  par ^= 1;
  uint32_t T = 1u;
  int take_eq = 1 << 30;
  if (n_cand > K) {
    block_minmax(kmn, kmx, red);
    uint32_t lo = kmn, hi = kmx;  // invariant: #{key >= lo} >= K
    while (lo < hi) {
      const uint32_t mid = lo + (uint32_t)((((uint64_t)hi - lo) + 1) >> 1);
      int c = 0;
#pragma unroll
      for (int u = 0; u < NK; ++u) c += key[u] >= mid;
      if (block_count(c, bits, red, par) >= K) lo = mid; else hi = mid - 1;
      par ^= 1;
    }
    T = lo;
    int c = 0;
#pragma unroll
    for (int u = 0; u < NK; ++u) c += key[u] > T;
    take_eq = K - block_count(c, bits, red, par);
  }
  int eq_l = 0;
#pragma unroll
  for (int u = 0; u < NK; ++u) eq_l += key[u] != 0u && key[u] == T;
  int tot;
  int eq_rank = block_excl_scan(eq_l, red, 0, &tot);
  int kept = 0;
#pragma unroll
  for (int u = 0; u < NK; ++u) {
    const bool eq = key[u] != 0u && key[u] == T;
    sel[u] = (key[u] != 0u && key[u] > T) || (eq && eq_rank < take_eq);
    eq_rank += eq;
    kept += sel[u];
  }
  return kept;
}

__global__ __launch_bounds__(kSelThreads) void select_chunk_kernel(
    int H_q, int H_kv, int k, int n_chunks, int pgsz, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ s_hat, SHatLayout lay, const float2* __restrict__ partials,
    int n_parts, uint32_t* __restrict__ cand_key, int32_t* __restrict__ cand_idx) {
  __shared__ Red red;
  __shared__ float s_lz2[16];
  const int chunk = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int tid = threadIdx.x;
  const int L = seq_lens[s];
  const int n = (L + pgsz - 1) / pgsz;
  const int G = H_q / H_kv;
  const int K = k - 2;
  const int p0 = chunk * kSelChunk;
  if (K <= 0 || n <= k || p0 > n - 2) return;  // uniform: nothing to rank in this chunk
  const long row0 = (long)s * H_q + (long)h * G;

  // ---- log2 Z_g from the scan blocks' (max, sum 2^x) partials, 16 threads per head
  {
    const int g = tid >> 4, sub = tid & 15;
    const float2* pp = partials + (row0 + (g < G ? g : 0)) * n_parts;
    float m = -INFINITY, l = 0.0f;
    for (int base = 0; base < n_parts; base += 16 * 8) {
      float2 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = base + sub + 16 * u;
        v[u] = pp[t < n_parts ? t : 0];
        if (!(g < G && t < n_parts)) v[u] = make_float2(-INFINITY, 0.0f);
      }
      float mm = m;
#pragma unroll
      for (int u = 0; u < 8; ++u) mm = fmaxf(mm, v[u].x);
      float ll = (m > -INFINITY) ? l * __builtin_amdgcn_exp2f(m - mm) : 0.0f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        ll += (v[u].y > 0.0f) ? v[u].y * __builtin_amdgcn_exp2f(v[u].x - mm) : 0.0f;
      m = mm;
      l = ll;
    }
    for (int o = 8; o > 0; o >>= 1) {
      const float om = __shfl_xor(m, o, 64), ol = __shfl_xor(l, o, 64);
      const float mm = fmaxf(m, om);
      l = (mm > -INFINITY) ? l * __builtin_amdgcn_exp2f(m - mm) + ol * __builtin_amdgcn_exp2f(om - mm)
                           : 0.0f;
      m = mm;
    }
    if (g < G && sub == 0) s_lz2[g] = m + __builtin_amdgcn_logf(l);
    __syncthreads();
  }

  // ---- keys of this thread's kPerThread consecutive pages (unconditional loads)
  uint32_t key[kPerThread];
  {
    const int j0 = p0 + kPerThread * tid;
    const float* base = s_hat + lay.base(s, h);
    float sv[kPerThread][kMaxGroup];
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      const long j = min(max(j0 + u, 1), n - 2);
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g) sv[u][g] = base[j * lay.page + (long)(g < G ? g : 0) * lay.head];
    }
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      float m = -INFINITY;
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g)
        if (g < G) m = fmaxf(m, sv[u][g] * kLog2e - s_lz2[g]);
      float sum = 0.0f;
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g)
        if (g < G) sum += __builtin_amdgcn_exp2f(sv[u][g] * kLog2e - s_lz2[g] - m);
      const int j = j0 + u;
      key[u] = (j >= 1 && j <= n - 2) ? max(1u, f32_order_key(m + __builtin_amdgcn_logf(sum))) : 0u;
    }
  }
  bool sel[kPerThread];
  const int kept = select_top<kPerThread>(key, K, sel, red);
  int tot;
  int pos = block_excl_scan(kept, red, 1, &tot);
  const long row = (((long)s * H_kv + h) * n_chunks + chunk) * K;
#pragma unroll
  for (int u = 0; u < kPerThread; ++u)
    if (sel[u]) {
      cand_key[row + pos] = key[u];
      cand_idx[row + pos] = p0 + kPerThread * tid + u;
      ++pos;
    }
  for (int t = tot + tid; t < K; t += kSelThreads) {
    cand_key[row + t] = 0u;
    cand_idx[row + t] = -1;
  }
}

// Final selection for one (sequence, KV head).  kRegs: every thread holds its
// run of survivors in registers (at most kMergeRegs each); otherwise the run is
// re-read from global memory in every pass.
template <bool kRegs>
__device__ void merge_select(int N, int K, const uint32_t* __restrict__ gk,
                             const int32_t* __restrict__ gi, int32_t* ids, Red& red) {
  const int tid = threadIdx.x;
  if (kRegs) {
    const int P = (N + kSelThreads - 1) / kSelThreads;  // <= kMergeRegs
    const int e0 = min(N, tid * P);
    uint32_t key[kMergeRegs];
#pragma unroll
    for (int u = 0; u < kMergeRegs; ++u) {
      const int e = e0 + u;
      const uint32_t v = gk[min(e, N - 1)];
      key[u] = (u < P && e < N) ? v : 0u;
    }
    bool sel[kMergeRegs];
    const int kept = select_top<kMergeRegs>(key, K, sel, red);
    int tot;
    int pos = 1 + block_excl_scan(kept, red, 1, &tot);
#pragma unroll
    for (int u = 0; u < kMergeRegs; ++u)
      if (sel[u]) ids[pos++] = gi[e0 + u];
  } else {
    // survivors in groups of kSelThreads * 4, each pass re-reading global memory
    const int P = (N + kSelThreads - 1) / kSelThreads;
    const int e0 = min(N, tid * P), e1 = min(N, e0 + P);
    uint32_t kmx = 0u, kmn = 0xffffffffu;
    for (int e = e0; e < e1; ++e) {
      const uint32_t v = gk[e];
      if (v) { kmx = max(kmx, v); kmn = min(kmn, v); }
    }
    block_minmax(kmn, kmx, red);
    const int bits = bit_length(P);
    int par = 0;
    uint32_t lo = kmn, hi = kmx;
    while (lo < hi) {
      const uint32_t mid = lo + (uint32_t)((((uint64_t)hi - lo) + 1) >> 1);
      int c = 0;
      for (int e = e0; e < e1; ++e) c += gk[e] >= mid;
      if (block_count(c, bits, red, par) >= K) lo = mid; else hi = mid - 1;
      par ^= 1;
    }
    const uint32_t T = lo;
    int c = 0, eq_l = 0;
    for (int e = e0; e < e1; ++e) {
      const uint32_t v = gk[e];
      c += v > T;
      eq_l += v != 0u && v == T;
    }
    const int take_eq = K - block_count(c, bits, red, par);
    int tot;
    int eq_rank = block_excl_scan(eq_l, red, 0, &tot);
    int kept = 0;
    {
      int r = eq_rank;
      for (int e = e0; e < e1; ++e) {
        const uint32_t v = gk[e];
        const bool eq = v != 0u && v == T;
        kept += (v != 0u && v > T) || (eq && r < take_eq);
        r += eq;
      }
    }
    int pos = 1 + block_excl_scan(kept, red, 1, &tot);
    for (int e = e0; e < e1; ++e) {
      const uint32_t v = gk[e];
      const bool eq = v != 0u && v == T;
      if ((v != 0u && v > T) || (eq && eq_rank < take_eq)) ids[pos++] = gi[e];
      eq_rank += eq;
    }
  }
}

__global__ __launch_bounds__(kSelThreads) void select_merge_kernel(
    int H_q, int H_kv, int k, int n_chunks, int pgsz, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ s_hat, SHatLayout lay, const uint32_t* __restrict__ cand_key,
    const int32_t* __restrict__ cand_idx, int32_t* __restrict__ out_ids,
    float* __restrict__ out_sel_lse) {
  __shared__ Red red;
  const int h = blockIdx.x, s = blockIdx.y;
  const int tid = threadIdx.x;
  const int L = seq_lens[s];
  const int n = (L + pgsz - 1) / pgsz;
  const int n_c = L / pgsz;
  const int G = H_q / H_kv;
  const int K = k - 2;
  const long row0 = (long)s * H_q + (long)h * G;
  int32_t* ids = out_ids + ((long)s * H_kv + h) * k;
  if (n <= k) {
    for (int t = tid; t < k; t += kSelThreads) ids[t] = t < n ? t : -1;
  } else {
    const int used = (n - 2) / kSelChunk + 1;  // chunks that hold candidates (pages 1..n-2)
    const int N = used * K;
    const long base = ((long)s * H_kv + h) * n_chunks * K;
    if (K > 0 && N <= kSelThreads * kMergeRegs)
      merge_select<true>(N, K, cand_key + base, cand_idx + base, ids, red);
    else if (K > 0)
      merge_select<false>(N, K, cand_key + base, cand_idx + base, ids, red);
    if (tid == 0) { ids[0] = 0; ids[k - 1] = n - 1; }
  }
  __syncthreads();
  const float* sb = s_hat + lay.base(s, h);
  for (int e = tid; e < G * k; e += kSelThreads) {
    const int g = e / k, t = e % k;
    const int id = ids[t];
    out_sel_lse[(row0 + g) * k + t] =
        (id >= 0 && id < n_c) ? sb[(long)id * lay.page + (long)g * lay.head] : __int_as_float(0x7fc00000);
  }
}

// ---------------------------------------------------------------------------
// Fast path (k - 2 <= kFastK, at most kUnionCap / 8 chunks of kFastChunk pages).
// Two kernels:
//   chunk - one 4-wave block per kFastChunk pages of a (sequence, KV head): Z_g
//           from the scan partials, the share-averaged key of every page
//           (also written out in full), and the
//           chunk's top `width` keys with their pages and physical blocks, by a
//           histogram cut; the key at which the chunk was truncated (0 if it
//           kept every candidate);
//   merge - one block per (sequence, KV head): union_table over the chunk
//           survivors, the estimated page LSEs of the table.
// The fused decode step runs the merge inside the attention kernel instead.
// Keys live in registers wave-major, then register-major: element u of lane l
// in wave w has position (w * NK + u) * 64 + l, which is page order, so ties
// resolve to lower pages.
// ---------------------------------------------------------------------------

constexpr int kChunkThreads = 256;
constexpr int kChunkWaves = kChunkThreads / 64;
constexpr int kChunkNK = kFastChunk / kChunkThreads;  // keys per lane in a chunk (2)

// xor-shuffle inside groups of four lanes (DPP quad permutation).
template <int O>
__device__ __forceinline__ float quad_xor(float v) {
  return __int_as_float(dpp<O == 1 ? 0xB1 : 0x4E>(__float_as_int(v)));
}

__device__ __forceinline__ uint32_t page_key(float m, float sum) {
  return max(1u, f32_order_key(m + __builtin_amdgcn_logf(sum)));
}

template <int kG>  // G when one page's G scores are contiguous (4, 8, 16), else 0
__global__ __launch_bounds__(kChunkThreads) void select_chunk_keys_kernel(
    int H_q, int H_kv, int k, int width, int max_pages, int pgsz,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ page_table,
    const float* __restrict__ s_hat, SHatLayout lay, const float2* __restrict__ partials,
    int n_parts, SelectBufs sb, int n_rows, const float2* __restrict__ part_x,
    const int32_t* __restrict__ sl_scan) {
  constexpr int kT = kChunkThreads;
  __shared__ float s_lz2[kMaxGroup];
  __shared__ __align__(16) uint32_t sk[kFastChunk];
  __shared__ CutLds<kChunkWaves> L;
  __shared__ HistLds<kChunkWaves> HL;
  const int chunk = blockIdx.x, h = blockIdx.y, s = blockIdx.z, tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int Ls = seq_lens[s];  // used after the loads below are issued
  const int G = H_q / H_kv;
  const int K = k - 2;
  const int p0 = chunk * kFastChunk;
  if (K <= 0) return;
  const long unit = (long)s * H_kv + h;
  const long row0 = (long)s * H_q + (long)h * G;
  const float* base = s_hat + lay.base(s, h);
  // The loads below do not wait for the sequence length: positions are clamped
  // to the page table's width, and values of positions outside 1 .. n - 2 are
  // never used.
  // contiguous layout: float4 number f = kT i + tid of the chunk's span holds
  // heads 4 (f % LP) .. +3 of page p0 + f / LP; the LP lanes of a page are
  // adjacent.  These loads are issued before Z_g is reduced.
  constexpr int LP = kG ? kG / 4 : 1, per = kG ? kFastChunk * kG / 4 / kT : 1;
  float4 v[per];
  if constexpr (kG != 0) {
#pragma unroll
    for (int i = 0; i < per; ++i) {
      const int po = (i * kT + tid) / LP;
      const long j = min(p0 + po, max_pages - 1);
      v[i] = *reinterpret_cast<const float4*>(base + j * kG + 4 * (tid % LP));
    }
  }
  // physical blocks of this thread's key positions
  int32_t blk[kChunkNK];
#pragma unroll
  for (int u = 0; u < kChunkNK; ++u) {
    const int j = p0 + (wave * kChunkNK + u) * 64 + lane;
    blk[u] = page_table[(long)s * max_pages + min(j, max_pages - 1)];
  }
  {
    constexpr int kPer = 16;  // partials per thread and pass (16 threads per head)
    const int g = tid >> 4, sub = tid & 15;
    const float2* pp = partials + (row0 + (g < G ? g : 0)) * n_parts;
    float m = -INFINITY, l = 0.0f;
    for (int b0 = 0; b0 < n_parts; b0 += 16 * kPer) {
      float2 pv[kPer];
#pragma unroll
      for (int u = 0; u < kPer; ++u) pv[u] = pp[min(b0 + sub + 16 * u, n_parts - 1)];
#pragma unroll
      for (int u = 0; u < kPer; ++u) pin(pv[u].x), pin(pv[u].y);
#pragma unroll
      for (int u = 0; u < kPer; ++u)
        if (!(g < G && b0 + sub + 16 * u < n_parts)) pv[u] = make_float2(-INFINITY, 0.0f);
      float mm = m;
#pragma unroll
      for (int u = 0; u < kPer; ++u) mm = fmaxf(mm, pv[u].x);
      float ll = (m > -INFINITY) ? l * __builtin_amdgcn_exp2f(m - mm) : 0.0f;
#pragma unroll
      for (int u = 0; u < kPer; ++u)
        ll += (pv[u].y > 0.0f) ? pv[u].y * __builtin_amdgcn_exp2f(pv[u].x - mm) : 0.0f;
      m = mm;
      l = ll;
    }
    if (part_x && sub == 0 && g < G && sl_scan[s] < Ls) {  // the page scored by the build
      const float2 x = part_x[row0 + g];
      const float mm = fmaxf(m, x.x);
      if (mm > -INFINITY) {
        l = (m > -INFINITY ? l * __builtin_amdgcn_exp2f(m - mm) : 0.0f) +
            (x.y > 0.0f ? x.y * __builtin_amdgcn_exp2f(x.x - mm) : 0.0f);
        m = mm;
      }
    }
    for (int o = 8; o > 0; o >>= 1) {
      const float om = __shfl_xor(m, o, 64), ol = __shfl_xor(l, o, 64);
      const float mm = fmaxf(m, om);
      l = (mm > -INFINITY) ? l * __builtin_amdgcn_exp2f(m - mm) + ol * __builtin_amdgcn_exp2f(om - mm)
                           : 0.0f;
      m = mm;
    }
    if (g < G && sub == 0) s_lz2[g] = m + __builtin_amdgcn_logf(l);
  }
  __syncthreads();
  const int n = (Ls + pgsz - 1) / pgsz;
  if (n <= k || p0 > n - 2) return;  // uniform across the block
  if constexpr (kG != 0) {
    const int q = tid % LP;
    float lzq[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) lzq[c] = s_lz2[4 * q + c];
#pragma unroll
    for (int i = 0; i < per; ++i) {
      const int po = (i * kT + tid) / LP;
      const float a0 = v[i].x * kLog2e - lzq[0], a1 = v[i].y * kLog2e - lzq[1];
      const float a2 = v[i].z * kLog2e - lzq[2], a3 = v[i].w * kLog2e - lzq[3];
      float m = fmaxf(fmaxf(a0, a1), fmaxf(a2, a3));
      if (LP >= 2) m = fmaxf(m, quad_xor<1>(m));
      if (LP >= 4) m = fmaxf(m, quad_xor<2>(m));
      float sum = __builtin_amdgcn_exp2f(a0 - m) + __builtin_amdgcn_exp2f(a1 - m) +
                  __builtin_amdgcn_exp2f(a2 - m) + __builtin_amdgcn_exp2f(a3 - m);
      if (LP >= 2) sum += quad_xor<1>(sum);
      if (LP >= 4) sum += quad_xor<2>(sum);
      const int j = p0 + po;
      if (q == 0) sk[po] = (j >= 1 && j <= n - 2) ? page_key(m, sum) : 0u;
    }
  } else {
    float lz[kMaxGroup];
#pragma unroll
    for (int g = 0; g < kMaxGroup; ++g) lz[g] = g < G ? s_lz2[g] : 0.0f;
#pragma unroll
    for (int part = 0; part < kFastChunk / kT; ++part) {
      const int j = p0 + part * kT + tid;
      const long jj = min(max(j, 1), n - 2);
      float sv[kMaxGroup];
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g)
        sv[g] = base[jj * lay.page + (long)(g < G ? g : 0) * lay.head];
      float m = -INFINITY;
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g)
        if (g < G) m = fmaxf(m, sv[g] * kLog2e - lz[g]);
      float sum = 0.0f;
#pragma unroll
      for (int g = 0; g < kMaxGroup; ++g)
        if (g < G) sum += __builtin_amdgcn_exp2f(sv[g] * kLog2e - lz[g] - m);
      sk[part * kT + tid] = (j >= 1 && j <= n - 2) ? page_key(m, sum) : 0u;
    }
  }
  __syncthreads();
  uint32_t key[kChunkNK];
#pragma unroll
  for (int u = 0; u < kChunkNK; ++u) key[u] = sk[(wave * kChunkNK + u) * 64 + lane];
  // every page's key (0 for the sink), for an exact recut when the survivors
  // do not suffice; the chunks that run cover pages 0 .. n - 2
#pragma unroll
  for (int u = 0; u < kChunkNK; ++u) {
    const int j = p0 + (wave * kChunkNK + u) * 64 + lane;
    if (j < n) sb.keys[unit * max_pages + j] = key[u];
  }
  const WaveCut cut = block_hist_cut<kChunkNK, kChunkWaves>(key, width, HL, L);
  const long row = (unit * n_rows + chunk) * width;
  const int tot = block_emit<kChunkNK, kChunkWaves>(key, cut, L, [&](int u, int slot) {
    sb.cand_key[row + slot] = key[u];
    sb.cand_idx[row + slot] = p0 + (wave * kChunkNK + u) * 64 + lane;
    sb.cand_blk[row + slot] = blk[u];
  });
  for (int t = tot + tid; t < width; t += kT) {
    sb.cand_key[row + t] = 0u;
    sb.cand_idx[row + t] = -1;
    sb.cand_blk[row + t] = -1;
  }
  if (tid == 0) sb.sat[unit * n_rows + chunk] = cut.take_eq > width ? 0u : cut.T;
}

__global__ __launch_bounds__(kChunkThreads) void select_merge_fast_kernel(
    int H_q, int H_kv, int k, int width, int n_rows, int max_pages, int pgsz,
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ page_table,
    const float* __restrict__ s_hat, SHatLayout lay, SelectBufs sb, int32_t* __restrict__ out_ids,
    float* __restrict__ out_sel_lse) {
  __shared__ UnionLds<kChunkWaves> UL;
  __shared__ int32_t s_tab[kFastK + 2], s_blk[kFastK + 2];
  const int h = blockIdx.x, s = blockIdx.y, tid = threadIdx.x;
  const int Ls = seq_lens[s];
  const int n = (Ls + pgsz - 1) / pgsz;
  const int n_c = Ls / pgsz;
  const int G = H_q / H_kv;
  const long row0 = (long)s * H_q + (long)h * G;
  const long unit = (long)s * H_kv + h;
  const int used = n > k ? (n - 2) / kFastChunk + 1 : 0;
  union_table<kUnionNK, kChunkWaves>(
      k, n, used, width, sb.cand_key + unit * n_rows * width, sb.cand_idx + unit * n_rows * width,
      sb.cand_blk + unit * n_rows * width, sb.sat + unit * n_rows, sb.keys + unit * max_pages,
      page_table + (long)s * max_pages, s_tab, s_blk, UL);
  if (tid < k) out_ids[unit * k + tid] = s_tab[tid];
  // estimated page LSE of every table entry (NaN for a partial page or padding)
  const float* sbase = s_hat + lay.base(s, h);
  constexpr int kPer = (kMaxGroup * (kFastK + 2) + kChunkThreads - 1) / kChunkThreads;
  float val[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int e = tid + kChunkThreads * u;
    const int g = e / k, t = e - g * k;
    const int id = e < G * k ? s_tab[t] : -1;
    const bool ok = id >= 0 && id < n_c;
    const float x = sbase[(long)(ok ? id : 0) * lay.page + (long)(ok ? g : 0) * lay.head];
    val[u] = ok ? x : __int_as_float(0x7fc00000);
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int e = tid + kChunkThreads * u;
    if (e < G * k) out_sel_lse[row0 * k + e] = val[u];
  }
}

}  // namespace

int select_fast_rows(const locks_cfg_t& c) {
  return (c.max_pages_per_seq + kFastChunk - 1) / kFastChunk;
}

// Survivors kept per chunk: the smallest power of two >= k - 2, or fewer so
// that all chunks' survivors fit one merge (at least 8).
int select_fast_width(const locks_cfg_t& c) {
  const int K = page_budget(c) - 2;
  const long rows = select_fast_rows(c);
  int w = 8;
  while (w < K && 2L * w * rows <= kUnionCap) w *= 2;
  return w;
}

bool select_fast_path(const locks_cfg_t& c) {
  const int K = page_budget(c) - 2;
  return K <= kFastK && (long)select_fast_rows(c) * select_fast_width(c) <= kUnionCap;
}

hipError_t launch_select_chunks(const locks_cfg_t& c, const int32_t* page_table,
                                const int32_t* seq_lens, const float* s_hat, SHatLayout lay,
                                const float2* partials, const SelectBufs& sb, hipStream_t st,
                                const float2* part_x, const int32_t* sl_scan) {
  const int k = page_budget(c);
  const int G = c.num_q_heads / c.num_kv_heads;
  const bool contiguous = lay.head == 1 && lay.page == G;
  auto* kern = select_chunk_keys_kernel<0>;
  if (contiguous && G == 16) kern = select_chunk_keys_kernel<16>;
  if (contiguous && G == 8) kern = select_chunk_keys_kernel<8>;
  if (contiguous && G == 4) kern = select_chunk_keys_kernel<4>;
  const int rows = select_fast_rows(c);
  hipLaunchKernelGGL(kern, dim3(rows, c.num_kv_heads, c.num_seqs), dim3(kChunkThreads), 0, st,
                     c.num_q_heads, c.num_kv_heads, k, select_fast_width(c), c.max_pages_per_seq,
                     c.page_size, seq_lens, page_table, s_hat, lay, partials, scan_blocks(c), sb,
                     rows, part_x, sl_scan);
  return hipGetLastError();
}

hipError_t launch_select(const locks_cfg_t& c, const int32_t* page_table, const int32_t* seq_lens,
                         const float* s_hat, SHatLayout lay, const float2* partials,
                         const SelectBufs& sb, int32_t* out_page_ids, float* out_sel_lse,
                         hipStream_t st) {
  const int k = page_budget(c);
  if (select_fast_path(c)) {
    hipError_t e = launch_select_chunks(c, page_table, seq_lens, s_hat, lay, partials, sb, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(select_merge_fast_kernel, dim3(c.num_kv_heads, c.num_seqs),
                       dim3(kChunkThreads), 0, st, c.num_q_heads, c.num_kv_heads, k,
                       select_fast_width(c), select_fast_rows(c), c.max_pages_per_seq, c.page_size,
                       seq_lens, page_table, s_hat, lay, sb, out_page_ids, out_sel_lse);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(select_chunk_kernel, dim3(sb.n_chunks, c.num_kv_heads, c.num_seqs),
                     dim3(kSelThreads), 0, st, c.num_q_heads, c.num_kv_heads, k, sb.n_chunks,
                     c.page_size, seq_lens, s_hat, lay, partials, scan_blocks(c), sb.cand_key,
                     sb.cand_idx);
  hipLaunchKernelGGL(select_merge_kernel, dim3(c.num_kv_heads, c.num_seqs), dim3(kSelThreads), 0,
                     st, c.num_q_heads, c.num_kv_heads, k, sb.n_chunks, c.page_size, seq_lens,
                     s_hat, lay, sb.cand_key, sb.cand_idx, out_page_ids, out_sel_lse);
  return hipGetLastError();
}

}  // namespace locks
