// Share-average combine and shared top-k table (Sec. 4 "Score"; Cor.
// "Group-shared selection"; App. E "union table").
//
// One kernel, grid (chunk of kSelChunk pages, KV head, sequence):
//  1. every block reduces the scan blocks' partials into lz2_g = log2 Z_g, then
//     scores the candidate pages of its chunk (neither page 0 nor the most recent
//     page):  log2 mbar_j + log2 G = log2 sum_g 2^(s2_j(q_g) - lz2_g); the score
//     becomes an order-preserving uint32 key (key 0 marks "no candidate");
//  2. the block keeps its chunk's top (k-2) keys: a bisection over the key space
//     finds T, the (k-2)-th largest key, then an ordered compaction keeps every key
//     above T and the lowest-index keys equal to T, so ties go to the lower page
//     index and the survivors come out in ascending page order;
//  3. the last block of the (sequence, KV head) to finish (device-scope counter)
//     runs the same selection over all chunks' survivors, adds page 0 and the most
//     recent page, writes the ascending table, gathers hat s of the selected pages
//     for every head of the group and leaves the counter at zero.
#include "locks_internal.h"

namespace locks {
namespace {

constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kPerThread = kSelChunk / kSelThreads;
constexpr int kLdsCand = 8192;  // survivors the merge keeps in LDS

struct Red {
  int v[2][kSelWaves];
  uint32_t mx[kSelWaves], mn[kSelWaves];
  int flag;
};

__device__ __forceinline__ int wave_sum_i(int v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Sum over the block (all threads must call; alternate `par` between calls).
__device__ __forceinline__ int block_sum(int v, Red& r, int par) {
  v = wave_sum_i(v);
  if ((threadIdx.x & 63) == 0) r.v[par][threadIdx.x >> 6] = v;
  __syncthreads();
  int t = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) t += r.v[par][w];
  return t;
}

// Exclusive prefix count of a flag in thread order, and the block total.
__device__ __forceinline__ int block_excl(bool p, Red& r, int par, int* total) {
  const uint64_t b = __ballot(p);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int in_wave = __popcll(lane ? (b & (~0ull >> (64 - lane))) : 0ull);
  if (lane == 0) r.v[par][wave] = __popcll(b);
  __syncthreads();
  int before = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    before += w < wave ? r.v[par][w] : 0;
    tot += r.v[par][w];
  }
  *total = tot;
  return before + in_wave;
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

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    int H_q, int H_kv, int max_pages, int k, int n_chunks, const int32_t* __restrict__ seq_lens,
    const float* __restrict__ s_hat, int s_hat_stride, const float2* __restrict__ partials,
    int n_parts, uint32_t* __restrict__ cand_key, int32_t* __restrict__ cand_idx, int* __restrict__ counters,
    int32_t* __restrict__ out_ids, float* __restrict__ out_sel_lse) {
  __shared__ Red red;
  __shared__ float s_lz2[16];
  __shared__ uint32_t s_key[kLdsCand];
  __shared__ int32_t s_idx[kLdsCand];
  const int chunk = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int tid = threadIdx.x;
  const int L = seq_lens[s];
  const int n = (L + kPage - 1) / kPage;
  const int n_c = L / kPage;
  const int G = H_q / H_kv;
  const int K = k - 2;
  const long row0 = (long)s * H_q + (long)h * G;
  const long ch_base = ((long)s * H_kv + h) * n_chunks;
  constexpr float kLog2e = 1.4426950408889634f;
  int par = 0;
  const int p0 = chunk * kSelChunk;

  // ---- log2 Z_g from the scan blocks' (max, sum 2^x) partials; 16 threads per head
  if (n > k && p0 <= n - 2) {
    const int g = tid >> 4, sub = tid & 15;
    const float2* pp = partials + (row0 + (g < G ? g : 0)) * n_parts;
    float m = -INFINITY, l = 0.0f;
    if (g < G)
      for (int t = sub; t < n_parts; t += 16) m = fmaxf(m, pp[t].x);
    for (int o = 8; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if (g < G && m > -INFINITY)
      for (int t = sub; t < n_parts; t += 16) {
        const float2 v = pp[t];
        if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
      }
    for (int o = 8; o > 0; o >>= 1) l += __shfl_xor(l, o, 64);
    if (g < G && sub == 0) s_lz2[g] = m + __builtin_amdgcn_logf(l);
    __syncthreads();
  }

  // ---- 1+2: chunk-local top K of the candidate pages
  if (n > k && p0 <= n - 2) {
    uint32_t key[kPerThread];
    uint32_t kmx = 0u, kmn = 0xffffffffu;
    int local = 0;
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      const int j = p0 + tid + kSelThreads * u;
      key[u] = 0u;
      if (j >= 1 && j <= n - 2) {
        float m = -INFINITY;
        for (int g = 0; g < G; ++g)
          m = fmaxf(m, s_hat[(row0 + g) * s_hat_stride + j] * kLog2e - s_lz2[g]);
        float sum = 0.0f;
        for (int g = 0; g < G; ++g)
          sum += __builtin_amdgcn_exp2f(s_hat[(row0 + g) * s_hat_stride + j] * kLog2e - s_lz2[g] - m);
        key[u] = max(1u, f32_order_key(m + __builtin_amdgcn_logf(sum)));
        kmx = max(kmx, key[u]);
        kmn = min(kmn, key[u]);
        ++local;
      }
    }
    const int n_cand = block_sum(local, red, par); par ^= 1;
    uint32_t T = 1u;
    int take_eq = 1 << 30;
    if (n_cand > K) {
      block_minmax(kmn, kmx, red);
      uint32_t lo = kmn, hi = kmx;  // invariant: #{key >= lo} >= K
      while (lo < hi) {
        const uint32_t mid = lo + (uint32_t)((((uint64_t)hi - lo) + 1) >> 1);
        int c = 0;
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) c += key[u] >= mid;
        if (block_sum(c, red, par) >= K) lo = mid; else hi = mid - 1;
        par ^= 1;
      }
      T = lo;
      int c = 0;
#pragma unroll
      for (int u = 0; u < kPerThread; ++u) c += key[u] > T;
      take_eq = K - block_sum(c, red, par); par ^= 1;
    }
    int run_eq = 0, run_sel = 0;
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
      int tot_eq, tot_sel;
      const bool eq = key[u] != 0u && key[u] == T;
      const int before_eq = block_excl(eq, red, par, &tot_eq); par ^= 1;
      const bool sel = (key[u] != 0u && key[u] > T) || (eq && run_eq + before_eq < take_eq);
      const int before_sel = block_excl(sel, red, par, &tot_sel); par ^= 1;
      if (sel) {
        cand_key[(ch_base + chunk) * K + run_sel + before_sel] = key[u];
        cand_idx[(ch_base + chunk) * K + run_sel + before_sel] = p0 + tid + kSelThreads * u;
      }
      run_eq += tot_eq;
      run_sel += tot_sel;
    }
    for (int t = run_sel + tid; t < K; t += kSelThreads) {
      cand_key[(ch_base + chunk) * K + t] = 0u;
      cand_idx[(ch_base + chunk) * K + t] = -1;
    }
  }

  // ---- 3: the last block of this (sequence, KV head) merges
  __threadfence();
  __syncthreads();
  if (tid == 0) red.flag = atomicAdd(&counters[s * H_kv + h], 1) == n_chunks - 1;
  __syncthreads();
  if (!red.flag) return;
  __threadfence();
  int32_t* ids = out_ids + ((long)s * H_kv + h) * k;
  if (n <= k) {
    for (int t = tid; t < k; t += kSelThreads) ids[t] = t < n ? t : -1;
  } else {
    const int used = (n - 2) / kSelChunk + 1;  // chunks that hold candidates (pages 1..n-2)
    const int N = used * K;
    const bool in_lds = N <= kLdsCand;
    const uint32_t* gk = cand_key + ch_base * K;
    const int32_t* gi = cand_idx + ch_base * K;
    if (in_lds) {
      for (int e = tid; e < N; e += kSelThreads) { s_key[e] = gk[e]; s_idx[e] = gi[e]; }
      __syncthreads();
    }
    uint32_t kmx = 0u, kmn = 0xffffffffu;
    for (int e = tid; e < N; e += kSelThreads) {
      const uint32_t v = in_lds ? s_key[e] : gk[e];
      if (v) { kmx = max(kmx, v); kmn = min(kmn, v); }
    }
    block_minmax(kmn, kmx, red);
    uint32_t lo = kmn, hi = kmx;
    while (lo < hi) {
      const uint32_t mid = lo + (uint32_t)((((uint64_t)hi - lo) + 1) >> 1);
      int c = 0;
      for (int e = tid; e < N; e += kSelThreads) c += (in_lds ? s_key[e] : gk[e]) >= mid;
      if (block_sum(c, red, par) >= K) lo = mid; else hi = mid - 1;
      par ^= 1;
    }
    const uint32_t T = lo;
    int c = 0;
    for (int e = tid; e < N; e += kSelThreads) c += (in_lds ? s_key[e] : gk[e]) > T;
    const int take_eq = K - block_sum(c, red, par);
    par ^= 1;
    // survivors are ascending in page index (chunk order, ascending inside a chunk)
    int run_eq = 0, run_sel = 0;
    for (int base = 0; base < N; base += kSelThreads) {
      const int e = base + tid;
      const uint32_t v = e < N ? (in_lds ? s_key[e] : gk[e]) : 0u;
      int tot_eq, tot_sel;
      const bool eq = v != 0u && v == T;
      const int before_eq = block_excl(eq, red, par, &tot_eq); par ^= 1;
      const bool sel = (v != 0u && v > T) || (eq && run_eq + before_eq < take_eq);
      const int before_sel = block_excl(sel, red, par, &tot_sel); par ^= 1;
      if (sel) ids[1 + run_sel + before_sel] = in_lds ? s_idx[e] : gi[e];
      run_eq += tot_eq;
      run_sel += tot_sel;
    }
    if (tid == 0) { ids[0] = 0; ids[k - 1] = n - 1; }
  }
  __syncthreads();
  for (int e = tid; e < G * k; e += kSelThreads) {
    const int g = e / k, t = e % k;
    const int id = ids[t];
    out_sel_lse[(row0 + g) * k + t] =
        (id >= 0 && id < n_c) ? s_hat[(row0 + g) * s_hat_stride + id] : __int_as_float(0x7fc00000);
  }
  if (tid == 0) counters[s * H_kv + h] = 0;
}

}  // namespace

hipError_t launch_select(const locks_cfg_t& c, const int32_t* seq_lens, const float* s_hat,
                         int s_hat_stride, const float2* partials, uint32_t* cand_key,
                         int32_t* cand_idx, int n_chunks, int* counters, int32_t* out_page_ids,
                         float* out_sel_lse, hipStream_t st) {
  const int k = page_budget(c);
  hipLaunchKernelGGL(select_kernel, dim3(n_chunks, c.num_kv_heads, c.num_seqs), dim3(kSelThreads),
                     0, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq, k, n_chunks,
                     seq_lens, s_hat, s_hat_stride, partials, scan_blocks(c), cand_key, cand_idx,
                     counters, out_page_ids, out_sel_lse);
  return hipGetLastError();
}

}  // namespace locks
