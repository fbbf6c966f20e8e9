// Share-average combine and shared top-k table (Sec. 4 "Score"; Cor.
// "Group-shared selection"; App. E "union table").
//
//  1. lz_kernel     log Z_g = log sum_j exp(hat s_j(q_g)) over every complete page,
//                   from the scan's per-tile (max, sum exp) partials.
//  2. key_kernel    per candidate page (neither page 0 nor the most recent page):
//                   log mbar_j + log G = log sum_g exp(hat s_j(q_g) - log Z_g),
//                   stored as an order-preserving uint32 key.
//  3. topk_kernel   one block per (sequence, KV head): radix select of the
//                   (k-2)-th largest key (4 passes of 8 bits), then an ordered
//                   compaction that keeps every larger key and the lowest-index
//                   equal keys, so ties go to the lower page index and the table
//                   comes out ascending; adds page 0 and the most recent page and
//                   gathers the selected pages' hat s for every head of the group.
#include "locks_internal.h"

namespace locks {
namespace {

constexpr int kKeyBlock = 256;
constexpr int kTopkBlock = 1024;
constexpr int kTopkWaves = kTopkBlock / 64;

__global__ __launch_bounds__(256) void lz_kernel(int H_q, const int32_t* __restrict__ seq_lens,
                                                 const float2* __restrict__ partials, int n_tiles,
                                                 float* __restrict__ lz) {
  const int hq = blockIdx.x, s = blockIdx.y;
  const int n_c = seq_lens[s] / kPage;
  const int used = (n_c + kScanTile - 1) / kScanTile;
  const float2* p = partials + ((long)s * H_q + hq) * n_tiles;
  __shared__ float red[4];
  float m = -INFINITY;
  for (int t = threadIdx.x; t < used; t += 256) m = fmaxf(m, p[t].x);
  m = warp_max(m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float l = 0.0f;
  if (m > -INFINITY)
    for (int t = threadIdx.x; t < used; t += 256) {
      const float2 v = p[t];
      if (v.y > 0.0f) l += v.y * __expf(v.x - m);
    }
  l = warp_sum(l);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = l;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float tot = red[0] + red[1] + red[2] + red[3];
    lz[(long)s * H_q + hq] = (m > -INFINITY) ? m + logf(tot) : -INFINITY;
  }
}

__global__ __launch_bounds__(kKeyBlock) void key_kernel(int H_q, int H_kv, int max_pages,
                                                        const int32_t* __restrict__ seq_lens,
                                                        const float* __restrict__ s_hat,
                                                        int s_hat_stride, const float* __restrict__ lz,
                                                        uint32_t* __restrict__ keys) {
  const int h = blockIdx.y, s = blockIdx.z;
  const int j = blockIdx.x * kKeyBlock + threadIdx.x;
  const int L = seq_lens[s];
  const int n = (L + kPage - 1) / kPage;
  if (j < 1 || j > n - 2) return;  // only candidates get a key
  const int G = H_q / H_kv;
  const long row0 = (long)s * H_q + h * G;
  float m = -INFINITY;
  for (int g = 0; g < G; ++g) m = fmaxf(m, s_hat[(row0 + g) * s_hat_stride + j] - lz[row0 + g]);
  float sum = 0.0f;
  for (int g = 0; g < G; ++g) sum += __expf(s_hat[(row0 + g) * s_hat_stride + j] - lz[row0 + g] - m);
  const float score = m + __logf(sum);
  keys[((long)s * H_kv + h) * max_pages + j] = f32_order_key(score);
}

// Exclusive prefix count of a per-thread flag over the whole block, in thread
// order.  Returns the count before this thread; *total gets the block total.
__device__ __forceinline__ int block_excl_count(bool flag, int* wave_tot, int* total) {
  const uint64_t ballot = __ballot(flag);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t below = lane ? (ballot & ((~0ull) >> (64 - lane))) : 0ull;
  const int in_wave = __popcll(below);
  if (lane == 0) wave_tot[wave] = __popcll(ballot);
  __syncthreads();
  int before = 0, tot = 0;
  for (int w = 0; w < kTopkWaves; ++w) {
    const int v = wave_tot[w];
    before += (w < wave) ? v : 0;
    tot += v;
  }
  __syncthreads();
  *total = tot;
  return before + in_wave;
}

__global__ __launch_bounds__(kTopkBlock) void topk_kernel(
    int H_q, int H_kv, int max_pages, int k, const int32_t* __restrict__ seq_lens,
    const uint32_t* __restrict__ keys_all, const float* __restrict__ s_hat, int s_hat_stride,
    int32_t* __restrict__ out_ids, float* __restrict__ out_sel_lse) {
  const int h = blockIdx.x, s = blockIdx.y;
  const int tid = threadIdx.x;
  const int L = seq_lens[s];
  const int n = (L + kPage - 1) / kPage;
  const int n_c = L / kPage;
  const int G = H_q / H_kv;
  int32_t* ids = out_ids + ((long)s * H_kv + h) * k;
  const uint32_t* keys = keys_all + ((long)s * H_kv + h) * max_pages;

  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_prefix, sh_mask, sh_remaining;
  __shared__ int wave_tot[kTopkWaves];

  if (n <= k) {
    for (int t = tid; t < k; t += kTopkBlock) ids[t] = t < n ? t : -1;
  } else {
    const int K = k - 2;
    if (tid == 0) { sh_prefix = 0; sh_mask = 0; sh_remaining = (uint32_t)K; }
    __syncthreads();
    for (int pass = 0; pass < 4; ++pass) {
      const int shift = 24 - 8 * pass;
      for (int t = tid; t < 256; t += kTopkBlock) hist[t] = 0;
      __syncthreads();
      const uint32_t prefix = sh_prefix, mask = sh_mask;
      for (int j = 1 + tid; j <= n - 2; j += kTopkBlock) {
        const uint32_t key = keys[j];
        if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid == 0) {
        uint32_t rem = sh_remaining, cum = 0;
        int dsel = 0;
        for (int dgt = 255; dgt >= 0; --dgt) {
          if (cum + hist[dgt] >= rem) { dsel = dgt; break; }
          cum += hist[dgt];
        }
        sh_remaining = rem - cum;
        sh_prefix = prefix | ((uint32_t)dsel << shift);
        sh_mask = mask | (255u << shift);
      }
      __syncthreads();
    }
    const uint32_t T = sh_prefix;
    const int take_eq = (int)sh_remaining;  // equal keys to keep, lowest index first
    int run_eq = 0, run_sel = 0;
    for (int base = 1; base <= n - 2; base += kTopkBlock) {
      const int j = base + tid;
      const bool in = j <= n - 2;
      const uint32_t key = in ? keys[j] : 0u;
      const bool gt = in && key > T;
      const bool eq = in && key == T;
      int tot_eq, tot_sel;
      const int before_eq = block_excl_count(eq, wave_tot, &tot_eq);
      const bool sel = gt || (eq && run_eq + before_eq < take_eq);
      const int before_sel = block_excl_count(sel, wave_tot, &tot_sel);
      if (sel) ids[1 + run_sel + before_sel] = j;
      run_eq += tot_eq;
      run_sel += tot_sel;
    }
    if (tid == 0) { ids[0] = 0; ids[k - 1] = n - 1; }
  }
  __syncthreads();
  // hat s of the selected pages for every head of the group (NaN without summary)
  for (int e = tid; e < G * k; e += kTopkBlock) {
    const int g = e / k, t = e % k;
    const int id = ids[t];
    const long row = (long)s * H_q + h * G + g;
    out_sel_lse[row * k + t] = (id >= 0 && id < n_c) ? s_hat[row * s_hat_stride + id] : __int_as_float(0x7fc00000);
  }
}

}  // namespace

hipError_t launch_select(const locks_cfg_t& c, const float* s_hat, int s_hat_stride,
                         const float2* partials, int n_tiles, const int32_t* seq_lens, float* lz,
                         uint32_t* keys, int32_t* out_page_ids, float* out_sel_lse,
                         hipStream_t st) {
  const int k = page_budget(c);
  hipLaunchKernelGGL(lz_kernel, dim3(c.num_q_heads, c.num_seqs), dim3(256), 0, st, c.num_q_heads,
                     seq_lens, partials, n_tiles, lz);
  hipLaunchKernelGGL(key_kernel,
                     dim3((c.max_pages_per_seq + kKeyBlock - 1) / kKeyBlock, c.num_kv_heads, c.num_seqs),
                     dim3(kKeyBlock), 0, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq,
                     seq_lens, s_hat, s_hat_stride, lz, keys);
  hipLaunchKernelGGL(topk_kernel, dim3(c.num_kv_heads, c.num_seqs), dim3(kTopkBlock), 0, st,
                     c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq, k, seq_lens, keys, s_hat,
                     s_hat_stride, out_page_ids, out_sel_lse);
  return hipGetLastError();
}

}  // namespace locks
