// The caller's KV write of a decode step (App. E, schedule of the KV write beside
// the selector): the newest token of every sequence, token seq_lens[s] - 1, is
// copied from the step's new key and value rows into its slot of the paged cache.
#include <type_traits>

#include "locks_internal.h"

namespace locks {
namespace {

// One wave per (sequence, KV head): lanes 0..31 copy the key row, lanes 32..63 the
// value row, four elements each (8 bytes of bf16, 16 bytes of fp32).
template <typename T>
__global__ __launch_bounds__(256) void append_kernel(const T* __restrict__ k_new,
                                                     const T* __restrict__ v_new,
                                                     T* __restrict__ k_cache, T* __restrict__ v_cache,
                                                     const int32_t* __restrict__ page_table,
                                                     const int32_t* __restrict__ seq_lens,
                                                     long n_units, int H_kv, int max_pages,
                                                     int pgsz) {
  using V4 = typename std::conditional<sizeof(T) == 2, uint2, uint4>::type;
  const long unit = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (unit >= n_units) return;
  const int lane = threadIdx.x & 63;
  const int s = (int)(unit / H_kv), h = (int)(unit % H_kv);
  const int L = seq_lens[s];
  if (L < 1) return;
  const int t = L - 1;
  const long blk = page_table[(long)s * max_pages + t / pgsz];
  const size_t dst = (((size_t)blk * H_kv + h) * pgsz + t % pgsz) * kDim + 4 * (lane & 31);
  const size_t src = (size_t)unit * kDim + 4 * (lane & 31);
  const T* from = lane < 32 ? k_new : v_new;
  T* to = lane < 32 ? k_cache : v_cache;
  *reinterpret_cast<V4*>(to + dst) = *reinterpret_cast<const V4*>(from + src);
}

}  // namespace

hipError_t launch_append(const locks_cfg_t& c, const void* k_new, const void* v_new,
                         void* k_cache, void* v_cache, const int32_t* page_table,
                         const int32_t* seq_lens, hipStream_t st) {
  const long units = (long)c.num_seqs * c.num_kv_heads;
  if (units <= 0) return hipSuccess;
  const dim3 grid((unsigned)((units + 3) / 4)), block(256);
  if (c.kv_dtype == LOCKS_BF16)
    hipLaunchKernelGGL(append_kernel<uint16_t>, grid, block, 0, st,
                       static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new),
                       static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), page_table,
                       seq_lens, units, c.num_kv_heads, c.max_pages_per_seq, c.page_size);
  else
    hipLaunchKernelGGL(append_kernel<float>, grid, block, 0, st,
                       static_cast<const float*>(k_new), static_cast<const float*>(v_new),
                       static_cast<float*>(k_cache), static_cast<float*>(v_cache), page_table,
                       seq_lens, units, c.num_kv_heads, c.max_pages_per_seq, c.page_size);
  return hipGetLastError();
}

}  // namespace locks
