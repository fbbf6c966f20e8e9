// Summary scan (Sec. 4 "Score", Eq. (1)): for every complete page j of a
// (sequence, KV head) and every query head g of its group,
//   hat s_j(q_g) = log sum_i exp[(q_g^T mu_j + (V_j^T q_g)^T c_i) / sqrt(d)],
// read from the page's stored record (int4 basis, int8 coefficients and centroid,
// float16 scales).  Also writes, per block of kScanTile pages and per query head,
// the partial (max, sum exp) that the combine step needs for the share normaliser.
//
// Mapping: one 64-lane wave per block, one page per lane, the group's queries in
// LDS (broadcast reads).  Integer codes are accumulated against q in fp32 and the
// scale is applied once per dot product, so the dequantisation is exact.
#include "locks_internal.h"

namespace locks {
namespace {

template <typename QT>
__device__ __forceinline__ float load_q(const QT* q, size_t i);
template <>
__device__ __forceinline__ float load_q<float>(const float* q, size_t i) { return q[i]; }
template <>
__device__ __forceinline__ float load_q<uint16_t>(const uint16_t* q, size_t i) {
  return bf16_bits_to_f32(q[i]);
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t b) {
  _Float16 h;
  __builtin_memcpy(&h, &b, 2);
  return (float)h;
}

template <typename QT, int R>
__global__ __launch_bounds__(64) void scan_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q,
    const uint8_t* __restrict__ summaries, const int32_t* __restrict__ page_table,
    const int32_t* __restrict__ seq_lens, float* __restrict__ s_hat, int s_hat_stride,
    float2* __restrict__ partials, int n_tiles) {
  constexpr int stride = rec_stride(R);
  __shared__ float sq[kMaxGroup][kDim];
  const int tile = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int lane = threadIdx.x;
  const int G = H_q / H_kv;
  const int n_c = seq_lens[s] / kPage;
  if (tile * kScanTile >= n_c) {
    // no complete page in this tile: an empty partial keeps the combine exact
    if (tile < n_tiles)
      for (int g = lane; g < G; g += 64)
        partials[((long)s * H_q + h * G + g) * n_tiles + tile] = make_float2(-INFINITY, 0.0f);
    return;
  }
  for (int e = lane; e < G * kDim; e += 64)
    sq[e / kDim][e % kDim] = load_q(q, ((long)s * H_q + h * G) * kDim + e);
  __syncthreads();

  const int j = tile * kScanTile + lane;
  const bool valid = j < n_c;
  const long blk = valid ? (long)page_table[(long)s * max_pages + j] : 0;
  const uint8_t* rec = summaries + (blk * H_kv + h) * (long)stride;

  // scales and coefficient codes of this lane's page
  const uint16_t* sc = reinterpret_cast<const uint16_t*>(rec + rec_scale_off(R));
  float vs[R];
#pragma unroll
  for (int l = 0; l < R; ++l) vs[l] = f16_bits_to_f32(sc[l]);
  const float ms = f16_bits_to_f32(sc[R + kPage]);
  constexpr float kLog2e = 1.4426950408889634f;
  const float zscale = kLog2e / sqrtf((float)kDim);

  for (int g = 0; g < G; ++g) {
    float a = 0.0f;
    float p[R];
#pragma unroll
    for (int l = 0; l < R; ++l) p[l] = 0.0f;
    for (int c0 = 0; c0 < kDim; c0 += 8) {
      const uint2 mb = *reinterpret_cast<const uint2*>(rec + rec_mu_off(R) + c0);
      float qq[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) qq[t] = sq[g][c0 + t];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t w = t < 4 ? mb.x : mb.y;
        const int code = (int)((w >> (8 * (t & 3))) & 0xffu) - 128;
        a = fmaf((float)code, qq[t], a);
      }
#pragma unroll
      for (int l = 0; l < R; ++l) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(rec + 64 * l + c0 / 2);
        float acc = p[l];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int code = (int)((w >> (4 * t)) & 0xfu) - 8;
          acc = fmaf((float)code, qq[t], acc);
        }
        p[l] = acc;
      }
    }
    a *= ms;
#pragma unroll
    for (int l = 0; l < R; ++l) p[l] *= vs[l];
    // 16 reconstructed logits (log2 domain) and their log-sum-exp
    float z[kPage];
    float zmax = -INFINITY;
#pragma unroll
    for (int i = 0; i < kPage; ++i) {
      float dot = 0.0f;
#pragma unroll
      for (int l = 0; l < R; ++l) {
        const int code = (int)rec[rec_coef_off(R) + i * R + l] - 128;
        dot = fmaf((float)code, p[l], dot);
      }
      const float cs = f16_bits_to_f32(sc[R + i]);
      z[i] = fmaf(cs, dot, a) * zscale;
      zmax = fmaxf(zmax, z[i]);
    }
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < kPage; ++i) sum += exp2f(z[i] - zmax);
    const float shat = (zmax + log2f(sum)) * 0.69314718055994531f;
    const long row = (long)s * H_q + h * G + g;
    if (valid) s_hat[row * s_hat_stride + j] = shat;
    // tile partial of the normaliser sum_j exp(hat s_j)
    const float m = warp_max(valid ? shat : -INFINITY);
    const float l = warp_sum(valid ? __expf(shat - m) : 0.0f);
    if (lane == 0) partials[row * n_tiles + tile] = make_float2(m, l);
  }
}

template <typename QT>
hipError_t dispatch(int r, dim3 grid, hipStream_t st, int H_q, int H_kv, int max_pages,
                    const QT* q, const uint8_t* sum, const int32_t* pt, const int32_t* sl,
                    float* s_hat, int s_hat_stride, float2* part, int n_tiles) {
#define LOCKS_SCAN_CASE(RR)                                                                   \
  case RR:                                                                                    \
    hipLaunchKernelGGL((scan_kernel<QT, RR>), grid, dim3(64), 0, st, H_q, H_kv, max_pages, q, \
                       sum, pt, sl, s_hat, s_hat_stride, part, n_tiles);                      \
    break;
  switch (r) {
    LOCKS_SCAN_CASE(1) LOCKS_SCAN_CASE(2) LOCKS_SCAN_CASE(3) LOCKS_SCAN_CASE(4)
    LOCKS_SCAN_CASE(5) LOCKS_SCAN_CASE(6) LOCKS_SCAN_CASE(7) LOCKS_SCAN_CASE(8)
    LOCKS_SCAN_CASE(9) LOCKS_SCAN_CASE(10) LOCKS_SCAN_CASE(11) LOCKS_SCAN_CASE(12)
    LOCKS_SCAN_CASE(13) LOCKS_SCAN_CASE(14) LOCKS_SCAN_CASE(15)
    default:
      return hipErrorInvalidValue;
  }
#undef LOCKS_SCAN_CASE
  return hipGetLastError();
}

}  // namespace

hipError_t launch_scan(const locks_cfg_t& c, const void* q, const void* summaries,
                       const int32_t* page_table, const int32_t* seq_lens, float* s_hat,
                       int s_hat_stride, float2* partials, int n_tiles, hipStream_t st) {
  const dim3 grid(n_tiles, c.num_kv_heads, c.num_seqs);
  if (c.q_dtype == LOCKS_BF16)
    return dispatch(c.rank, grid, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq,
                    static_cast<const uint16_t*>(q), static_cast<const uint8_t*>(summaries),
                    page_table, seq_lens, s_hat, s_hat_stride, partials, n_tiles);
  return dispatch(c.rank, grid, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq,
                  static_cast<const float*>(q), static_cast<const uint8_t*>(summaries),
                  page_table, seq_lens, s_hat, s_hat_stride, partials, n_tiles);
}

}  // namespace locks
