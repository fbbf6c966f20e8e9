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

// ---------------------------------------------------------------------------
// Matrix-core scan (group size G <= 16).
//
// A wave owns 64 consecutive pages (four tiles of 16) of one (sequence, KV head).
// Per tile:
//  * stage 1, the projections p = V^T q and a = mu^T q, run on 16x16x32 f16 MFMA:
//    rows are (page, basis column) pairs (16/r pages per set), columns are query
//    heads, K = d.  Each lane loads its 16-byte slice of one basis column straight
//    into its A operand; nibbles are decoded exactly to f16 through the 1024.0
//    exponent trick (OR into the mantissa, subtract the excess-8 bias in packed
//    f16).  The queries (bf16 or fp32 split hi + lo, both exact in f16 after a
//    power-of-two range scale) are the B operand, built once per wave.
//  * the rest of each record (coefficients, centroid, scales) is staged in LDS;
//    the centroid projection runs as one more MFMA set with one page per row.
//  * stage 2, the 16 logits z_i = a + c_i^T p, runs on 16x16x4 fp32 MFMA with the
//    16 tokens as rows; the 16 columns pack 16/G pages x G heads and the K axis is
//    block-diagonal over those pages, so small groups waste no lanes.
//  * log-sum-exp over the 16 rows: 4 values per lane, then two cross-lane steps.
// ---------------------------------------------------------------------------

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

template <int R>
struct Geom {
  static constexpr int kPPS = (16 / R) > 0 ? 16 / R : 1;          // pages per stage-1 set
  static constexpr int kSets = (16 + kPPS - 1) / kPPS;
  static constexpr int kStride = rec_stride(R);
  static constexpr int kTail = kStride - 64 * R;                   // coef .. end of record
  static constexpr int kTailCh = kTail / 16;
  static constexpr int kTailLoads = (16 * kTailCh + 63) / 64;
  static constexpr int kMu = 16 * R;                               // offsets inside the tail
  static constexpr int kSc = 16 * R + kDim;
};

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }

// 8 excess-8 nibbles (element t in bits 4t..4t+3) -> 8 exact f16 codes in the
// order t = 0,4,1,5,2,6,3,7.
__device__ __forceinline__ h8 nib8_to_h8(uint32_t w) {
  const uint32_t M = 0x64006400u;  // f16 1024.0 in both halves
  const uint32_t w8 = w >> 8;
  const h2 y0 = as_h2((w & 0x000F000Fu) | M) - h2{(_Float16)1032.0f, (_Float16)1032.0f};
  const h2 y1 = as_h2((w & 0x00F000F0u) | M) * h2{(_Float16)0.0625f, (_Float16)0.0625f} -
                h2{(_Float16)72.0f, (_Float16)72.0f};
  const h2 y2 = as_h2((w8 & 0x000F000Fu) | M) - h2{(_Float16)1032.0f, (_Float16)1032.0f};
  const h2 y3 = as_h2((w8 & 0x00F000F0u) | M) * h2{(_Float16)0.0625f, (_Float16)0.0625f} -
                h2{(_Float16)72.0f, (_Float16)72.0f};
  return h8{y0.x, y0.y, y1.x, y1.y, y2.x, y2.y, y3.x, y3.y};
}

// 8 excess-128 bytes -> 8 exact f16 codes in natural order.
__device__ __forceinline__ h8 byte8_to_h8(uint32_t w0, uint32_t w1) {
  const uint32_t M = 0x64646464u;
  const h2 k{(_Float16)1152.0f, (_Float16)1152.0f};
  const h2 a = as_h2(__builtin_amdgcn_perm(M, w0, 0x04010400u)) - k;
  const h2 b = as_h2(__builtin_amdgcn_perm(M, w0, 0x04030402u)) - k;
  const h2 c = as_h2(__builtin_amdgcn_perm(M, w1, 0x04010400u)) - k;
  const h2 d = as_h2(__builtin_amdgcn_perm(M, w1, 0x04030402u)) - k;
  return h8{a.x, a.y, b.x, b.y, c.x, c.y, d.x, d.y};
}

__device__ __forceinline__ float lds_f16(const uint8_t* p) {
  return (float)*reinterpret_cast<const _Float16*>(p);
}

template <typename QT, int R>
__global__ __launch_bounds__(256) void scan_mfma_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q,
    const uint8_t* __restrict__ summaries, const int32_t* __restrict__ page_table,
    const int32_t* __restrict__ seq_lens, float* __restrict__ s_hat, int s_hat_stride,
    float2* __restrict__ partials, int n_parts) {
  using Gm = Geom<R>;
  constexpr bool kSplitQ = sizeof(QT) == 4;  // fp32 queries: f16 hi + lo
  __shared__ __align__(16) uint8_t sTail[4][16][Gm::kTail];
  __shared__ float sP[4][16][R][16];
  __shared__ float sA[4][16][16];
  __shared__ float2 sRun[4][16];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = blockIdx.y, s = blockIdx.z;
  const int G = H_q / H_kv;
  const int n_c = seq_lens[s] / kPage;
  const int pg = blockIdx.x * 4 + wave;  // 64-page group of this wave
  const long row0 = (long)s * H_q + (long)h * G;
  if (pg * 64 >= n_c) {
    if (pg < n_parts && lane < G) partials[(row0 + lane) * n_parts + pg] = make_float2(-INFINITY, 0.0f);
    return;
  }

  // ---- B operands: column = query head, K permuted to match the decoders
  constexpr int kPerm[8] = {0, 4, 1, 5, 2, 6, 3, 7};
  float qv[4][8], qm[4][8];
  float qmax = 0.0f;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int cv = 32 * grp + 8 * ks + kPerm[j], cm = 32 * grp + 8 * ks + j;
      const float a = col < G ? load_q(q, (row0 + col) * kDim + cv) : 0.0f;
      const float b = col < G ? load_q(q, (row0 + col) * kDim + cm) : 0.0f;
      qv[ks][j] = a;
      qm[ks][j] = b;
      qmax = fmaxf(qmax, fabsf(a));
    }
  qmax = warp_max(qmax);
  // power-of-two range scale so that every query element fits f16 exactly
  float qs = 1.0f;
  while (qmax * qs > 16384.0f) qs *= 0.5f;
  const float inv_qs = 1.0f / qs;
  h8 bv[4], bm[4], bvl[4], bml[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float a = qv[ks][j] * qs, b = qm[ks][j] * qs;
      const _Float16 ah = (_Float16)a, bh = (_Float16)b;
      bv[ks][j] = ah;
      bm[ks][j] = bh;
      bvl[ks][j] = (_Float16)(a - (float)ah);
      bml[ks][j] = (_Float16)(b - (float)bh);
    }

  constexpr float kLog2e = 1.4426950408889634f;
  const float c0 = kLog2e * 0.08838834764831845f;  // log2(e) / sqrt(128)
  const int npack = 16 / G;                         // pages per stage-2 pass
  const int kpass = npack * R;
  const int ksteps = (kpass + 3) / 4;
  const int pcol = col / G, gcol = col % G;
  const bool colvalid = pcol < npack;
  float run_m = -INFINITY, run_s = 0.0f;

  for (int t = 0; t < 4; ++t) {
    const int page0 = (pg * 4 + t) * 16;
    if (page0 >= n_c) break;
    const int my_blk = (lane < 16 && page0 + lane < n_c)
                           ? page_table[(long)s * max_pages + page0 + lane] : -1;
    // ---- issue the loads: basis slices into registers, record tails into LDS
    uint4 vb[Gm::kSets];
#pragma unroll
    for (int st = 0; st < Gm::kSets; ++st) {
      const int pp = col / R, l = col % R;
      const int page = st * Gm::kPPS + pp;
      const int blk = __shfl(my_blk, page < 16 ? page : 0, 64);
      const bool ok = col < Gm::kPPS * R && page < 16 && blk >= 0;
      vb[st] = ok ? *reinterpret_cast<const uint4*>(summaries + ((long)blk * H_kv + h) * Gm::kStride +
                                                    64 * l + 16 * grp)
                  : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < Gm::kTailLoads; ++u) {
      const int c = lane + 64 * u;
      const int page = c / Gm::kTailCh, off = (c % Gm::kTailCh) * 16;
      const int blk = __shfl(my_blk, page < 16 ? page : 0, 64);
      if (c < 16 * Gm::kTailCh) {
        const uint4 v = blk >= 0 ? *reinterpret_cast<const uint4*>(
                                       summaries + ((long)blk * H_kv + h) * Gm::kStride + 64 * R + off)
                                 : make_uint4(0, 0, 0, 0);
        *reinterpret_cast<uint4*>(&sTail[wave][page][off]) = v;
      }
    }
    __builtin_amdgcn_wave_barrier();

    // ---- stage 1: p = V^T q (scaled by the basis column scales)
#pragma unroll
    for (int st = 0; st < Gm::kSets; ++st) {
      f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
      const uint32_t w[4] = {vb[st].x, vb[st].y, vb[st].z, vb[st].w};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const h8 a = nib8_to_h8(w[ks]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bv[ks], acc, 0, 0, 0);
        if (kSplitQ) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bvl[ks], acc, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int m = 4 * grp + j;
        const int pp = m / R, l = m % R;
        const int page = st * Gm::kPPS + pp;
        if (m < Gm::kPPS * R && page < 16 && col < G)
          sP[wave][page][l][col] = acc[j] * inv_qs * lds_f16(&sTail[wave][page][Gm::kSc + 2 * l]);
      }
    }
    // ---- centroid term a = mu^T q, one page per row
    {
      const uint4 m0 = *reinterpret_cast<const uint4*>(&sTail[wave][col][Gm::kMu + 32 * grp]);
      const uint4 m1 = *reinterpret_cast<const uint4*>(&sTail[wave][col][Gm::kMu + 32 * grp + 16]);
      const uint32_t w[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
      f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const h8 a = byte8_to_h8(w[2 * ks], w[2 * ks + 1]);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bm[ks], acc, 0, 0, 0);
        if (kSplitQ) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bml[ks], acc, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int page = 4 * grp + j;
        if (col < G)
          sA[wave][page][col] = acc[j] * inv_qs * lds_f16(&sTail[wave][page][Gm::kSc + 2 * (R + 16)]);
      }
    }
    __builtin_amdgcn_wave_barrier();

    // ---- stage 2: 16 logits per (page, head), npack pages per pass
    for (int p0 = 0; p0 < 16; p0 += npack) {
      f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
      for (int kstep = 0; kstep < ksteps; ++kstep) {
        const int k = 4 * kstep + grp;
        const int ppk = k / R, l = k % R;
        const int pk = p0 + ppk;
        const bool kv = k < kpass && pk < 16;
        const float a = kv ? (float)((int)sTail[wave][pk][col * R + l] - 128) : 0.0f;
        const float b = (kv && colvalid && ppk == pcol) ? sP[wave][pk][l][gcol] : 0.0f;
        acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
      }
      const int page = p0 + pcol;
      const bool live = colvalid && page < 16 && page0 + page < n_c;
      const int pl = page < 16 ? page : 15;
      const float av = sA[wave][pl][gcol] * c0;
      float z[4];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float cs = lds_f16(&sTail[wave][pl][Gm::kSc + 2 * (R + 4 * grp + j)]);
        z[j] = fmaf(cs * c0, acc[j], av);
        mx = fmaxf(mx, z[j]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      float sm = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) sm += exp2f(z[j] - mx);
      sm += __shfl_xor(sm, 16, 64);
      sm += __shfl_xor(sm, 32, 64);
      const float shat = (mx + log2f(sm)) * 0.69314718055994531f;
      if (live) {
        if (grp == 0) s_hat[(row0 + gcol) * s_hat_stride + page0 + page] = shat;
        const float nm = fmaxf(run_m, shat);
        run_s = run_s * exp2f((run_m - nm) * kLog2e) + exp2f((shat - nm) * kLog2e);
        run_m = nm;
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  // ---- per-head partial (max, sum exp) of this wave's 64 pages
  if (lane < 16) sRun[wave][lane] = make_float2(run_m, run_s);
  __builtin_amdgcn_wave_barrier();
  if (lane < G) {
    float m = -INFINITY, l = 0.0f;
    for (int c = lane; c < npack * G; c += G) m = fmaxf(m, sRun[wave][c].x);
    if (m > -INFINITY)
      for (int c = lane; c < npack * G; c += G) {
        const float2 v = sRun[wave][c];
        if (v.y > 0.0f) l += v.y * exp2f((v.x - m) * kLog2e);
      }
    partials[(row0 + lane) * n_parts + pg] = make_float2(m, l);
  }
}

template <typename QT>
hipError_t dispatch_mfma(int r, dim3 grid, hipStream_t st, int H_q, int H_kv, int max_pages,
                         const QT* q, const uint8_t* sum, const int32_t* pt, const int32_t* sl,
                         float* s_hat, int s_hat_stride, float2* part, int n_parts) {
#define LOCKS_SCAN_MFMA_CASE(RR)                                                             \
  case RR:                                                                                  \
    hipLaunchKernelGGL((scan_mfma_kernel<QT, RR>), grid, dim3(256), 0, st, H_q, H_kv,       \
                       max_pages, q, sum, pt, sl, s_hat, s_hat_stride, part, n_parts);      \
    break;
  switch (r) {
    LOCKS_SCAN_MFMA_CASE(1) LOCKS_SCAN_MFMA_CASE(2) LOCKS_SCAN_MFMA_CASE(3)
    LOCKS_SCAN_MFMA_CASE(4) LOCKS_SCAN_MFMA_CASE(5) LOCKS_SCAN_MFMA_CASE(6)
    LOCKS_SCAN_MFMA_CASE(7) LOCKS_SCAN_MFMA_CASE(8) LOCKS_SCAN_MFMA_CASE(9)
    LOCKS_SCAN_MFMA_CASE(10) LOCKS_SCAN_MFMA_CASE(11) LOCKS_SCAN_MFMA_CASE(12)
    LOCKS_SCAN_MFMA_CASE(13) LOCKS_SCAN_MFMA_CASE(14) LOCKS_SCAN_MFMA_CASE(15)
    default:
      return hipErrorInvalidValue;
  }
#undef LOCKS_SCAN_MFMA_CASE
  return hipGetLastError();
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
  const int G = c.num_q_heads / c.num_kv_heads;
  if (G <= 16) {
    const dim3 grid((n_tiles + 3) / 4, c.num_kv_heads, c.num_seqs);
    if (c.q_dtype == LOCKS_BF16)
      return dispatch_mfma(c.rank, grid, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq,
                           static_cast<const uint16_t*>(q), static_cast<const uint8_t*>(summaries),
                           page_table, seq_lens, s_hat, s_hat_stride, partials, n_tiles);
    return dispatch_mfma(c.rank, grid, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq,
                         static_cast<const float*>(q), static_cast<const uint8_t*>(summaries),
                         page_table, seq_lens, s_hat, s_hat_stride, partials, n_tiles);
  }
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
