// Summary scan (Sec. 4 "Score", Eq. (1)): for every complete page j of a
// (sequence, KV head) and every query head g of its group,
//   hat s_j(q_g) = log sum_i exp[(q_g^T mu_j + (V_j^T q_g)^T c_i) / sqrt(d)],
// read from the page's stored record (int4 basis, int8 coefficients and centroid,
// float16 scales).  Every block also writes, per query head, the partial
// (max, sum 2^x) of its pages' scores in the log2 domain; the select kernel
// reduces them into log Z_g = log sum_j exp(hat s_j(q_g)).
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

// Chunk of pages a scan block covers (blockIdx.x keeps naming its partials slot).
// Blocks go to the XCDs round-robin by linear block id, x fastest, so chunk c of
// every (sequence, KV head) would sit on XCD c mod 8: the leading chunks, which
// every sequence has, would pile onto the first XCDs when lengths vary (a batch
// with lengths uniform in [8K, 64K] scanned ~1.25x slower than the same pages in
// equal lengths).  Rotating the chunk order by the sequence index spreads them
// out, while the KV heads of one sequence keep one chunk-to-XCD map: their
// records of a page are adjacent, so the cache lines they share stay in one L2
// (rotating by head as well raised the counted fetch bytes by up to a third).
__device__ __forceinline__ int scan_chunk() {
  return (int)((blockIdx.x + blockIdx.z) % gridDim.x);
}

// ---------------------------------------------------------------------------

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));

template <int R, int BB = 0>
struct Geom {
  static constexpr int kPPS = (16 / R) > 0 ? 16 / R : 1;          // pages per stage-1 set
  static constexpr int kSets = (16 + kPPS - 1) / kPPS;
  static constexpr int kColB = rec_col_bytes(BB);                  // bytes per basis column
  static constexpr int kVW = 1 << BB;                              // 16-byte basis loads per lane and set
  static constexpr int kStride = rec_stride(R, BB);
  static constexpr int kTail = kStride - kColB * R;                // coef .. end of record
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

// Log-sum-exp, log2 domain, over lanes {l, l ^ 16} (V = 2) or {l, l ^ 16, l ^ 32,
// l ^ 48} (V = 4); each of those lanes gets the same bits.
template <int V>
__device__ __forceinline__ float merge_sub_lse(float v) {
  auto lse2 = [](float a, float b) {
    const float mx = fmaxf(a, b);
    return mx + __builtin_amdgcn_logf(__builtin_amdgcn_exp2f(a - mx) + __builtin_amdgcn_exp2f(b - mx));
  };
  if (V == 4) {
    auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = lse2(__uint_as_float(p[0]), __uint_as_float(p[1]));
  }
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return lse2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Reduction over the four lanes {l, l^16, l^32, l^48} with two VALU lane swaps.
__device__ __forceinline__ float red4_max(float v) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float red4_sum(float v) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Combines running (max, sum 2^(x - max)) pairs, log2 domain, over the lanes that
// share lane % M; every lane ends with its class's total.
template <int M>
__device__ __forceinline__ void merge_lanes_mod(float& m, float& l) {
#pragma unroll
  for (int o = M; o < 64; o <<= 1) {
    const float om = __shfl_xor(m, o, 64), ol = __shfl_xor(l, o, 64);
    const float mm = fmaxf(m, om);
    l = (mm > -INFINITY)
            ? l * __builtin_amdgcn_exp2f(m - mm) + ol * __builtin_amdgcn_exp2f(om - mm)
            : 0.0f;
    m = mm;
  }
}

template <int R, int BB = 0>
struct TileRegs {
  uint4 vb[BB == 0 ? Geom<R, BB>::kSets : 1][Geom<R, BB>::kVW];  // basis slices (int4: per tile)
  uint4 tl[Geom<R, BB>::kTailLoads];  // record tails, 16-byte chunks
  int blk;                            // lanes 0..15: block of page page0 + lane (-1: none)
};

// The basis slices of stage-1 set st of a tile: lane (grp, col) takes the 32
// elements 32 grp .. 32 grp + 31 of column l = col % R of page st kPPS + col / R
// (16 << BB bytes).
template <int R, int BB>
__device__ __forceinline__ void load_set(uint4* vb, const uint8_t* __restrict__ summaries,
                                         int my_blk, int st, int H_kv, int h, int lane) {
  using Gm = Geom<R, BB>;
  const int col = lane & 15, grp = lane >> 4;
  const int pp = col / R, l = col % R;
  const int page = st * Gm::kPPS + pp;
  const int blk = __shfl(my_blk, page < 16 ? page : 0, 64);
  const bool ok = col < Gm::kPPS * R && page < 16 && blk >= 0;
#pragma unroll
  for (int w = 0; w < Gm::kVW; ++w)
    vb[w] = ok ? *reinterpret_cast<const uint4*>(summaries + ((long)blk * H_kv + h) * Gm::kStride +
                                                 Gm::kColB * l + (16 << BB) * grp + 16 * w)
               : make_uint4(0, 0, 0, 0);
}

// Issue the loads of one 16-page tile (no wait): the record tails, and for an
// int4 basis every stage-1 slice (wider bases load theirs set by set).
template <int R, int BB = 0>
__device__ __forceinline__ void issue_tile(TileRegs<R, BB>& T, const uint8_t* __restrict__ summaries,
                                           const int32_t* __restrict__ pt_row, int page0, int n_c,
                                           int H_kv, int h, int lane) {
  using Gm = Geom<R, BB>;
  const int my_blk = (lane < 16 && page0 + lane < n_c) ? pt_row[page0 + lane] : -1;
  T.blk = my_blk;
  if constexpr (BB == 0) {
#pragma unroll
    for (int st = 0; st < Gm::kSets; ++st) load_set<R, BB>(T.vb[st], summaries, my_blk, st, H_kv, h, lane);
  }
#pragma unroll
  for (int u = 0; u < Gm::kTailLoads; ++u) {
    const int c = lane + 64 * u;
    const int page = c / Gm::kTailCh, off = (c % Gm::kTailCh) * 16;
    const int blk = __shfl(my_blk, page < 16 ? page : 0, 64);
    T.tl[u] = (c < 16 * Gm::kTailCh && blk >= 0)
                  ? *reinterpret_cast<const uint4*>(summaries + ((long)blk * H_kv + h) * Gm::kStride +
                                                    Gm::kColB * R + off)
                  : make_uint4(0, 0, 0, 0);
  }
}

// BB: basis precision (0 int4, 1 int8, 2 bf16).  Wider bases decode their slice
// to f16 in natural element order (int8 codes exactly; bf16 values to the nearest
// f16) and meet the natural-order query operand.
template <typename QT, int R, int BB = 0>
__global__ __launch_bounds__(256) void scan_mfma_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q,
    const uint8_t* __restrict__ summaries, const int32_t* __restrict__ page_table,
    const int32_t* __restrict__ seq_lens, float* __restrict__ s_hat, SHatLayout lay,
    float2* __restrict__ partials) {
  using Gm = Geom<R, BB>;
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
  const int pg = scan_chunk() * 4 + wave;  // 64-page group of this wave
  const long row0 = (long)s * H_q + (long)h * G;
  const int32_t* pt_row = page_table + (long)s * max_pages;
  const int n_parts = gridDim.x;
  float run_m = -INFINITY, run_s = 0.0f;  // running normaliser, log2 domain
  const int npack = 16 / G;                // pages per stage-2 pass
  if (pg * 64 < n_c) {
  TileRegs<R, BB> buf[2];
  issue_tile<R, BB>(buf[0], summaries, pt_row, pg * 64, n_c, H_kv, h, lane);

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

  constexpr float kLn2 = 0.69314718055994531f;
  const float c0 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)
  const int kpass = npack * R;
  const int ksteps = (kpass + 3) / 4;
  const int pcol = col / G, gcol = col % G;
  const bool colvalid = pcol < npack;

#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int page0 = (pg * 4 + t) * 16;
    if (page0 < n_c) {
      TileRegs<R, BB>& cur = buf[t & 1];
      if (t + 1 < 4 && page0 + 16 < n_c)
        issue_tile<R, BB>(buf[(t + 1) & 1], summaries, pt_row, page0 + 16, n_c, H_kv, h, lane);
      // wider bases: every set of this tile in flight at once, ahead of the LDS
      // staging of its tail
      uint4 vall[BB == 0 ? 1 : Gm::kSets][Gm::kVW];
      if constexpr (BB != 0) {
#pragma unroll
        for (int st = 0; st < Gm::kSets; ++st) load_set<R, BB>(vall[st], summaries, cur.blk, st, H_kv, h, lane);
      }
#pragma unroll
      for (int u = 0; u < Gm::kTailLoads; ++u) {
        const int c = lane + 64 * u;
        if (c < 16 * Gm::kTailCh)
          *reinterpret_cast<uint4*>(&sTail[wave][c / Gm::kTailCh][(c % Gm::kTailCh) * 16]) = cur.tl[u];
      }
      __builtin_amdgcn_wave_barrier();

      // ---- stage 1: p = V^T q (scaled by the basis column scales)
#pragma unroll
      for (int st = 0; st < Gm::kSets; ++st) {
        f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        if constexpr (BB == 0) {
          const uint32_t w[4] = {cur.vb[st][0].x, cur.vb[st][0].y, cur.vb[st][0].z, cur.vb[st][0].w};
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
            const h8 a = nib8_to_h8(w[ks]);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bv[ks], acc, 0, 0, 0);
            if (kSplitQ) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bvl[ks], acc, 0, 0, 0);
          }
        } else {
          const uint4* vw = vall[st];
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
            h8 a;
            if constexpr (BB == 1) {
              const uint4 v = vw[ks >> 1];
              a = (ks & 1) ? byte8_to_h8(v.z, v.w) : byte8_to_h8(v.x, v.y);
            } else {
              const uint4 v = vw[ks];
              const uint32_t u[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                a[2 * e] = (_Float16)__uint_as_float(u[e] << 16);
                a[2 * e + 1] = (_Float16)__uint_as_float(u[e] & 0xffff0000u);
              }
            }
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bm[ks], acc, 0, 0, 0);
            if (kSplitQ) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bml[ks], acc, 0, 0, 0);
          }
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
            sA[wave][page][col] =
                acc[j] * inv_qs * c0 * lds_f16(&sTail[wave][page][Gm::kSc + 2 * (R + 16)]);
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
        const float av = sA[wave][pl][gcol];
        const uint2 csw = *reinterpret_cast<const uint2*>(&sTail[wave][pl][Gm::kSc + 2 * (R + 4 * grp)]);
        const h2 cs01 = as_h2(csw.x), cs23 = as_h2(csw.y);
        float z[4];
        z[0] = fmaf((float)cs01.x * c0, acc[0], av);
        z[1] = fmaf((float)cs01.y * c0, acc[1], av);
        z[2] = fmaf((float)cs23.x * c0, acc[2], av);
        z[3] = fmaf((float)cs23.y * c0, acc[3], av);
        float mx = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
        mx = red4_max(mx);
        float sm = __builtin_amdgcn_exp2f(z[0] - mx) + __builtin_amdgcn_exp2f(z[1] - mx) +
                   __builtin_amdgcn_exp2f(z[2] - mx) + __builtin_amdgcn_exp2f(z[3] - mx);
        sm = red4_sum(sm);
        const float s2 = mx + __builtin_amdgcn_logf(sm);  // log2-domain page score
        if (live) {
          if (grp == 0) s_hat[lay.base(s, h) + gcol * lay.head + (long)(page0 + page) * lay.page] = s2 * kLn2;
          const float e = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
          if (s2 > run_m) { run_s = fmaf(run_s, e, 1.0f); run_m = s2; }
          else run_s += e;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  }  // pages of this wave
  // ---- block partial (max, sum exp) per head over its 256 pages (log2 domain)
  if (lane < 16) sRun[wave][lane] = make_float2(run_m, run_s);
  __syncthreads();
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float m = -INFINITY, l = 0.0f;
    for (int w = 0; w < 4; ++w)
      for (int c = g; c < npack * G; c += G) m = fmaxf(m, sRun[w][c].x);
    if (m > -INFINITY)
      for (int w = 0; w < 4; ++w)
        for (int c = g; c < npack * G; c += G) {
          const float2 v = sRun[w][c];
          if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
        }
    partials[(row0 + g) * n_parts + blockIdx.x] = make_float2(m, l);
  }
}

// ---------------------------------------------------------------------------
// Fast path for r in {2, 4, 8} and G in {4, 16} (G = 16 / NPACK); dispatched for
// r in {2, 4} at G = 16 only (r = 8, and G = 4, have the kernels further below).
//
// Differences from the generic kernel above:
//  * stage 1 runs on 16x16x64 int8 MFMA.  A basis nibble becomes an int8 with
//    three ops per eight codes; each query head is written as a 20-bit fixed-point
//    integer (power-of-two scale per head) split into three signed 8-bit digits,
//    and one int32 accumulator takes the digits most significant first, shifted
//    by 8 bits in between (Horner's rule).  The excess-8 bias of the codes is
//    removed exactly by adding -8 * sum(digit) at each stage.  Dot products of
//    codes and queries are therefore exact integers.
//  * stage-1 rows are assigned so that output register j of lane group grp holds
//    slot 4j + grp = (page, basis column); those registers are directly the B
//    operand of stage 2 (block-diagonal over the pages of a pass), so the
//    projections never go through LDS.
//  * every load is unconditional (clamped to a valid record) and 32-bit offset.
// ---------------------------------------------------------------------------

typedef int i4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// The summary store as a raw buffer resource: 32-bit byte offsets, no 64-bit
// address arithmetic per load, and loads past the store's end return zeros.
constexpr int kBufWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t summ_rsrc(const uint8_t* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p), (short)0, (int)bytes, kBufWord3);
}
__device__ __forceinline__ uint4 bld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 bld8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
  return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint32_t bld4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
// Byte offset of the record of (physical block b, KV head h): b * (H_kv * stride)
// + h * stride, with a 24-bit multiply (b < 2^24, the store is below 4 GiB).
__device__ __forceinline__ uint32_t rec_off(int b, uint32_t blk_bytes, uint32_t head_off) {
  return __umul24((uint32_t)b, blk_bytes) + head_off;
}

template <int R>
struct FastGeom {
  static constexpr int kPPS = 16 / R;                 // pages per stage-1 set
  static constexpr int kSets = R;                     // 16 pages x R slots / 16 rows
  static constexpr int kStride = rec_stride(R);
  static constexpr int kTail = kStride - 64 * R;
  static constexpr int kTailCh = kTail / 16;
  static constexpr int kTailLoads = (16 * kTailCh + 63) / 64;
  static constexpr int kMu = 16 * R;
  static constexpr int kSc = 16 * R + kDim;
};

template <int R>
struct FastRegs {
  uint4 vb[FastGeom<R>::kSets];
  uint4 tl[FastGeom<R>::kTailLoads];
};

template <int R>
__device__ __forceinline__ void fast_issue(FastRegs<R>& T, const uint8_t* __restrict__ summ,
                                           const int32_t* __restrict__ pt_row, int page0, int n_c,
                                           int H_kv, int h, int lane) {
  using Gm = FastGeom<R>;
  const int col = lane & 15, grp = lane >> 4;
  const int qs = 4 * (col & 3) + (col >> 2);  // stage-1 slot of A row `col`
  const int a_pp = qs / R, a_l = qs % R;
  // block of page0 + lane (lanes >= 16 and pages past the end reuse page0's block)
  const int pl = page0 + (lane & 15);
  const int my_blk = pt_row[pl < n_c ? pl : page0];
#pragma unroll
  for (int st = 0; st < Gm::kSets; ++st) {
    const int blk = __shfl(my_blk, st * Gm::kPPS + a_pp, 64);
    const uint32_t off = (uint32_t)(blk * H_kv + h) * (uint32_t)Gm::kStride + 64u * a_l + 16u * grp;
    T.vb[st] = *reinterpret_cast<const uint4*>(summ + off);
  }
#pragma unroll
  for (int u = 0; u < Gm::kTailLoads; ++u) {
    int c = lane + 64 * u;
    c = c < 16 * Gm::kTailCh ? c : 16 * Gm::kTailCh - 1;
    const int page = c / Gm::kTailCh, o = (c % Gm::kTailCh) * 16;
    const int blk = __shfl(my_blk, page, 64);
    const uint32_t off = (uint32_t)(blk * H_kv + h) * (uint32_t)Gm::kStride + 64u * R + o;
    T.tl[u] = *reinterpret_cast<const uint4*>(summ + off);
  }
}

// Query digits of head gcol for the int8 projection: q is scaled by a power of
// two to a 20-bit fixed-point integer Q (|Q| < 2^20) and split into three signed
// 8-bit digits (most significant first).  Element e of MFMA half hh <-> d =
// 32 grp + 16 hh + perm16[e], the order in which the decoders expand the packed
// codes.  bias[t] = -8 * sum(digit t) removes the excess-8 offset of the int4
// codes.
//
// The digits are the bytes of U = Q + 0x808080 minus 128: U lies in [0, 2^24),
// byte i of U is digit i + 128, and the lower two digits land in [-128, 127]
// (the balanced base-256 digits of Q).  Four elements' bytes are gathered into
// one digit word per digit by byte permutes, the +128 offsets flipped back by
// one XOR, and each word's digit sum taken by one signed 4-way dot product.
struct QDigits {
  i4v bd[3][2];
  int bias[3];
  float inv_scale;  // fixed-point unit * log2(e) / sqrt(d)
};

template <typename QT>
__device__ __forceinline__ QDigits q_digits(const QT* __restrict__ qrow, int grp) {
  constexpr int kPerm16[16] = {0, 2, 4, 6, 1, 3, 5, 7, 8, 10, 12, 14, 9, 11, 13, 15};
  constexpr float c0 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)
  QDigits D;
  float qf[32];
  float qmax = 0.0f;
#pragma unroll
  for (int c = 0; c < 32; ++c) {
    qf[c] = load_q(qrow + 32 * grp, c);
    qmax = fmaxf(qmax, fabsf(qf[c]));
  }
  qmax = red4_max(qmax);
  int ex = 0;
  (void)frexpf(qmax, &ex);  // qmax < 2^ex
  const float qscale = ldexpf(1.0f, 20 - ex);
  D.inv_scale = ldexpf(1.0f, ex - 20) * c0;
  int bsum[3] = {0, 0, 0};
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
#pragma unroll
    for (int dw = 0; dw < 4; ++dw) {
      uint32_t U[4];
#pragma unroll
      for (int bb = 0; bb < 4; ++bb) {
        const int e = 4 * dw + bb;
        const int Q = (qmax > 0.0f)
                          ? min(max((int)rintf(qf[16 * hh + kPerm16[e]] * qscale), -0xFFFFF), 0xFFFFF)
                          : 0;
        U[bb] = (uint32_t)(Q + 0x808080);
      }
      // bytes (U0.b0, U1.b0, U0.b1, U1.b1), (U0.b2, U1.b2, ..) and the same for U2, U3
      const uint32_t lo01 = __builtin_amdgcn_perm(U[1], U[0], 0x05010400u);
      const uint32_t lo23 = __builtin_amdgcn_perm(U[3], U[2], 0x05010400u);
      const uint32_t hi01 = __builtin_amdgcn_perm(U[1], U[0], 0x07030602u);
      const uint32_t hi23 = __builtin_amdgcn_perm(U[3], U[2], 0x07030602u);
      const uint32_t w2 = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u) ^ 0x80808080u;
      const uint32_t w1 = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u) ^ 0x80808080u;
      const uint32_t w0 = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u) ^ 0x80808080u;
      bsum[0] = __builtin_amdgcn_sdot4((int)w0, 0x01010101, bsum[0], false);
      bsum[1] = __builtin_amdgcn_sdot4((int)w1, 0x01010101, bsum[1], false);
      bsum[2] = __builtin_amdgcn_sdot4((int)w2, 0x01010101, bsum[2], false);
      D.bd[0][hh][dw] = (int)w0;
      D.bd[1][hh][dw] = (int)w1;
      D.bd[2][hh][dw] = (int)w2;
    }
#pragma unroll
  for (int t = 0; t < 3; ++t) D.bias[t] = -8 * (int)red4_sum((float)bsum[t]);
  return D;
}

// A 16-byte basis slice (32 excess-8 nibbles) as the int8 A operands of the two
// K halves.
__device__ __forceinline__ void nib_operands(const uint4& v, i4v (&a)[2]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int hh = 0; hh < 2; ++hh) {
    const uint32_t x0 = w[2 * hh], x1 = w[2 * hh + 1];
    a[hh] = i4v{(int)(x0 & 0x0F0F0F0Fu), (int)((x0 >> 4) & 0x0F0F0F0Fu), (int)(x1 & 0x0F0F0F0Fu),
                (int)((x1 >> 4) & 0x0F0F0F0Fu)};
  }
}

// Exact integer projection sum_d (n_d - 8) Q_d of excess-8 nibble codes n_d onto
// a 20-bit query Q = 2^16 D0 + 2^8 D1 + D2, by Horner's rule over the digits in
// one int32 accumulator: acc = 256 (256 (D0 . n') + D1 . n') + D2 . n'.  Every
// partial value is bounded by |acc| <= 128 * 8 * 2^20 = 2^30, so nothing wraps.
__device__ __forceinline__ i4v proj_horner(const i4v (&a)[2], const QDigits& QD) {
  i4v acc = i4v{QD.bias[0], QD.bias[0], QD.bias[0], QD.bias[0]};
  acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[0], QD.bd[0][0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[1], QD.bd[0][1], acc, 0, 0, 0);
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = (int)(((uint32_t)acc[j] << 8) + (uint32_t)QD.bias[1]);
  acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[0], QD.bd[1][0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[1], QD.bd[1][1], acc, 0, 0, 0);
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = (int)(((uint32_t)acc[j] << 8) + (uint32_t)QD.bias[2]);
  acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[0], QD.bd[2][0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(a[1], QD.bd[2][1], acc, 0, 0, 0);
  return acc;
}

// Two independent projections by the same Horner steps, interleaved so that the
// matrix-core work of one covers the shifts of the other.
__device__ __forceinline__ void proj_horner2(const i4v (&a0)[2], const i4v (&a1)[2],
                                             const QDigits& QD, i4v& r0, i4v& r1) {
  i4v x = i4v{QD.bias[0], QD.bias[0], QD.bias[0], QD.bias[0]};
  i4v y = x;
#pragma unroll
  for (int t = 0; t < 3; ++t) {
    x = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0[0], QD.bd[t][0], x, 0, 0, 0);
    y = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1[0], QD.bd[t][0], y, 0, 0, 0);
    x = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0[1], QD.bd[t][1], x, 0, 0, 0);
    y = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1[1], QD.bd[t][1], y, 0, 0, 0);
    if (t < 2) {
#pragma unroll
      for (int j = 0; j < 4; ++j) x[j] = (int)(((uint32_t)x[j] << 8) + (uint32_t)QD.bias[t + 1]);
#pragma unroll
      for (int j = 0; j < 4; ++j) y[j] = (int)(((uint32_t)y[j] << 8) + (uint32_t)QD.bias[t + 1]);
    }
  }
  r0 = x;
  r1 = y;
}

template <typename QT, int R, int NPACK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void scan_fast_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q, const uint8_t* __restrict__ summ,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    float* __restrict__ s_hat, SHatLayout lay, float2* __restrict__ partials) {
  using Gm = FastGeom<R>;
  constexpr int G = 16 / NPACK;
  constexpr int kPasses = 16 / NPACK;
  constexpr int kKS = (NPACK * R) / 4 > 0 ? (NPACK * R) / 4 : 1;  // k-steps per pass
  __shared__ __align__(16) uint8_t sTail[4][16][Gm::kTail];
  __shared__ float sA[4][16][16];
  __shared__ float2 sRun[4][16];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = blockIdx.y, s = blockIdx.z;
  const int n_c = seq_lens[s] / kPage;
  const int pg = scan_chunk() * 4 + wave;
  const long row0 = (long)s * H_q + (long)h * G;
  const int32_t* pt_row = page_table + (long)s * max_pages;
  const int gcol = col % G, pcol = col / G;
  constexpr float c0 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)
  float run_m = -INFINITY, run_s = 0.0f;

  if (pg * 64 < n_c) {
    FastRegs<R> cur;
    fast_issue<R>(cur, summ, pt_row, pg * 64, n_c, H_kv, h, lane);

    const QDigits QD = q_digits(q + (row0 + gcol) * kDim, grp);
    const float inv_scale = QD.inv_scale;
    const i4v(&bd)[3][2] = QD.bd;

#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int page0 = (pg * 4 + t) * 16;
      if (page0 < n_c) {
#pragma unroll
        for (int u = 0; u < Gm::kTailLoads; ++u) {
          const int c = lane + 64 * u;
          if (c < 16 * Gm::kTailCh)
            *reinterpret_cast<uint4*>(&sTail[wave][c / Gm::kTailCh][(c % Gm::kTailCh) * 16]) = cur.tl[u];
        }
        __builtin_amdgcn_wave_barrier();

        // ---- stage 1 (int8 MFMA): projections of every (page, basis column) slot
        float vals[4 * Gm::kSets];
#pragma unroll
        for (int st = 0; st < Gm::kSets; ++st) {
          if (st % 4 == 0) __builtin_amdgcn_sched_barrier(0);
          i4v a[2];
          nib_operands(cur.vb[st], a);
          const i4v acc = proj_horner(a, QD);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int slot = 4 * j + grp;
            const int page = st * Gm::kPPS + slot / R, l = slot % R;
            const float vs = lds_f16(&sTail[wave][page][Gm::kSc + 2 * l]);
            vals[4 * st + j] = (float)acc[j] * (vs * inv_scale);
          }
        }
        // the record registers are consumed: fetch the next 16 pages into them while
        // the rest of this step runs from LDS and registers
        __builtin_amdgcn_sched_barrier(0);
        if (t + 1 < 4 && page0 + 16 < n_c)
          fast_issue<R>(cur, summ, pt_row, page0 + 16, n_c, H_kv, h, lane);
        __builtin_amdgcn_sched_barrier(0);
        // ---- centroid term (int8 MFMA, one page per row): sA[page][col]
        {
          const uint4 m0 = *reinterpret_cast<const uint4*>(&sTail[wave][col][Gm::kMu + 32 * grp]);
          const uint4 m1 = *reinterpret_cast<const uint4*>(&sTail[wave][col][Gm::kMu + 32 * grp + 16]);
          const uint32_t mw[8] = {m0.x ^ 0x80808080u, m0.y ^ 0x80808080u, m0.z ^ 0x80808080u,
                                  m0.w ^ 0x80808080u, m1.x ^ 0x80808080u, m1.y ^ 0x80808080u,
                                  m1.z ^ 0x80808080u, m1.w ^ 0x80808080u};
          i4v acc[3];
#pragma unroll
          for (int d = 0; d < 3; ++d) acc[d] = i4v{0, 0, 0, 0};
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t y0 = mw[4 * hh], y1 = mw[4 * hh + 1], y2 = mw[4 * hh + 2], y3 = mw[4 * hh + 3];
            const i4v a = {(int)__builtin_amdgcn_perm(y1, y0, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y1, y0, 0x07050301u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x07050301u)};
#pragma unroll
            for (int d = 0; d < 3; ++d)
              acc[d] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, bd[d][hh], acc[d], 0, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int page = 4 * grp + j;
            const float ms = lds_f16(&sTail[wave][page][Gm::kSc + 2 * (R + 16)]);
            const float v = fmaf((float)acc[0][j], 65536.0f, fmaf((float)acc[1][j], 256.0f, (float)acc[2][j]));
            sA[wave][page][col] = v * (ms * inv_scale);
          }
        }
        __builtin_amdgcn_wave_barrier();

        // ---- stage 2 (fp32 MFMA): 16 logits per (page, head), NPACK pages per pass
#pragma unroll
        for (int ps = 0; ps < kPasses; ++ps) {
          if (ps % 4 == 0) __builtin_amdgcn_sched_barrier(0);
          const int pcpage = ps * NPACK + pcol;  // page of this lane's column
          f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
          for (int kk = 0; kk < kKS; ++kk) {
            const int rho = (NPACK * R >= 4) ? ps * kKS + kk : (ps * NPACK * R) / 4;
            const int st = rho / 4, j = rho % 4;
            const int slot = 4 * j + grp;
            const int pk = st * Gm::kPPS + slot / R, l = slot % R;
            const float a = (float)((int)sTail[wave][pk][col * R + l] - 128);
            const float b = (pk == pcpage) ? vals[rho] : 0.0f;
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
          }
          const float av = sA[wave][pcpage][col];
          const uint2 csw = *reinterpret_cast<const uint2*>(&sTail[wave][pcpage][Gm::kSc + 2 * (R + 4 * grp)]);
          const h2 cs01 = as_h2(csw.x), cs23 = as_h2(csw.y);
          float z0 = fmaf((float)cs01.x, acc[0], av), z1 = fmaf((float)cs01.y, acc[1], av);
          float z2 = fmaf((float)cs23.x, acc[2], av), z3 = fmaf((float)cs23.y, acc[3], av);
          float mx = fmaxf(fmaxf(z0, z1), fmaxf(z2, z3));
          mx = red4_max(mx);
          float sm = __builtin_amdgcn_exp2f(z0 - mx) + __builtin_amdgcn_exp2f(z1 - mx) +
                     __builtin_amdgcn_exp2f(z2 - mx) + __builtin_amdgcn_exp2f(z3 - mx);
          sm = red4_sum(sm);
          const float s2 = mx + __builtin_amdgcn_logf(sm);
          const bool live = page0 + pcpage < n_c;
          if (live && grp == 0)
            s_hat[lay.base(s, h) + gcol * lay.head + (long)(page0 + pcpage) * lay.page] = s2 * 0.69314718055994531f;
          const float e = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
          const bool up = s2 > run_m;
          const float ns = up ? fmaf(run_s, e, 1.0f) : run_s + e;
          run_s = live ? ns : run_s;
          run_m = (live && up) ? s2 : run_m;
        }
        __builtin_amdgcn_wave_barrier();
      }
    }
  }
  // ---- block partial (max, sum exp) per head over its 256 pages, log2 domain
  if (lane < 16) sRun[wave][lane] = make_float2(run_m, run_s);
  __syncthreads();
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float m = -INFINITY, l = 0.0f;
    for (int w = 0; w < 4; ++w)
      for (int c = g; c < 16; c += G) m = fmaxf(m, sRun[w][c].x);
    if (m > -INFINITY)
      for (int w = 0; w < 4; ++w)
        for (int c = g; c < 16; c += G) {
          const float2 v = sRun[w][c];
          if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
        }
    partials[(row0 + g) * gridDim.x + blockIdx.x] = make_float2(m, l);
  }
}

// Byte offsets of what this lane loads from the records of the 16 pages whose
// blocks lanes 0..15 hold in `blk`: its basis slice of each set and its record
// tail chunks.  All the lane exchanges of a step are issued together.
//
// Pages of 16 V tokens (V = 2, 4) are scanned as V consecutive 16-token
// sub-pages.  A step then covers 16 / V pages, so only R / V basis sets are
// loaded, and the tail of sub-page u is assembled in the 16-token layout: its
// 16 coefficient rows (16 u .. 16 u + 15), the page's centroid, the basis
// scales, its 16 coefficient row scales and the centroid scale.
template <int R, int V = 1>
struct StepOffs {
  uint32_t vb[FastGeom<R>::kSets / V];
  uint32_t tl[FastGeom<R>::kTailLoads];
};

// Offset inside a record of 16 V-token pages of tail chunk o (16-token layout)
// of sub-page u.
template <int R, int V>
__device__ __forceinline__ uint32_t sub_tail_off(int o, int u) {
  static_assert(V == 1 || R == 8, "sub-pages assume one 16-byte chunk of basis scales");
  constexpr int kCoef = 64 * R, kMu = kCoef + 16 * V * R, kSc = kMu + kDim;
  if (V == 1) return kCoef + 16 * o;
  if (o < R) return kCoef + 16 * R * u + 16 * o;                  // coefficient rows
  if (o < R + 8) return kMu + 16 * (o - R);                        // centroid
  if (o == R + 8) return kSc;                                      // basis scales
  if (o < R + 11) return kSc + 2 * R + 32 * u + 16 * (o - R - 9);  // coefficient row scales
  return kSc + 2 * R + 32 * V;                                     // centroid scale
}

template <int R, int V = 1>
__device__ __forceinline__ StepOffs<R, V> step_offsets(int blk, uint32_t blk_bytes,
                                                       uint32_t head_off, int lane) {
  using Gm = FastGeom<R>;
  const int col = lane & 15, grp = lane >> 4;
  const int qs = 4 * (col & 3) + (col >> 2);
  StepOffs<R, V> o;
#pragma unroll
  for (int st = 0; st < Gm::kSets / V; ++st) {
    const int b = __shfl(blk, (st * Gm::kPPS + qs / R) * V, 64);
    o.vb[st] = rec_off(b, blk_bytes, head_off) + 64u * (qs % R) + 16u * grp;
  }
#pragma unroll
  for (int u = 0; u < Gm::kTailLoads; ++u) {
    int c = lane + 64 * u;
    c = c < 16 * Gm::kTailCh ? c : 16 * Gm::kTailCh - 1;
    const int sp = c / Gm::kTailCh;
    const int b = __shfl(blk, sp, 64);
    o.tl[u] = rec_off(b, blk_bytes, head_off) + sub_tail_off<R, V>(c % Gm::kTailCh, sp % V);
  }
  return o;
}

// Physical block of (sub-)page page0 + (lane & 15); lanes past the end of the
// sequence take page0's block (a valid record that is loaded but not used).
template <int V = 1>
__device__ __forceinline__ int lane_block(const int32_t* __restrict__ pt_row, int page0, int n_c,
                                          int lane) {
  const int pl = page0 + (lane & 15);
  return pt_row[(pl < n_c ? pl : page0) / V];
}

template <int N>
struct IntTag {
  static constexpr int value = N;
};

// ---------------------------------------------------------------------------
// r = 8, G = 16: stage 2 with (page, token) rows.
//
// Stage 1 is the int8 projection above.  Stage 2 reconstructs the logits of
// four pages at a time with one f16 MFMA 16x16x32 (B as hi + lo): rows m are
// (page a = m / 4 of the quad, token 4 ps + m % 4), K index 8 kg + e is (page
// e / 2 of the quad, basis column 4 (e % 2) + kg), so A is block diagonal and B
// is exactly stage-1 registers vals[8 Q + e] of lane group kg.  After the four
// passes of a quad each lane holds all 16 logits of (page 4 Q + grp, head col)
// and takes the page LSE in registers.  The centroid MFMA reads its rows in the
// order page 4 (row & 3) + (row >> 2), which leaves a(page 4 j + grp, head col)
// in register j of the same lanes.  Coefficient rows are copied to LDS with
// their bytes reordered to l = 0, 4, 1, 5, 2, 6, 3, 7, so that the two codes a
// lane needs (l = grp, 4 + grp) are one 16-bit read.  Stage 1 runs per quad
// (basis sets 2 Q, 2 Q + 1, their Horner steps interleaved), and each consumed
// register set is refilled at once with the next 16 pages' records.
// ---------------------------------------------------------------------------
// 16-page steps per wave (a block covers 4 x 16 x kSteps pages): 4 for large
// grids, 1 when four steps would leave most compute units idle.
//
// Pages of 16 V tokens (V = 2, 4) run as V sub-pages each (see StepOffs): a
// step's 16 sub-pages are 16 / V pages, stage 1 runs once per page (R / V basis
// sets per step, in pairs), and the V sub-page LSEs of a page, which sit in
// lanes l, l ^ 16 (and l ^ 32, l ^ 48), are merged before the page's s_hat is
// stored and counted in the normaliser.
template <typename QT, int kSteps, int V = 1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void scan_r8_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q, const uint8_t* __restrict__ summ,
    uint32_t summ_bytes, const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    float* __restrict__ s_hat, SHatLayout lay, float2* __restrict__ partials) {
  constexpr int R = 8;
  using Gm = FastGeom<R>;
  constexpr int G = 16;
  __shared__ __align__(16) uint8_t sTail[4][16][Gm::kTail];
  __shared__ float2 sRun[4][64];
  __shared__ __align__(16) float sVsc[4][16][R];   // basis column scales x the query scale
  __shared__ __align__(16) float sCsc[4][16][16];  // coefficient row scales

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = blockIdx.y, s = blockIdx.z;
  const int n_c = seq_lens[s] / (kPage * V) * V;  // sub-pages of the complete pages
  const int pg = scan_chunk() * 4 + wave;
  const long row0 = (long)s * H_q + (long)h * G;
  const int32_t* pt_row = page_table + (long)s * max_pages;
  float run_m = -INFINITY, run_s = 0.0f;

  constexpr int kWavePages = 16 * kSteps;
  constexpr uint32_t kRecStride = rec_stride(R, 0, kPage * V);
  constexpr int kSetsV = Gm::kSets / V;  // basis sets per step
  if (pg * kWavePages < n_c) {
    const __amdgpu_buffer_rsrc_t rs = summ_rsrc(summ, summ_bytes);
    const uint32_t blk_bytes = (uint32_t)H_kv * kRecStride, head_off = (uint32_t)h * kRecStride;
    const int first = pg * kWavePages;
    const int n_steps = min(kSteps, (n_c - first + 15) / 16);
    uint4 vb[kSetsV];
    uint4 tl[Gm::kTailLoads];
    // the record slices of the step whose pages' blocks lanes 0..15 hold in blk
    auto load_step = [&](int blk) {
      const StepOffs<R, V> o0 = step_offsets<R, V>(blk, blk_bytes, head_off, lane);
#pragma unroll
      for (int st = 0; st < kSetsV; ++st) vb[st] = bld16(rs, o0.vb[st]);
#pragma unroll
      for (int u = 0; u < Gm::kTailLoads; ++u) tl[u] = bld16(rs, o0.tl[u]);
    };
    QDigits QD;  // formed once the first step's loads are in flight
    const int a_row = col >> 2, t_row = col & 3;  // A row of this lane: (page, token)
    // this lane's page score slot of page group grp / V; the wave-uniform page
    // offset is added per quad
    float* shat_lane = s_hat + lay.base(s, h) + (long)col * lay.head + (long)(grp / V) * lay.page;
    i4v pacc[2];  // stage-1 results of the current pair of basis sets

    // kN consecutive steps from page `start` whose first step's slices are
    // loaded (blk_n1: blocks of the second step's pages), fully unrolled so
    // that every wait for a prefetched register counts exactly the loads
    // issued after it
    auto run = [&](int start, auto n_tag, int blk_n1) {
      constexpr int kN = decltype(n_tag)::value;
#pragma unroll
      for (int t = 0; t < kN; ++t) {
        const int page0 = start + 16 * t;
        const bool more = t + 1 < kN;
        const int blk_n2 = t + 2 < kN ? lane_block<V>(pt_row, page0 + 32, n_c, lane) : 0;
        StepOffs<R, V> nx;
        if (more) nx = step_offsets<R, V>(blk_n1, blk_bytes, head_off, lane);
        // ---- record tails to LDS; coefficient rows reordered to l = 0,4,1,5,2,6,3,7
  #pragma unroll
        for (int u = 0; u < Gm::kTailLoads; ++u) {
          const int c = lane + 64 * u;
          if (c < 16 * Gm::kTailCh) {
            const int o = c % Gm::kTailCh;
            uint4 v = tl[u];
            if (o < 8) {
              v = make_uint4(__builtin_amdgcn_perm(v.y, v.x, 0x05010400u),
                             __builtin_amdgcn_perm(v.y, v.x, 0x07030602u),
                             __builtin_amdgcn_perm(v.w, v.z, 0x05010400u),
                             __builtin_amdgcn_perm(v.w, v.z, 0x07030602u));
            }
            *reinterpret_cast<uint4*>(&sTail[wave][c / Gm::kTailCh][o * 16]) = v;
          }
        }
        __builtin_amdgcn_wave_barrier();
        if (more) {
  #pragma unroll
          for (int u = 0; u < Gm::kTailLoads; ++u) tl[u] = bld16(rs, nx.tl[u]);
        }
        // the step's scales in fp32, once for its four quads: basis column scales
        // times the query scale, coefficient row scales
  #pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int e = lane + 64 * u, pgi = e >> 3, l = e & 7;
          sVsc[wave][pgi][l] = lds_f16(&sTail[wave][pgi][Gm::kSc + 2 * l]) * QD.inv_scale;
        }
  #pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int e = lane + 64 * u, pgi = e >> 4, t2 = e & 15;
          sCsc[wave][pgi][t2] = lds_f16(&sTail[wave][pgi][Gm::kSc + 2 * (R + t2)]);
        }
        __builtin_amdgcn_wave_barrier();

        // ---- centroid term: areg[j] = a(page 4 j + grp, head col)
        float areg[4];
        {
          const int cp = 4 * (col & 3) + (col >> 2);
          const uint4 m0 = *reinterpret_cast<const uint4*>(&sTail[wave][cp][Gm::kMu + 32 * grp]);
          const uint4 m1 = *reinterpret_cast<const uint4*>(&sTail[wave][cp][Gm::kMu + 32 * grp + 16]);
          const uint32_t mw[8] = {m0.x ^ 0x80808080u, m0.y ^ 0x80808080u, m0.z ^ 0x80808080u,
                                  m0.w ^ 0x80808080u, m1.x ^ 0x80808080u, m1.y ^ 0x80808080u,
                                  m1.z ^ 0x80808080u, m1.w ^ 0x80808080u};
          i4v acc[3];
  #pragma unroll
          for (int d = 0; d < 3; ++d) acc[d] = i4v{0, 0, 0, 0};
  #pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t y0 = mw[4 * hh], y1 = mw[4 * hh + 1], y2 = mw[4 * hh + 2], y3 = mw[4 * hh + 3];
            const i4v a = {(int)__builtin_amdgcn_perm(y1, y0, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y1, y0, 0x07050301u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x07050301u)};
  #pragma unroll
            for (int d = 0; d < 3; ++d)
              acc[d] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, QD.bd[d][hh], acc[d], 0, 0, 0);
          }
  #pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float ms = lds_f16(&sTail[wave][4 * j + grp][Gm::kSc + 2 * (R + 16)]);
            const float v = fmaf((float)acc[0][j], 65536.0f, (float)(acc[1][j] * 256 + acc[2][j]));
            areg[j] = v * (ms * QD.inv_scale);
          }
        }

  #pragma unroll
        for (int Q = 0; Q < 4; ++Q) {
          __builtin_amdgcn_sched_barrier(0);
          // ---- stage 1 (int8 MFMA), basis sets 2 m, 2 m + 1 for pair m = Q / V
          //      (register j of set st: p(page 2 st + j / 2, l = 4 (j % 2) + grp));
          //      vals[4 i + j] = p(sub-page 4 Q + 2 i + j / 2, l = 4 (j % 2) + grp)
          float vals[8];
          {
            const int m = Q / V;
            if (Q % V == 0) {
              i4v a0[2], a1[2];
              nib_operands(vb[2 * m], a0);
              nib_operands(vb[2 * m + 1], a1);
              proj_horner2(a0, a1, QD, pacc[0], pacc[1]);
              if (more) {
                vb[2 * m] = bld16(rs, nx.vb[2 * m]);
                vb[2 * m + 1] = bld16(rs, nx.vb[2 * m + 1]);
              }
            }
  #pragma unroll
            for (int i = 0; i < 2; ++i)
  #pragma unroll
              for (int j = 0; j < 4; ++j) {
                const int sp = 4 * Q + 2 * i + j / 2, pv = sp / V, l = 4 * (j % 2) + grp;
                vals[4 * i + j] = (float)pacc[pv / 2 - 2 * m][2 * (pv % 2) + j % 2] * sVsc[wave][sp][l];
              }
          }
          // ---- stage 2 for the quad, then the page LSE in registers
          h8 bh, bl;
  #pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const auto hi = __builtin_amdgcn_cvt_pkrtz(vals[e], vals[e + 1]);
            const auto lo = __builtin_amdgcn_cvt_pkrtz(vals[e] - (float)hi[0], vals[e + 1] - (float)hi[1]);
            bh[e] = hi[0];
            bh[e + 1] = hi[1];
            bl[e] = lo[0];
            bl[e + 1] = lo[1];
          }
          float z[16];
  #pragma unroll
          for (int ps = 0; ps < 4; ++ps) {
            const uint32_t pr = *reinterpret_cast<const uint16_t*>(
                &sTail[wave][4 * Q + a_row][(4 * ps + t_row) * R + 2 * grp]);
            const h2 pair = as_h2(__builtin_amdgcn_perm(0x64646464u, pr, 0x05010400u)) -
                            h2{(_Float16)1152.0f, (_Float16)1152.0f};
            const uint32_t pw = __builtin_bit_cast(uint32_t, pair);
            const uint4 aw = make_uint4(a_row == 0 ? pw : 0u, a_row == 1 ? pw : 0u,
                                        a_row == 2 ? pw : 0u, a_row == 3 ? pw : 0u);
            const h8 A = __builtin_bit_cast(h8, aw);
            f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, bh, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, bl, acc, 0, 0, 0);
            const float4 cs4 = *reinterpret_cast<const float4*>(&sCsc[wave][4 * Q + grp][4 * ps]);
            z[4 * ps + 0] = cs4.x * acc[0];
            z[4 * ps + 1] = cs4.y * acc[1];
            z[4 * ps + 2] = cs4.z * acc[2];
            z[4 * ps + 3] = cs4.w * acc[3];
          }
          // z are the logits minus the centroid logit a.  The deviations of a
          // page's tokens sum to ~0 (the coefficient columns are orthogonal to
          // the all-ones vector), so the largest is >= ~0 and sum 2^z is safe
          // without a max; a max-shifted sum is taken only if it is not finite.
          float ez[16];
  #pragma unroll
          for (int i = 0; i < 16; ++i) ez[i] = __builtin_amdgcn_exp2f(z[i]);
  #pragma unroll
          for (int w = 1; w < 16; w <<= 1)  // pairwise: four dependent adds, not fifteen
  #pragma unroll
            for (int i = 0; i < 16; i += 2 * w) ez[i] += ez[i + w];
          float sm = ez[0];
          float shift = 0.0f;
          if (!(sm > 0.0f && sm < INFINITY)) {
            shift = z[0];
  #pragma unroll
            for (int i = 1; i < 16; ++i) shift = fmaxf(shift, z[i]);
            sm = 0.0f;
  #pragma unroll
            for (int i = 0; i < 16; ++i) sm += __builtin_amdgcn_exp2f(z[i] - shift);
          }
          float s2 = areg[Q] + shift + __builtin_amdgcn_logf(sm);
          const int sub = page0 + 4 * Q + grp;
          const bool live = sub < n_c && grp % V == 0;
          if (V > 1) s2 = merge_sub_lse<V>(s2);
          if (live) shat_lane[(long)((page0 + 4 * Q) / V) * lay.page] = s2 * 0.69314718055994531f;
          const float e = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
          const bool up = s2 > run_m;
          const float ns = up ? fmaf(run_s, e, 1.0f) : run_s + e;
          run_s = live ? ns : run_s;
          run_m = (live && up) ? s2 : run_m;
        }
        blk_n1 = blk_n2;
        __builtin_amdgcn_wave_barrier();
      }
    };
    if (n_steps == kSteps) {
      load_step(lane_block<V>(pt_row, first, n_c, lane));
      const int blk1 = kSteps > 1 ? lane_block<V>(pt_row, first + 16, n_c, lane) : 0;
      QD = q_digits(q + (row0 + col) * kDim, grp);
      run(first, IntTag<kSteps>{}, blk1);
    } else {
      QD = q_digits(q + (row0 + col) * kDim, grp);
#pragma unroll 1
      for (int t = 0; t < n_steps; ++t) {
        load_step(lane_block<V>(pt_row, first + 16 * t, n_c, lane));
        run(first + 16 * t, IntTag<1>{}, 0);
      }
    }
  }
  // ---- block partial (max, sum exp) per head over its pages, log2 domain: lane
  // l holds head l % 16; the wave's lanes are merged first
  merge_lanes_mod<16>(run_m, run_s);
  if (lane < G) sRun[wave][lane] = make_float2(run_m, run_s);
  __syncthreads();
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float m = -INFINITY, l = 0.0f;
    for (int w = 0; w < 4; ++w) m = fmaxf(m, sRun[w][g].x);
    if (m > -INFINITY)
      for (int w = 0; w < 4; ++w) {
        const float2 v = sRun[w][g];
        if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
      }
    partials[(row0 + g) * gridDim.x + blockIdx.x] = make_float2(m, l);
  }
}

// ---------------------------------------------------------------------------
// r = 8, G = 4: stage 2 with a block-diagonal B.
//
// A wave covers 16 pages per step, as four quads of 4 pages; every operand is
// loaded straight from the records into the register layout it is used in.
// For quad Q:
//  * stage 1 (int8 MFMA, two basis sets i = 0, 1): A row m is (page 4 Q + m / 4,
//    basis column 4 i + m % 4); the 16 B columns are the 4 heads repeated 4
//    times.  Lane (grp, col) receives p(page 4 Q + grp, l = 4 i + j, head col % 4)
//    in register j, so its 8 values over both sets are the basis projections of
//    one (page, head) in natural l order.
//  * stage 2 (f16 MFMA 16x16x32, B as hi + lo): rows are the 16 tokens, K index
//    8 a + l is (page 4 Q + a, basis column l), columns are (a, g) = (col / 4,
//    col % 4).  B is block diagonal: a lane contributes its 8 stage-1 values
//    where grp == col / 4 and zeros elsewhere (its scale factor is zero), A is
//    the coefficient row of token col of page 4 Q + grp.  Register j of lane
//    (grp, col) is then the logit of token 4 grp + j of page 4 Q + col / 4 for
//    head col % 4, minus the centroid logit.
//  * page LSE: 4 values per lane, then the 4 lanes of a column.
// The centroid MFMA (once per step) puts page 4 (m % 4) + m / 4 in row m, so
// register Q of lane (grp, col) holds a(page 4 Q + grp, head col % 4): the
// centroid of the lanes with grp == col / 4, which keep the result.
//
// Pages of 16 V tokens (V = 2, 4) run as V sub-pages of 16 tokens (coefficient
// rows and row scales 16 u .. 16 u + 15 of sub-page u, the page's basis and
// centroid).  Stage 1 then runs once per four pages: at V = 4 a quad is one
// page, lane (grp, col) gets p(page grp of the step, l, head g), and three row
// swaps (16 and 32 lanes) broadcast page u's rows for quad u; at V = 2 a pass
// covers two quads, its rows ordered so that one 16-lane swap yields both quads'
// layouts.  The sub-page LSEs of a page sit in the diagonal lanes 20 a + g (a
// the quad's sub-page) and are merged with lane exchanges at distance 20 and 40.
// ---------------------------------------------------------------------------

// Block of (sub-)page min(page0 + (lane & 15), n_c - 1): always a valid page of
// the sequence.
template <int V = 1>
__device__ __forceinline__ int lane_block_clamped(const int32_t* __restrict__ pt_row, int page0,
                                                  int n_c, int lane) {
  const int pl = page0 + (lane & 15);
  return pt_row[(pl < n_c ? pl : n_c - 1) / V];
}

// Log-sum-exp, log2 domain, of the sub-page values in lanes l, l ^ 20 (V = 2) and
// l ^ 40, l ^ 60 (V = 4); each of those lanes gets the same bits.
template <int V>
__device__ __forceinline__ float merge_diag_lse(float v) {
  auto lse2 = [](float a, float b) {
    const float mx = fmaxf(a, b);
    return mx + __builtin_amdgcn_logf(__builtin_amdgcn_exp2f(a - mx) + __builtin_amdgcn_exp2f(b - mx));
  };
  v = lse2(v, __shfl_xor(v, 20, 64));
  if (V == 4) v = lse2(v, __shfl_xor(v, 40, 64));
  return v;
}

template <typename QT, int kSteps, int V = 1>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void scan_r8g4_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q, const uint8_t* __restrict__ summ,
    uint32_t summ_bytes, const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    float* __restrict__ s_hat, SHatLayout lay, float2* __restrict__ partials) {
  constexpr int R = 8, G = 4, P = kPage * V;
  constexpr uint32_t kStride = rec_stride(R, 0, P);
  constexpr uint32_t kCoef = rec_coef_off(R), kMu = rec_mu_off(R, 0, P), kSc = rec_scale_off(R, 0, P);
  __shared__ float2 sRun[4][64];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = blockIdx.y, s = blockIdx.z;
  const int n_c = seq_lens[s] / P * V;  // sub-pages of the complete pages
  const int pg = scan_chunk() * 4 + wave;
  const long row0 = (long)s * H_q + (long)h * G;
  const int32_t* pt_row = page_table + (long)s * max_pages;
  const int ca = col >> 2, g = col & 3;
  const bool diag = grp == ca;
  // sub-page of the pages this lane reads through ra (4 Q + ca) and rb (4 Q + grp)
  const uint32_t sub_a = (uint32_t)(ca % V), sub_b = (uint32_t)(grp % V);
  float run_m = -INFINITY, run_s = 0.0f;

  constexpr int kWavePages = 16 * kSteps;
  const int first = pg * kWavePages;
  if (first < n_c) {
    const int n_steps = min(kSteps, (n_c - first + 15) / 16);
    // the query digits are formed once the first step's loads are in flight
    QDigits QD;
    float inv_m = 0.0f;  // scale of the stage-1 values; zero off the block diagonal of B
    auto form_digits = [&]() {
      QD = q_digits(q + (row0 + g) * kDim, grp);
      inv_m = diag ? QD.inv_scale : 0.0f;
    };
    // this lane's page score slot of page group ca / V; the wave-uniform page
    // offset is added per quad
    float* shat_lane = s_hat + lay.base(s, h) + (long)g * lay.head + (long)(ca / V) * lay.page;

    // record offsets of one step: ra[Q] page 4 Q + ca, rb[Q] page 4 Q + grp,
    // rm page 4 g + ca (the centroid row of this lane); when stage 1 is shared
    // (V > 1), pa[m] and pb[m] are the records of the pages of pass m in rows
    // ca and grp: pages 4 m + x at V = 4, pages 4 m + ((x & 1) << 1 | x >> 1) at
    // V = 2 (rows ordered 0, 2, 1, 3 so that one 16-lane swap splits the pass
    // into its two quads)
    constexpr int kShare = V;  // quads per stage-1 pass
    constexpr int kPasses = 4 / kShare;
    struct Offs {
      uint32_t ra[4], rb[4], rm;
      uint32_t pa[kPasses], pb[kPasses];
    };
    const __amdgpu_buffer_rsrc_t rs = summ_rsrc(summ, summ_bytes);
    const uint32_t blk_bytes = (uint32_t)H_kv * kStride, head_off = (uint32_t)h * kStride;
    auto offsets = [&](int blk) {
      Offs o;
      auto rec = [&](int page) { return rec_off(__shfl(blk, page, 64), blk_bytes, head_off); };
#pragma unroll
      for (int Q = 0; Q < 4; ++Q) {
        o.ra[Q] = rec(4 * Q + ca);
        o.rb[Q] = rec(4 * Q + grp);
      }
      o.rm = rec(4 * g + ca);
      if constexpr (kShare > 1) {
        auto row_page = [](int x) { return V == 2 ? ((x & 1) << 1 | x >> 1) : x; };
#pragma unroll
        for (int m = 0; m < kPasses; ++m) {
          o.pa[m] = rec((4 * m + row_page(ca)) * V);
          o.pb[m] = rec((4 * m + row_page(grp)) * V);
        }
      }
      return o;
    };
    uint4 vb[kPasses][2];  // basis rows of stage-1 pass m (quad m if V = 1), set i
    uint2 cf[4];       // coefficient row `col` of page 4 Q + grp
    uint2 cs[4];       // row scales of tokens 4 grp .. 4 grp + 3 of page 4 Q + ca
    uint4 vs[kPasses];     // basis column scales of the pass's page grp
    uint32_t msw[4];   // centroid scale of page 4 Q + grp (low half)
    uint4 mu[2];       // centroid bytes 32 grp .. 32 grp + 31 of page 4 g + ca
    // loads of one step's registers; in a run the next step's are issued right
    // after the register's last use in the current one
    auto ld_vb = [&](const Offs& o, int m, int i) {
      vb[m][i] = bld16(rs, (kShare == 1 ? o.ra[m] : o.pa[m]) + 64u * (4 * i + g) + 16u * grp);
    };
    auto ld_cf = [&](const Offs& o, int Q) {
      cf[Q] = bld8(rs, o.rb[Q] + kCoef + 8u * (16u * sub_b + col));
    };
    auto ld_cs = [&](const Offs& o, int Q) {
      cs[Q] = bld8(rs, o.ra[Q] + kSc + 2u * (R + 16u * sub_a + 4 * grp));
    };
    auto ld_vs = [&](const Offs& o, int m) {
      vs[m] = bld16(rs, (kShare == 1 ? o.rb[m] : o.pb[m]) + kSc);
    };
    auto ld_ms = [&](const Offs& o, int Q) { msw[Q] = bld4(rs, o.rb[Q] + kSc + 2u * (R + P)); };
    auto ld_mu = [&](const Offs& o) {
      mu[0] = bld16(rs, o.rm + kMu + 32u * grp);
      mu[1] = bld16(rs, o.rm + kMu + 32u * grp + 16u);
    };

    // every register of the step whose pages' blocks lanes 0..15 hold in blk
    auto load_step = [&](int blk) {
      const Offs o0 = offsets(blk);
      ld_mu(o0);
#pragma unroll
      for (int Q = 0; Q < 4; ++Q) {
        if (Q < kPasses) {
          ld_vb(o0, Q, 0);
          ld_vb(o0, Q, 1);
          ld_vs(o0, Q);
        }
        ld_cf(o0, Q);
        ld_ms(o0, Q);
        ld_cs(o0, Q);
      }
    };

    // kN consecutive 16-page steps from page `start` whose first step's
    // registers are loaded (blk_next: blocks of the second step's pages), fully
    // unrolled so that every wait for a prefetched register counts exactly the
    // loads issued after it
    auto run = [&](int start, auto n_tag, int blk_next) {
      constexpr int kN = decltype(n_tag)::value;
#pragma unroll
      for (int t = 0; t < kN; ++t) {
        const bool pf = t + 1 < kN;
        const int page0 = start + 16 * t;
        Offs on;
        int blk_after = 0;
        if (pf) {
          on = offsets(blk_next);
          if (t + 2 < kN) blk_after = lane_block_clamped<V>(pt_row, page0 + 32, n_c, lane);
        }

        // ---- centroid term: areg[j] = a(page 4 j + grp, head g) / (scale of that page)
        float areg[4];
        {
          const uint32_t mw[8] = {mu[0].x ^ 0x80808080u, mu[0].y ^ 0x80808080u,
                                  mu[0].z ^ 0x80808080u, mu[0].w ^ 0x80808080u,
                                  mu[1].x ^ 0x80808080u, mu[1].y ^ 0x80808080u,
                                  mu[1].z ^ 0x80808080u, mu[1].w ^ 0x80808080u};
          if (pf) ld_mu(on);
          i4v acc[3];
#pragma unroll
          for (int d = 0; d < 3; ++d) acc[d] = i4v{0, 0, 0, 0};
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t y0 = mw[4 * hh], y1 = mw[4 * hh + 1], y2 = mw[4 * hh + 2], y3 = mw[4 * hh + 3];
            const i4v a = {(int)__builtin_amdgcn_perm(y1, y0, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y1, y0, 0x07050301u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x07050301u)};
#pragma unroll
            for (int d = 0; d < 3; ++d)
              acc[d] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, QD.bd[d][hh], acc[d], 0, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j)
            areg[j] = fmaf((float)acc[0][j], 65536.0f, (float)(acc[1][j] * 256 + acc[2][j]));
        }

        float bq[kShare][8];  // shared stage 1: the values of the step's quads
#pragma unroll
        for (int Q = 0; Q < 4; ++Q) {
          __builtin_amdgcn_sched_barrier(0);
          // ---- stage 1: vals[4 i + j] = p(page 4 Q + grp, l = 4 i + j, head g), zero off-diagonal
          float vals[8];
          if (Q % kShare == 0) {
            const int m = Q / kShare;
            i4v acc1[2];
            {
              i4v a0[2], a1[2];
              nib_operands(vb[m][0], a0);
              nib_operands(vb[m][1], a1);
              proj_horner2(a0, a1, QD, acc1[0], acc1[1]);
              if (pf) {
                ld_vb(on, m, 0);
                ld_vb(on, m, 1);
              }
            }
            const uint32_t vsw[4] = {vs[m].x, vs[m].y, vs[m].z, vs[m].w};
            const float sc = kShare == 1 ? inv_m : QD.inv_scale;
#pragma unroll
            for (int l = 0; l < 8; ++l) {
              const int j = l & 3;
              const h2 pr = as_h2(vsw[l >> 1]);
              const float vsc = (float)((l & 1) ? pr.y : pr.x);
              vals[l] = (float)acc1[l >> 2][j] * (vsc * sc);
            }
            if (pf) ld_vs(on, m);
            if constexpr (kShare > 1) {
              // the 16-lane swap of rows r0..r3 (lanes 16 u ..) gives X = (r0, r0,
              // r2, r2) and Y = (r1, r1, r3, r3).  V = 4: rows hold pages 0..3 and
              // the 32-lane swaps of X and Y put each row everywhere.  V = 2: rows
              // hold pages 4 m + 0, 2, 1, 3, so X is quad 2 m's layout (pages
              // 4 m, 4 m, 4 m + 1, 4 m + 1) and Y quad 2 m + 1's.
#pragma unroll
              for (int l = 0; l < 8; ++l) {
                const uint32_t x = __float_as_uint(vals[l]);
                const auto xy = __builtin_amdgcn_permlane16_swap(x, x, false, false);
                if constexpr (V == 4) {
                  const auto xx = __builtin_amdgcn_permlane32_swap(xy[0], xy[0], false, false);
                  const auto yy = __builtin_amdgcn_permlane32_swap(xy[1], xy[1], false, false);
                  bq[0][l] = __uint_as_float(xx[0]);
                  bq[1][l] = __uint_as_float(yy[0]);
                  bq[2][l] = __uint_as_float(xx[1]);
                  bq[3][l] = __uint_as_float(yy[1]);
                } else {
                  bq[0][l] = __uint_as_float(xy[0]);
                  bq[1][l] = __uint_as_float(xy[1]);
                }
              }
            }
          }
          if constexpr (kShare > 1) {
#pragma unroll
            for (int l = 0; l < 8; ++l) vals[l] = diag ? bq[Q % kShare][l] : 0.0f;
          }
          const h8 A = byte8_to_h8(cf[Q].x, cf[Q].y);
          if (pf) ld_cf(on, Q);
          const float am = areg[Q] * ((float)as_h2(msw[Q]).x * QD.inv_scale);
          if (pf) ld_ms(on, Q);
          // ---- stage 2 for the quad
          h8 bh, bl;
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const auto hi = __builtin_amdgcn_cvt_pkrtz(vals[e], vals[e + 1]);
            const auto lo = __builtin_amdgcn_cvt_pkrtz(vals[e] - (float)hi[0], vals[e + 1] - (float)hi[1]);
            bh[e] = hi[0];
            bh[e + 1] = hi[1];
            bl[e] = lo[0];
            bl[e + 1] = lo[1];
          }
          f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, bh, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, bl, acc, 0, 0, 0);
          const h2 c01 = as_h2(cs[Q].x), c23 = as_h2(cs[Q].y);
          float z[4] = {(float)c01.x * acc[0], (float)c01.y * acc[1], (float)c23.x * acc[2],
                        (float)c23.y * acc[3]};
          if (pf) ld_cs(on, Q);
          // z are the logits minus the centroid logit (sum over a page's tokens
          // ~0, so sum 2^z needs no max); a max-shifted sum is taken if any
          // lane's sum is not finite and positive.
          float sm = __builtin_amdgcn_exp2f(z[0]) + __builtin_amdgcn_exp2f(z[1]) +
                     __builtin_amdgcn_exp2f(z[2]) + __builtin_amdgcn_exp2f(z[3]);
          sm = red4_sum(sm);
          float shift = 0.0f;
          if (__any(!(sm > 0.0f && sm < INFINITY))) {
            shift = red4_max(fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3])));
            sm = __builtin_amdgcn_exp2f(z[0] - shift) + __builtin_amdgcn_exp2f(z[1] - shift) +
                 __builtin_amdgcn_exp2f(z[2] - shift) + __builtin_amdgcn_exp2f(z[3] - shift);
            sm = red4_sum(sm);
          }
          float s2 = am + shift + __builtin_amdgcn_logf(sm);
          const int sub = page0 + 4 * Q + ca;
          const bool live = diag && sub < n_c && ca % V == 0;
          if (V > 1) s2 = merge_diag_lse<V>(s2);
          if (live) shat_lane[(long)((page0 + 4 * Q) / V) * lay.page] = s2 * 0.69314718055994531f;
          const float e = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
          const bool up = s2 > run_m;
          const float ns = up ? fmaf(run_s, e, 1.0f) : run_s + e;
          run_s = live ? ns : run_s;
          run_m = (live && up) ? s2 : run_m;
        }
        blk_next = blk_after;
      }
    };
    if (n_steps == kSteps) {
      const int blk0 = lane_block_clamped<V>(pt_row, first, n_c, lane);
      const int blk1 = kSteps > 1 ? lane_block_clamped<V>(pt_row, first + 16, n_c, lane) : 0;
      load_step(blk0);
      form_digits();
      run(first, IntTag<kSteps>{}, blk1);
    } else {
      form_digits();
#pragma unroll 1
      for (int t = 0; t < n_steps; ++t) {
        load_step(lane_block_clamped<V>(pt_row, first + 16 * t, n_c, lane));
        run(first + 16 * t, IntTag<1>{}, 0);
      }
    }
  }
  // ---- block partial (max, sum exp) per head over its pages, log2 domain: lane
  // l holds head l % 4; the wave's lanes are merged first
  merge_lanes_mod<4>(run_m, run_s);
  if (lane < G) sRun[wave][lane] = make_float2(run_m, run_s);
  __syncthreads();
  if (threadIdx.x < G) {
    const int gg = threadIdx.x;
    float m = -INFINITY, l = 0.0f;
    for (int w = 0; w < 4; ++w) m = fmaxf(m, sRun[w][gg].x);
    if (m > -INFINITY)
      for (int w = 0; w < 4; ++w) {
        const float2 v = sRun[w][gg];
        if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
      }
    partials[(row0 + gg) * gridDim.x + blockIdx.x] = make_float2(m, l);
  }
}

// ---------------------------------------------------------------------------
// Low rank (r in {2, 4}), G = 4: projections on the matrix cores, logits on the
// vector ALU.
//
// A wave covers 16 pages per step.  The step's 16 records are gathered whole by
// 16-byte buffer loads and parked in the wave's LDS slot; the loads of the next
// step are issued right after, so they are in flight for the whole step (the
// scan is bound by memory latency at these record sizes, not by arithmetic).
// Stage 1 (int8 MFMA, Horner over the query digits) has rows (page, basis
// column) -- 16 / R pages per tile -- and the 4 heads repeated over the 16
// columns; lanes of columns 0..3 scale their projections and leave them in LDS,
// next to the centroid terms.  Stage 2 gives every lane one (page, head) pair:
// z_i = a + s_i sum_l (c_il - 128) p_l for the 16 tokens in fp32 (the
// excess-128 offset enters as one subtraction of 128 sum_l p_l), the page LSE in
// registers, and a coalesced store of the page score.
// ---------------------------------------------------------------------------
constexpr int kLowSteps = 4;  // 16-page steps per wave: a block covers 256 pages

template <typename QT, int R>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 4))) void scan_low_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q, const uint8_t* __restrict__ summ,
    uint32_t summ_bytes, const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    float* __restrict__ s_hat, SHatLayout lay, float2* __restrict__ partials) {
  constexpr int G = 4;
  constexpr int kPPT = 16 / R;                        // pages per stage-1 tile
  constexpr uint32_t kStride = rec_stride(R);
  constexpr int kCh = kStride / 16;                   // 16-byte chunks per record
  constexpr int kLoads = (16 * kCh + 63) / 64;        // chunk loads per lane and step
  constexpr int kCoef = rec_coef_off(R), kMu = rec_mu_off(R), kSc = rec_scale_off(R);
  __shared__ __align__(16) uint8_t sRec[4][16][kStride];
  __shared__ __align__(16) float sP[4][16][G][R];
  __shared__ float sA[4][16][G];
  __shared__ float2 sRun[4][64];
  __shared__ __align__(16) i4v sQ[3][2][64];  // query digit operands, shared by the waves

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = blockIdx.y, s = blockIdx.z;
  const int n_c = seq_lens[s] / kPage;
  const long row0 = (long)s * H_q + (long)h * G;
  constexpr int kWavePages = 16 * kLowSteps;
  if (scan_chunk() * 4 * kWavePages >= n_c) {  // no complete page in this block
    if (threadIdx.x < G)
      partials[(row0 + threadIdx.x) * gridDim.x + blockIdx.x] = make_float2(-INFINITY, 0.0f);
    return;
  }
  const int pg = scan_chunk() * 4 + wave;
  const int first = pg * kWavePages;
  const bool has = first < n_c;
  const int32_t* pt_row = page_table + (long)s * max_pages;
  const int pp = lane >> 2, gg = lane & 3;            // stage 2: (page, head) of this lane
  float run_m = -INFINITY, run_s = 0.0f;

  const __amdgpu_buffer_rsrc_t rs = summ_rsrc(summ, summ_bytes);
  const uint32_t blk_bytes = (uint32_t)H_kv * kStride, head_off = (uint32_t)h * kStride;
  // blocks of the wave's 64 pages, page first + l in lane l (pages past the end
  // repeat the last complete one)
  const int blk_all = has ? pt_row[min(first + lane, n_c - 1)] : 0;
  // chunk c = lane + 64 u of step t is chunk c % kCh of page 16 t + c / kCh; it
  // lands at byte 16 c of the wave's LDS slot
  auto issue = [&](int t, uint4 (&ld)[kLoads]) {
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      int c = lane + 64 * u;
      c = c < 16 * kCh ? c : 16 * kCh - 1;
      const int b = __shfl(blk_all, 16 * t + c / kCh, 64);
      ld[u] = bld16(rs, rec_off(b, blk_bytes, head_off) + (c % kCh) * 16);
    }
  };
  // the query digits (identical for the four waves) stay in LDS and are read at
  // each use, leaving the registers to the loads in flight
  int bias[3];
  float inv_scale;
  {
    const QDigits QD = q_digits(q + (row0 + (col & 3)) * kDim, grp);
    if (wave == 0) {
#pragma unroll
      for (int d = 0; d < 3; ++d)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) sQ[d][hh][lane] = QD.bd[d][hh];
    }
#pragma unroll
    for (int d = 0; d < 3; ++d) bias[d] = QD.bias[d];
    inv_scale = QD.inv_scale;
  }
  // the first step's records (the page-table load was in flight while the
  // digits were formed)
  uint4 ld[kLoads];
  if (has) issue(0, ld);
  __syncthreads();
  // (the empty asm makes every use a fresh LDS read: hoisted out of the step loop
  // the operands would take 24 registers again)
  auto qop = [&](int d, int hh) {
    int li = lane;
    asm volatile("" : "+v"(li));
    return sQ[d][hh][li];
  };

  if (has) {
    const int n_steps = min(kLowSteps, (n_c - first + 15) / 16);
    float* shat_base = s_hat + lay.base(s, h) + (long)gg * lay.head;
    uint8_t* slot = &sRec[wave][0][0];

    // the wave's kN steps, fully unrolled so that each wait for a step's records
    // counts exactly the memory operations issued after them (the first step's
    // loads are in ld); the page score of a step is stored after the next step's
    // loads are issued
    auto run = [&](auto n_tag) {
      constexpr int kN = decltype(n_tag)::value;
      float st_val = 0.0f;
      int st_page = -1;
#pragma unroll
      for (int t = 0; t < kN; ++t) {
        const int page0 = first + 16 * t;
        // ---- this step's records to LDS, then the next step's loads
#pragma unroll
        for (int u = 0; u < kLoads; ++u) {
          const int c = lane + 64 * u;
          if (c < 16 * kCh) *reinterpret_cast<uint4*>(slot + 16 * c) = ld[u];
        }
        __builtin_amdgcn_wave_barrier();
        if (t + 1 < kN) issue(t + 1, ld);
        if (t > 0 && st_page >= 0) shat_base[(long)st_page * lay.page] = st_val;
        // ---- centroid term (one page per row; int8 codes: three digit chains)
        {
          const uint4 m0 = *reinterpret_cast<const uint4*>(&sRec[wave][col][kMu + 32 * grp]);
          const uint4 m1 = *reinterpret_cast<const uint4*>(&sRec[wave][col][kMu + 32 * grp + 16]);
          const uint32_t mw[8] = {m0.x ^ 0x80808080u, m0.y ^ 0x80808080u, m0.z ^ 0x80808080u,
                                  m0.w ^ 0x80808080u, m1.x ^ 0x80808080u, m1.y ^ 0x80808080u,
                                  m1.z ^ 0x80808080u, m1.w ^ 0x80808080u};
          i4v acc[3];
  #pragma unroll
          for (int d = 0; d < 3; ++d) acc[d] = i4v{0, 0, 0, 0};
  #pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const uint32_t y0 = mw[4 * hh], y1 = mw[4 * hh + 1], y2 = mw[4 * hh + 2], y3 = mw[4 * hh + 3];
            const i4v a = {(int)__builtin_amdgcn_perm(y1, y0, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y1, y0, 0x07050301u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x06040200u),
                           (int)__builtin_amdgcn_perm(y3, y2, 0x07050301u)};
  #pragma unroll
            for (int d = 0; d < 3; ++d)
              acc[d] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, qop(d, hh), acc[d], 0, 0, 0);
          }
          if (col < G) {
  #pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int page = 4 * grp + j;
              const float ms = lds_f16(&sRec[wave][page][kSc + 2 * (R + 16)]);
              const float v = fmaf((float)acc[0][j], 65536.0f, (float)(acc[1][j] * 256 + acc[2][j]));
              sA[wave][page][col] = v * (ms * inv_scale);
            }
          }
        }
        // ---- stage 1: projections of every (page, basis column) onto the 4 heads
  #pragma unroll
        for (int T = 0; T < R; T += 2) {
          i4v a0[2], a1[2], acc[2];
          const int T1 = T + 1 < R ? T + 1 : T;
          nib_operands(*reinterpret_cast<const uint4*>(
                           &sRec[wave][T * kPPT + col / R][64 * (col % R) + 16 * grp]),
                       a0);
          nib_operands(*reinterpret_cast<const uint4*>(
                           &sRec[wave][T1 * kPPT + col / R][64 * (col % R) + 16 * grp]),
                       a1);
          {
            i4v x = i4v{bias[0], bias[0], bias[0], bias[0]};
            i4v y = x;
  #pragma unroll
            for (int d = 0; d < 3; ++d) {
              const i4v b0 = qop(d, 0), b1 = qop(d, 1);
              x = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0[0], b0, x, 0, 0, 0);
              y = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1[0], b0, y, 0, 0, 0);
              x = __builtin_amdgcn_mfma_i32_16x16x64_i8(a0[1], b1, x, 0, 0, 0);
              y = __builtin_amdgcn_mfma_i32_16x16x64_i8(a1[1], b1, y, 0, 0, 0);
              if (d < 2) {
  #pragma unroll
                for (int j = 0; j < 4; ++j) x[j] = (int)(((uint32_t)x[j] << 8) + (uint32_t)bias[d + 1]);
  #pragma unroll
                for (int j = 0; j < 4; ++j) y[j] = (int)(((uint32_t)y[j] << 8) + (uint32_t)bias[d + 1]);
              }
            }
            acc[0] = x;
            acc[1] = y;
          }
          if (col < G) {
  #pragma unroll
            for (int i = 0; i < 2 && T + i < R; ++i)
  #pragma unroll
              for (int j = 0; j < 4; ++j) {
                const int row = 4 * grp + j;
                const int page = (T + i) * kPPT + row / R, l = row % R;
                const float vs = lds_f16(&sRec[wave][page][kSc + 2 * l]);
                sP[wave][page][col][l] = (float)acc[i][j] * (vs * inv_scale);
              }
          }
        }
        __builtin_amdgcn_wave_barrier();
        // ---- stage 2: the 16 logits of (page pp, head gg) and their LSE
        {
          float pv[R];
          float psum = 0.0f;
  #pragma unroll
          for (int l = 0; l < R; ++l) {
            pv[l] = sP[wave][pp][gg][l];
            psum += pv[l];
          }
          const float k128 = 128.0f * psum;
          const float a = sA[wave][pp][gg];
          uint32_t cw[4 * R];  // coefficient codes, row-major (16 rows x R bytes)
  #pragma unroll
          for (int v = 0; v < R; ++v) {
            const uint4 c4 = *reinterpret_cast<const uint4*>(&sRec[wave][pp][kCoef + 16 * v]);
            cw[4 * v] = c4.x;
            cw[4 * v + 1] = c4.y;
            cw[4 * v + 2] = c4.z;
            cw[4 * v + 3] = c4.w;
          }
          uint32_t sw[8];  // coefficient row scales (fp16 pairs)
  #pragma unroll
          for (int v = 0; v < 8; ++v)
            sw[v] = *reinterpret_cast<const uint32_t*>(&sRec[wave][pp][kSc + 2 * R + 4 * v]);
          float e[16];
  #pragma unroll
          for (int i = 0; i < 16; ++i) {
            float tz = -k128;
  #pragma unroll
            for (int l = 0; l < R; ++l) {
              const int b = i * R + l;  // byte index of code (i, l)
              const float c = (float)((cw[b >> 2] >> (8 * (b & 3))) & 0xffu);
              tz = fmaf(c, pv[l], tz);
            }
            const h2 sc = as_h2(sw[i >> 1]);
            e[i] = tz * (float)((i & 1) ? sc.y : sc.x);  // logit minus the centroid term
          }
          float sm = 0.0f;
  #pragma unroll
          for (int i = 0; i < 16; ++i) sm += __builtin_amdgcn_exp2f(e[i]);
          float shift = 0.0f;
          if (!(sm > 0.0f && sm < INFINITY)) {
            shift = e[0];
  #pragma unroll
            for (int i = 1; i < 16; ++i) shift = fmaxf(shift, e[i]);
            sm = 0.0f;
  #pragma unroll
            for (int i = 0; i < 16; ++i) sm += __builtin_amdgcn_exp2f(e[i] - shift);
          }
          const float s2 = a + shift + __builtin_amdgcn_logf(sm);
          const int page = page0 + pp;
          const bool live = page < n_c;
          // stored after the next step's loads are issued (its wait then skips the store)
          st_val = s2 * 0.69314718055994531f;
          st_page = live ? page : -1;
          const float ex = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
          const bool up = s2 > run_m;
          const float ns = up ? fmaf(run_s, ex, 1.0f) : run_s + ex;
          run_s = live ? ns : run_s;
          run_m = (live && up) ? s2 : run_m;
        }
        __builtin_amdgcn_wave_barrier();
      }
      if (st_page >= 0) shat_base[(long)st_page * lay.page] = st_val;
    };
    static_assert(kLowSteps == 4, "one unrolled run per step count");
    if (n_steps == 4) run(IntTag<4>{});
    else if (n_steps == 3) run(IntTag<3>{});
    else if (n_steps == 2) run(IntTag<2>{});
    else run(IntTag<1>{});
  }
  // ---- block partial (max, sum exp) per head over its pages, log2 domain: lane
  // l holds head l % 4; the wave's lanes are merged first
  merge_lanes_mod<4>(run_m, run_s);
  if (lane < G) sRun[wave][lane] = make_float2(run_m, run_s);
  __syncthreads();
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float m = -INFINITY, l = 0.0f;
    for (int w = 0; w < 4; ++w) m = fmaxf(m, sRun[w][g].x);
    if (m > -INFINITY)
      for (int w = 0; w < 4; ++w) {
        const float2 v = sRun[w][g];
        if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
      }
    partials[(row0 + g) * gridDim.x + blockIdx.x] = make_float2(m, l);
  }
}


// ---------------------------------------------------------------------------
// Pages of B = 32 or 64 tokens (App. D.3 "Page size"), int4 basis.  The generic
// kernel's two stages with tiles of 8 pages: stage 1 (f16 MFMA, rows (page, basis
// column), columns the query heads) and the centroid projection are unchanged,
// the record tail holds B coefficient rows, and stage 2 runs one page at a time on
// fp32 MFMA 16x16x4 with the B tokens as rows (B / 16 row tiles) and the heads as
// columns; each lane then holds 4 B / 16 logits of one head and the page LSE
// takes its max and sum over them and the three other lanes of the head.
// ---------------------------------------------------------------------------
template <int R, int B>
struct PageGeom {
  static constexpr int kTP = 8;                                   // pages per tile
  static constexpr int kPPS = (16 / R) > 0 ? 16 / R : 1;          // pages per stage-1 set
  static constexpr int kSets = (kTP + kPPS - 1) / kPPS;
  static constexpr int kStride = rec_stride(R, 0, B);
  static constexpr int kTail = kStride - 64 * R;                  // coef .. end of record
  static constexpr int kTailCh = kTail / 16;
  static constexpr int kTailLoads = (kTP * kTailCh + 63) / 64;
  static constexpr int kMu = B * R;                               // offsets inside the tail
  static constexpr int kSc = B * R + kDim;
  static constexpr int kTiles = 64 / kTP;                         // tiles per wave (64 pages)
};

template <int R, int B>
struct PageRegs {
  uint4 vb[PageGeom<R, B>::kSets];
  uint4 tl[PageGeom<R, B>::kTailLoads];
};

// wave_blk: lane l holds the block of the wave's page l (-1 past the sequence's
// complete pages), read once per wave; tile t covers the wave's pages
// t kTP .. t kTP + kTP - 1.
template <int R, int B>
__device__ __forceinline__ void issue_page_tile(PageRegs<R, B>& T, const uint8_t* __restrict__ summ,
                                                int wave_blk, int t, int H_kv, int h, int lane) {
  using Gm = PageGeom<R, B>;
  const int col = lane & 15, grp = lane >> 4;
  const int pp = col / R, l = col % R;
#pragma unroll
  for (int st = 0; st < Gm::kSets; ++st) {
    const int page = st * Gm::kPPS + pp;
    const int blk = __shfl(wave_blk, (t * Gm::kTP + (page < Gm::kTP ? page : 0)) & 63, 64);
    const bool ok = col < Gm::kPPS * R && page < Gm::kTP && blk >= 0;
    T.vb[st] = ok ? *reinterpret_cast<const uint4*>(summ + ((long)blk * H_kv + h) * Gm::kStride +
                                                    64 * l + 16 * grp)
                  : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < Gm::kTailLoads; ++u) {
    const int c = lane + 64 * u;
    const int page = c / Gm::kTailCh, off = (c % Gm::kTailCh) * 16;
    const int blk = __shfl(wave_blk, (t * Gm::kTP + (page < Gm::kTP ? page : 0)) & 63, 64);
    T.tl[u] = (c < Gm::kTP * Gm::kTailCh && blk >= 0)
                  ? *reinterpret_cast<const uint4*>(summ + ((long)blk * H_kv + h) * Gm::kStride +
                                                    64 * R + off)
                  : make_uint4(0, 0, 0, 0);
  }
}

// NPG: pages per stage-2 pass (16 / G when the group size G divides 16 and is
// below 16: the 16 MFMA columns then hold (page, head) pairs, the K axis runs over
// (page, basis column) and each page's coefficients meet only its own
// projections; 1: the heads are the columns, any G <= 16).
template <typename QT, int R, int B, int NPG = 1>
__global__ __launch_bounds__(256) void scan_page_kernel(
    int H_q, int H_kv, int max_pages, const QT* __restrict__ q,
    const uint8_t* __restrict__ summaries, const int32_t* __restrict__ page_table,
    const int32_t* __restrict__ seq_lens, float* __restrict__ s_hat, SHatLayout lay,
    float2* __restrict__ partials, int wave_pages) {
  using Gm = PageGeom<R, B>;
  constexpr bool kSplitQ = sizeof(QT) == 4;  // fp32 queries: f16 hi + lo
  constexpr int kKS = (R + 3) / 4;           // stage-2 k-steps
  constexpr int kRT = B / 16;                // stage-2 row tiles
  __shared__ __align__(16) uint8_t sTail[4][Gm::kTP][Gm::kTail];
  __shared__ float sP[4][Gm::kTP][R][16];
  __shared__ float sA[4][Gm::kTP][16];
  __shared__ float2 sRun[4][16];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int h = blockIdx.y, s = blockIdx.z;
  const int G = H_q / H_kv;
  const int n_c = seq_lens[s] / B;
  // pages wave_pages (16, 32 or 64) from `base` are this wave's
  const int base = (scan_chunk() * 4 + wave) * wave_pages;
  const long row0 = (long)s * H_q + (long)h * G;
  const int32_t* pt_row = page_table + (long)s * max_pages;
  float run_m = -INFINITY, run_s = 0.0f;  // running normaliser of head col, log2 domain
  if (base < n_c) {
    const int wave_blk = lane < wave_pages && base + lane < n_c ? pt_row[base + lane] : -1;
    PageRegs<R, B> buf[2];
    issue_page_tile<R, B>(buf[0], summaries, wave_blk, 0, H_kv, h, lane);

    // ---- B operands: column = query head, K permuted to match the decoders
    constexpr int kPerm[8] = {0, 4, 1, 5, 2, 6, 3, 7};
    float qv[4][8], qm[4][8];
    float qmax = 0.0f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) {
        const int cv = 32 * grp + 8 * ks + kPerm[jj], cm = 32 * grp + 8 * ks + jj;
        const float a = col < G ? load_q(q, (row0 + col) * kDim + cv) : 0.0f;
        const float b = col < G ? load_q(q, (row0 + col) * kDim + cm) : 0.0f;
        qv[ks][jj] = a;
        qm[ks][jj] = b;
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
      for (int jj = 0; jj < 8; ++jj) {
        const float a = qv[ks][jj] * qs, b = qm[ks][jj] * qs;
        const _Float16 ah = (_Float16)a, bh = (_Float16)b;
        bv[ks][jj] = ah;
        bm[ks][jj] = bh;
        bvl[ks][jj] = (_Float16)(a - (float)ah);
        bml[ks][jj] = (_Float16)(b - (float)bh);
      }

    constexpr float kLn2 = 0.69314718055994531f;
    const float c0 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)

    // (unrolled, so the two tile buffers are named registers, not private memory)
#pragma unroll
    for (int t = 0; t < Gm::kTiles; ++t) {
      const int page0 = base + t * Gm::kTP;
      if (t * Gm::kTP >= wave_pages || page0 >= n_c) break;
      PageRegs<R, B>& cur = buf[t & 1];
      if (t + 1 < Gm::kTiles && (t + 1) * Gm::kTP < wave_pages && page0 + Gm::kTP < n_c)
        issue_page_tile<R, B>(buf[(t + 1) & 1], summaries, wave_blk, t + 1, H_kv, h, lane);
#pragma unroll
      for (int u = 0; u < Gm::kTailLoads; ++u) {
        const int c = lane + 64 * u;
        if (c < Gm::kTP * Gm::kTailCh)
          *reinterpret_cast<uint4*>(&sTail[wave][c / Gm::kTailCh][(c % Gm::kTailCh) * 16]) =
              cur.tl[u];
      }
      __builtin_amdgcn_wave_barrier();

      // ---- stage 1: p = V^T q (scaled by the basis column scales)
#pragma unroll
      for (int st = 0; st < Gm::kSets; ++st) {
        f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        const uint32_t w[4] = {cur.vb[st].x, cur.vb[st].y, cur.vb[st].z, cur.vb[st].w};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const h8 a = nib8_to_h8(w[ks]);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bv[ks], acc, 0, 0, 0);
          if (kSplitQ) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bvl[ks], acc, 0, 0, 0);
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int m = 4 * grp + jj;
          const int pp = m / R, l = m % R;
          const int page = st * Gm::kPPS + pp;
          if (m < Gm::kPPS * R && page < Gm::kTP && col < G)
            sP[wave][page][l][col] = acc[jj] * inv_qs * lds_f16(&sTail[wave][page][Gm::kSc + 2 * l]);
        }
      }
      // ---- centroid term a = mu^T q, one page per row
      {
        const int cp = col < Gm::kTP ? col : 0;
        const uint4 m0 = *reinterpret_cast<const uint4*>(&sTail[wave][cp][Gm::kMu + 32 * grp]);
        const uint4 m1 = *reinterpret_cast<const uint4*>(&sTail[wave][cp][Gm::kMu + 32 * grp + 16]);
        const uint32_t w[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
        f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          const h8 a = byte8_to_h8(w[2 * ks], w[2 * ks + 1]);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bm[ks], acc, 0, 0, 0);
          if (kSplitQ) acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, bml[ks], acc, 0, 0, 0);
        }
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int page = 4 * grp + jj;
          if (page < Gm::kTP && col < G)
            sA[wave][page][col] =
                acc[jj] * inv_qs * c0 * lds_f16(&sTail[wave][page][Gm::kSc + 2 * (R + B)]);
        }
      }
      __builtin_amdgcn_wave_barrier();

      if constexpr (NPG == 1) {
        // ---- stage 2, one page at a time: z[token][head] over B / 16 row tiles
        for (int p = 0; p < Gm::kTP; ++p) {
          if (page0 + p >= n_c) break;
          float z[kRT][4];
  #pragma unroll
          for (int rt = 0; rt < kRT; ++rt) {
            f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  #pragma unroll
            for (int kstep = 0; kstep < kKS; ++kstep) {
              const int l = 4 * kstep + grp;
              const int tok = 16 * rt + col;
              const float a = l < R ? (float)((int)sTail[wave][p][tok * R + l] - 128) : 0.0f;
              const float b = (l < R && col < G) ? sP[wave][p][l < R ? l : 0][col] : 0.0f;
              acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
            }
            const uint2 csw = *reinterpret_cast<const uint2*>(
                &sTail[wave][p][Gm::kSc + 2 * (R + 16 * rt + 4 * grp)]);
            const h2 cs01 = as_h2(csw.x), cs23 = as_h2(csw.y);
            const float av = sA[wave][p][col];
            z[rt][0] = fmaf((float)cs01.x * c0, acc[0], av);
            z[rt][1] = fmaf((float)cs01.y * c0, acc[1], av);
            z[rt][2] = fmaf((float)cs23.x * c0, acc[2], av);
            z[rt][3] = fmaf((float)cs23.y * c0, acc[3], av);
          }
          float mx = -INFINITY;
  #pragma unroll
          for (int rt = 0; rt < kRT; ++rt)
            mx = fmaxf(mx, fmaxf(fmaxf(z[rt][0], z[rt][1]), fmaxf(z[rt][2], z[rt][3])));
          mx = red4_max(mx);
          float sm = 0.0f;
  #pragma unroll
          for (int rt = 0; rt < kRT; ++rt)
  #pragma unroll
            for (int jj = 0; jj < 4; ++jj) sm += __builtin_amdgcn_exp2f(z[rt][jj] - mx);
          sm = red4_sum(sm);
          const float s2 = mx + __builtin_amdgcn_logf(sm);  // log2-domain page score
          if (col < G) {
            if (grp == 0)
              s_hat[lay.base(s, h) + col * lay.head + (long)(page0 + p) * lay.page] = s2 * kLn2;
            const float e = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
            if (s2 > run_m) { run_s = fmaf(run_s, e, 1.0f); run_m = s2; }
            else run_s += e;
          }
        }
      } else {
        // ---- stage 2, NPG pages at a time: z[token][(page pc, head gc)]
        constexpr int kG = 16 / NPG;
        const int pc = col / kG, gc = col % kG;
#pragma unroll
        for (int p0 = 0; p0 < Gm::kTP; p0 += NPG) {
          if (page0 + p0 >= n_c) break;
          float z[kRT][4];
#pragma unroll
          for (int rt = 0; rt < kRT; ++rt) {
            f4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            const int tok = 16 * rt + col;
#pragma unroll
            for (int pp = 0; pp < NPG; ++pp)
#pragma unroll
              for (int kstep = 0; kstep < kKS; ++kstep) {
                const int l = 4 * kstep + grp;
                const int la = l < R ? l : 0;
                const float a = l < R ? (float)((int)sTail[wave][p0 + pp][tok * R + la] - 128) : 0.0f;
                const float b = (l < R && pc == pp) ? sP[wave][p0 + pp][la][gc] : 0.0f;
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
              }
            const uint2 csw = *reinterpret_cast<const uint2*>(
                &sTail[wave][p0 + pc][Gm::kSc + 2 * (R + 16 * rt + 4 * grp)]);
            const h2 cs01 = as_h2(csw.x), cs23 = as_h2(csw.y);
            const float av = sA[wave][p0 + pc][gc];
            z[rt][0] = fmaf((float)cs01.x * c0, acc[0], av);
            z[rt][1] = fmaf((float)cs01.y * c0, acc[1], av);
            z[rt][2] = fmaf((float)cs23.x * c0, acc[2], av);
            z[rt][3] = fmaf((float)cs23.y * c0, acc[3], av);
          }
          float mx = -INFINITY;
#pragma unroll
          for (int rt = 0; rt < kRT; ++rt)
            mx = fmaxf(mx, fmaxf(fmaxf(z[rt][0], z[rt][1]), fmaxf(z[rt][2], z[rt][3])));
          mx = red4_max(mx);
          float sm = 0.0f;
#pragma unroll
          for (int rt = 0; rt < kRT; ++rt)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) sm += __builtin_amdgcn_exp2f(z[rt][jj] - mx);
          sm = red4_sum(sm);
          const float s2 = mx + __builtin_amdgcn_logf(sm);  // log2-domain page score
          if (page0 + p0 + pc < n_c) {
            if (grp == 0)
              s_hat[lay.base(s, h) + gc * lay.head + (long)(page0 + p0 + pc) * lay.page] = s2 * kLn2;
            const float e = __builtin_amdgcn_exp2f(-fabsf(s2 - run_m));
            if (s2 > run_m) { run_s = fmaf(run_s, e, 1.0f); run_m = s2; }
            else run_s += e;
          }
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  // ---- block partial (max, sum exp) per head over its pages (log2 domain):
  //      head g's running pairs sit in the columns p G + g, p < NPG, of every wave
  if (lane < 16) sRun[wave][lane] = make_float2(run_m, run_s);
  __syncthreads();
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float m = -INFINITY, l = 0.0f;
    for (int w = 0; w < 4; ++w)
      for (int p = 0; p < NPG; ++p) m = fmaxf(m, sRun[w][p * G + g].x);
    if (m > -INFINITY)
      for (int w = 0; w < 4; ++w)
        for (int p = 0; p < NPG; ++p) {
          const float2 v = sRun[w][p * G + g];
          if (v.y > 0.0f) l += v.y * __builtin_amdgcn_exp2f(v.x - m);
        }
    partials[(row0 + g) * gridDim.x + blockIdx.x] = make_float2(m, l);
  }
}

// r = 8, G = 16 over pages of 16 V tokens, V = 2 or 4 (sub-pages of 16 tokens).
template <typename QT>
hipError_t dispatch_scan_r8_sub(int V, int steps, dim3 grid, hipStream_t st, int H_q, int H_kv,
                                int max_pages, const QT* q, const uint8_t* sum,
                                uint32_t summ_bytes, const int32_t* pt, const int32_t* sl,
                                float* s_hat, SHatLayout lay, float2* part) {
#define LOCKS_SCAN_R8_SUB(VV, SS)                                                           \
  if (V == VV && steps == SS) {                                                            \
    hipLaunchKernelGGL((scan_r8_kernel<QT, SS, VV>), grid, dim3(256), 0, st, H_q, H_kv,    \
                       max_pages, q, sum, summ_bytes, pt, sl, s_hat, lay, part);           \
    return hipGetLastError();                                                              \
  }
  LOCKS_SCAN_R8_SUB(2, 1) LOCKS_SCAN_R8_SUB(2, 4) LOCKS_SCAN_R8_SUB(4, 1) LOCKS_SCAN_R8_SUB(4, 4)
#undef LOCKS_SCAN_R8_SUB
  return hipErrorInvalidValue;
}

// r = 8, G = 4 over pages of 16 V tokens, V = 2 or 4.
template <typename QT>
hipError_t dispatch_scan_r8g4_sub(int V, int steps, dim3 grid, hipStream_t st, int H_q, int H_kv,
                                  int max_pages, const QT* q, const uint8_t* sum,
                                  uint32_t summ_bytes, const int32_t* pt, const int32_t* sl,
                                  float* s_hat, SHatLayout lay, float2* part) {
#define LOCKS_SCAN_R8G4_SUB(VV, SS)                                                         \
  if (V == VV && steps == SS) {                                                            \
    hipLaunchKernelGGL((scan_r8g4_kernel<QT, SS, VV>), grid, dim3(256), 0, st, H_q, H_kv,  \
                       max_pages, q, sum, summ_bytes, pt, sl, s_hat, lay, part);           \
    return hipGetLastError();                                                              \
  }
  LOCKS_SCAN_R8G4_SUB(2, 1) LOCKS_SCAN_R8G4_SUB(2, 4) LOCKS_SCAN_R8G4_SUB(4, 1)
  LOCKS_SCAN_R8G4_SUB(4, 4)
#undef LOCKS_SCAN_R8G4_SUB
  return hipErrorInvalidValue;
}

template <typename QT>
hipError_t dispatch_scan_page(int r, int B, int wp, dim3 grid, hipStream_t st, int H_q, int H_kv,
                              int max_pages, const QT* q, const uint8_t* sum, const int32_t* pt,
                              const int32_t* sl, float* s_hat, SHatLayout lay, float2* part) {
#define LOCKS_SCAN_PAGE_CASE(RR)                                                              \
  case RR:                                                                                   \
    if (B == 32)                                                                             \
      hipLaunchKernelGGL((scan_page_kernel<QT, RR, 32>), grid, dim3(256), 0, st, H_q, H_kv,  \
                         max_pages, q, sum, pt, sl, s_hat, lay, part, wp);                   \
    else                                                                                     \
      hipLaunchKernelGGL((scan_page_kernel<QT, RR, 64>), grid, dim3(256), 0, st, H_q, H_kv,  \
                         max_pages, q, sum, pt, sl, s_hat, lay, part, wp);                   \
    break;
  if (B != 32 && B != 64) return hipErrorInvalidValue;
  // four-head groups at the common ranks: four pages per stage-2 pass
  if (H_q == 4 * H_kv && (r == 2 || r == 4 || r == 8)) {
#define LOCKS_SCAN_PAGE4(RR)                                                                  \
    if (r == RR) {                                                                           \
      if (B == 32)                                                                           \
        hipLaunchKernelGGL((scan_page_kernel<QT, RR, 32, 4>), grid, dim3(256), 0, st, H_q,   \
                           H_kv, max_pages, q, sum, pt, sl, s_hat, lay, part, wp);           \
      else                                                                                   \
        hipLaunchKernelGGL((scan_page_kernel<QT, RR, 64, 4>), grid, dim3(256), 0, st, H_q,   \
                           H_kv, max_pages, q, sum, pt, sl, s_hat, lay, part, wp);           \
      return hipGetLastError();                                                              \
    }
    LOCKS_SCAN_PAGE4(2) LOCKS_SCAN_PAGE4(4) LOCKS_SCAN_PAGE4(8)
#undef LOCKS_SCAN_PAGE4
  }
  switch (r) {
    LOCKS_SCAN_PAGE_CASE(1) LOCKS_SCAN_PAGE_CASE(2) LOCKS_SCAN_PAGE_CASE(3)
    LOCKS_SCAN_PAGE_CASE(4) LOCKS_SCAN_PAGE_CASE(5) LOCKS_SCAN_PAGE_CASE(6)
    LOCKS_SCAN_PAGE_CASE(7) LOCKS_SCAN_PAGE_CASE(8) LOCKS_SCAN_PAGE_CASE(9)
    LOCKS_SCAN_PAGE_CASE(10) LOCKS_SCAN_PAGE_CASE(11) LOCKS_SCAN_PAGE_CASE(12)
    LOCKS_SCAN_PAGE_CASE(13) LOCKS_SCAN_PAGE_CASE(14) LOCKS_SCAN_PAGE_CASE(15)
    default:
      return hipErrorInvalidValue;
  }
#undef LOCKS_SCAN_PAGE_CASE
  return hipGetLastError();
}

template <typename QT>
hipError_t dispatch_scan(int r, int G, int basis, int steps, dim3 grid, hipStream_t st, int H_q,
                         int H_kv, int max_pages, const QT* q, const uint8_t* sum,
                         uint32_t summ_bytes, const int32_t* pt, const int32_t* sl, float* s_hat,
                         SHatLayout lay, float2* part) {
  if (basis != LOCKS_BASIS_INT4) {  // int8 / bf16 bases: the generic kernel, r in {2, 4, 8}
#define LOCKS_SCAN_BASIS(RR, BB)                                                            \
    if (r == RR && basis == BB) {                                                           \
      hipLaunchKernelGGL((scan_mfma_kernel<QT, RR, BB>), grid, dim3(256), 0, st, H_q, H_kv, \
                         max_pages, q, sum, pt, sl, s_hat, lay, part);                      \
      return hipGetLastError();                                                             \
    }
    LOCKS_SCAN_BASIS(2, 1) LOCKS_SCAN_BASIS(4, 1) LOCKS_SCAN_BASIS(8, 1)
    LOCKS_SCAN_BASIS(2, 2) LOCKS_SCAN_BASIS(4, 2) LOCKS_SCAN_BASIS(8, 2)
#undef LOCKS_SCAN_BASIS
    return hipErrorInvalidValue;
  }
#define LOCKS_SCAN_FAST(RR, NP)                                                              \
  if (r == RR && G == 16 / NP) {                                                            \
    hipLaunchKernelGGL((scan_fast_kernel<QT, RR, NP>), grid, dim3(256), 0, st, H_q, H_kv,   \
                       max_pages, q, sum, pt, sl, s_hat, lay, part);               \
    return hipGetLastError();                                                               \
  }
  if (r == 8 && G == 16) {
    if (steps == 1)
      hipLaunchKernelGGL((scan_r8_kernel<QT, 1>), grid, dim3(256), 0, st, H_q, H_kv, max_pages, q,
                         sum, summ_bytes, pt, sl, s_hat, lay, part);
    else
      hipLaunchKernelGGL((scan_r8_kernel<QT, 4>), grid, dim3(256), 0, st, H_q, H_kv, max_pages, q,
                         sum, summ_bytes, pt, sl, s_hat, lay, part);
    return hipGetLastError();
  }
  if ((r == 2 || r == 4) && G == 4) {
    if (r == 2)
      hipLaunchKernelGGL((scan_low_kernel<QT, 2>), grid, dim3(256), 0, st, H_q, H_kv, max_pages, q,
                         sum, summ_bytes, pt, sl, s_hat, lay, part);
    else
      hipLaunchKernelGGL((scan_low_kernel<QT, 4>), grid, dim3(256), 0, st, H_q, H_kv, max_pages, q,
                         sum, summ_bytes, pt, sl, s_hat, lay, part);
    return hipGetLastError();
  }
  if (r == 8 && G == 4) {
    if (steps == 1)
      hipLaunchKernelGGL((scan_r8g4_kernel<QT, 1>), grid, dim3(256), 0, st, H_q, H_kv, max_pages,
                         q, sum, summ_bytes, pt, sl, s_hat, lay, part);
    else
      hipLaunchKernelGGL((scan_r8g4_kernel<QT, 4>), grid, dim3(256), 0, st, H_q, H_kv, max_pages,
                         q, sum, summ_bytes, pt, sl, s_hat, lay, part);
    return hipGetLastError();
  }
  // r = 2 and 4 at G = 16 (G = 4 took the low-rank kernel above)
  LOCKS_SCAN_FAST(4, 1) LOCKS_SCAN_FAST(2, 1)
#undef LOCKS_SCAN_FAST
#define LOCKS_SCAN_MFMA_CASE(RR)                                                             \
  case RR:                                                                                  \
    hipLaunchKernelGGL((scan_mfma_kernel<QT, RR>), grid, dim3(256), 0, st, H_q, H_kv,       \
                       max_pages, q, sum, pt, sl, s_hat, lay, part);               \
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

}  // namespace

// r = 8, G = 16 with an int4 basis, at every page size (larger pages as 16-token
// sub-pages).
static bool use_r8_kernel(const locks_cfg_t& c) {
  return c.basis == LOCKS_BASIS_INT4 && c.rank == 8 && c.num_q_heads == 16 * c.num_kv_heads;
}

static bool use_r8g4_kernel(const locks_cfg_t& c) {
  return c.basis == LOCKS_BASIS_INT4 && c.rank == 8 && c.num_q_heads == 4 * c.num_kv_heads;
}

// 16-page steps per wave of the r = 8 kernels: 4, or 1 when a 4-step grid would
// have fewer blocks than the GPU has compute units.
static int r8_steps(const locks_cfg_t& c) {
  const long sub = (long)c.max_pages_per_seq << sub_page_log2(c);
  const long blocks4 = (sub + 255) / 256 * c.num_kv_heads * c.num_seqs;
  return blocks4 < 256 ? 1 : 4;
}

// Pages per wave of the 32/64-token scan: 64, or 32 / 16 when 64 would leave
// fewer than two waves per SIMD of the GPU (1,024 SIMDs).
static int page_wave_pages(const locks_cfg_t& c) {
  for (int wp = 64; wp > 16; wp /= 2)
    if ((long)((c.max_pages_per_seq + wp - 1) / wp) * c.num_kv_heads * c.num_seqs >= 2048) return wp;
  return 16;
}

int scan_pages_per_block(const locks_cfg_t& c) {
  if (use_r8_kernel(c) || use_r8g4_kernel(c)) return (64 * r8_steps(c)) >> sub_page_log2(c);
  if (c.page_size != kPage) return 4 * page_wave_pages(c);
  return kScanPagesPerBlock;
}

hipError_t launch_scan(const locks_cfg_t& c, const void* q, const void* summaries,
                       const int32_t* page_table, const int32_t* seq_lens, float* s_hat,
                       SHatLayout lay, float2* partials, hipStream_t st) {
  const dim3 grid(scan_blocks(c), c.num_kv_heads, c.num_seqs);
  const int G = c.num_q_heads / c.num_kv_heads;
  const uint32_t bytes = (uint32_t)summary_store_bytes(c);
  const int steps = r8_steps(c);
  if (c.page_size != kPage && use_r8_kernel(c)) {
    const int V = 1 << sub_page_log2(c);
    if (c.q_dtype == LOCKS_BF16)
      return dispatch_scan_r8_sub(V, steps, grid, st, c.num_q_heads, c.num_kv_heads,
                                  c.max_pages_per_seq, static_cast<const uint16_t*>(q),
                                  static_cast<const uint8_t*>(summaries), bytes, page_table,
                                  seq_lens, s_hat, lay, partials);
    return dispatch_scan_r8_sub(V, steps, grid, st, c.num_q_heads, c.num_kv_heads,
                                c.max_pages_per_seq, static_cast<const float*>(q),
                                static_cast<const uint8_t*>(summaries), bytes, page_table,
                                seq_lens, s_hat, lay, partials);
  }
  if (c.page_size != kPage && use_r8g4_kernel(c)) {
    const int V = 1 << sub_page_log2(c);
    if (c.q_dtype == LOCKS_BF16)
      return dispatch_scan_r8g4_sub(V, steps, grid, st, c.num_q_heads, c.num_kv_heads,
                                    c.max_pages_per_seq, static_cast<const uint16_t*>(q),
                                    static_cast<const uint8_t*>(summaries), bytes, page_table,
                                    seq_lens, s_hat, lay, partials);
    return dispatch_scan_r8g4_sub(V, steps, grid, st, c.num_q_heads, c.num_kv_heads,
                                  c.max_pages_per_seq, static_cast<const float*>(q),
                                  static_cast<const uint8_t*>(summaries), bytes, page_table,
                                  seq_lens, s_hat, lay, partials);
  }
  if (c.page_size != kPage) {
    if (c.q_dtype == LOCKS_BF16)
      return dispatch_scan_page(c.rank, c.page_size, page_wave_pages(c), grid, st, c.num_q_heads,
                                c.num_kv_heads,
                                c.max_pages_per_seq, static_cast<const uint16_t*>(q),
                                static_cast<const uint8_t*>(summaries), page_table, seq_lens,
                                s_hat, lay, partials);
    return dispatch_scan_page(c.rank, c.page_size, page_wave_pages(c), grid, st, c.num_q_heads,
                              c.num_kv_heads,
                              c.max_pages_per_seq, static_cast<const float*>(q),
                              static_cast<const uint8_t*>(summaries), page_table, seq_lens, s_hat,
                              lay, partials);
  }
  if (c.q_dtype == LOCKS_BF16)
    return dispatch_scan(c.rank, G, c.basis, steps, grid, st, c.num_q_heads, c.num_kv_heads,
                         c.max_pages_per_seq, static_cast<const uint16_t*>(q),
                         static_cast<const uint8_t*>(summaries), bytes, page_table, seq_lens,
                         s_hat, lay, partials);
  return dispatch_scan(c.rank, G, c.basis, steps, grid, st, c.num_q_heads, c.num_kv_heads,
                       c.max_pages_per_seq, static_cast<const float*>(q),
                       static_cast<const uint8_t*>(summaries), bytes, page_table, seq_lens, s_hat,
                       lay, partials);
}

}  // namespace locks
