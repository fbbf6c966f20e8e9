// Per-page summary construction for pages of B = 32 or 64 tokens (Sec. 4
// "Build"; App. D.3 "Page size"): centre the page's B keys, form the B x B Gram of
// the deviations, find its eigenpairs, keep the r leading nonzero modes, form
// V = D^T U_r S_r^{-1} and C = U_r S_r, quantise and pack.
//
// The symmetric eigenproblem is solved with B lanes, one row each: Householder
// reduction to a tridiagonal T (the rows in LDS; the reflector and its update
// vectors broadcast through LDS), the wanted eigenvalues of T by multisection on
// Sturm counts (B / n lanes per eigenvalue), the r leading eigenvectors of T by
// inverse iteration on its LDL^T factorisation (lane l solves for vector l; two
// rounds, each followed by modified Gram-Schmidt over the r vectors, so a
// near-degenerate pair still yields an orthonormal basis of its eigenspace), and
// the back-transformation through the stored reflectors.  Everything is fp32.
// Cross-lane sums use DPP within 16-lane rows and row swaps across them.
//
// Mapping: one wave per block holding 64 / B items (page, KV head); lane (it, i)
// owns row i of item it.
#include "locks_internal.h"

namespace locks {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr float kZeroRel = 1e-6f;
constexpr float kZeroAbs = 1e-10f;
constexpr int kInvRounds = 2;     // inverse-iteration rounds (solve + orthogonalise)

template <int B>
struct PG {
  static constexpr int kItems = 64 / B;       // items per wave
  static constexpr int kCols = kDim / B;      // key columns per lane (centroid, basis)
  static constexpr int kPad = B + 4;          // LDS row stride (floats) of the Gram
  static constexpr int kVec = B + 1;          // LDS stride (floats) of a lane's vector
  static constexpr int kKeyParts = B == 32 ? 2 : 1;  // column parts of the key rows in LDS
};

template <int C>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), C, 0xF, 0xF, false));
}
// Sum / max over the B lanes of an item (lane groups of B consecutive lanes):
// within a 16-lane row by DPP (quad xor 1, quad xor 2, half-row mirror, row
// mirror), across rows by lane swaps.
// (a row swap pairs rows 0-1 and 2-3, a half swap the two halves of the wave:
// the two results summed hold the pair's total in both)
template <int B>
__device__ __forceinline__ float group_sum(float v) {
  v += dpp_f<0xB1>(v);
  v += dpp_f<0x4E>(v);
  v += dpp_f<0x141>(v);
  v += dpp_f<0x140>(v);
  if (B >= 32) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  }
  if (B >= 64) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  }
  return v;
}
template <int B>
__device__ __forceinline__ float group_max(float v) {
  v = fmaxf(v, dpp_f<0xB1>(v));
  v = fmaxf(v, dpp_f<0x4E>(v));
  v = fmaxf(v, dpp_f<0x141>(v));
  v = fmaxf(v, dpp_f<0x140>(v));
  if (B >= 32) {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  }
  if (B >= 64) {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  }
  return v;
}
template <int B>
__device__ __forceinline__ int group_min_int(int v) {
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
  if (B >= 32) {
    const auto p = __builtin_amdgcn_permlane16_swap((uint32_t)v, (uint32_t)v, false, false);
    v = min((int)p[0], (int)p[1]);
  }
  if (B >= 64) {
    const auto p = __builtin_amdgcn_permlane32_swap((uint32_t)v, (uint32_t)v, false, false);
    v = min((int)p[0], (int)p[1]);
  }
  return v;
}

// Elements of a 16-byte chunk of bf16 or fp32 keys as floats.
template <typename KT>
__device__ __forceinline__ void chunk_to_f(const uint4& w, float* out);
template <>
__device__ __forceinline__ void chunk_to_f<uint16_t>(const uint4& w, float* out) {
  const uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    out[2 * e] = __uint_as_float(u[e] << 16);
    out[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void chunk_to_f<float>(const uint4& w, float* out) {
  out[0] = __uint_as_float(w.x); out[1] = __uint_as_float(w.y);
  out[2] = __uint_as_float(w.z); out[3] = __uint_as_float(w.w);
}

__device__ __forceinline__ float f16_scale(float amax, float qmax) {
  float s = fminf(amax / qmax, 65504.0f);
  return (float)(_Float16)s;
}
__device__ __forceinline__ int quant(float x, float s, int qmax) {
  if (!(s > 0.0f)) return 0;
  float c = rintf(x / s);
  c = fminf(fmaxf(c, (float)-qmax), (float)qmax);
  return (int)c;
}
__device__ __forceinline__ uint16_t f16_bits(float s) {
  _Float16 h = (_Float16)s;
  return *reinterpret_cast<uint16_t*>(&h);
}
__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

template <typename KT>
__device__ __forceinline__ float key_at(const KT* p, int c) { return load_elem(p, c); }

template <typename KT, int B, bool kFactors, int kMaxR>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2))) void build_page_kernel(
    int S, int H_kv, int max_pages, int r, const KT* __restrict__ k_cache,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ build_list, int n_items, int all_pages,
    uint8_t* __restrict__ summaries, float* __restrict__ mu_out, float* __restrict__ basis_out,
    float* __restrict__ coef_out, float* __restrict__ sigma2_out, int basis) {
  using P = PG<B>;
  constexpr int kI = P::kItems;
  // phase-shared LDS: key rows (load, centroid, Gram), then the Gram rows and the
  // reflectors, then U, then the packed record; the inverse-iteration arrays
  // have their own
  constexpr int kKBytes = kI * B * (kDim / P::kKeyParts) * (int)sizeof(KT);  // one part of the key rows
  constexpr int kABytes = kI * B * P::kPad * 4;
  constexpr int kRecBytes = kI * rec_stride(kMaxR, LOCKS_BASIS_BF16, B);
  constexpr int kBig0 = kKBytes > kABytes ? kKBytes : kABytes;
  constexpr int kBig = kBig0 > kRecBytes ? kBig0 : kRecBytes;
  __shared__ __align__(16) uint8_t sBuf[kBig];
  __shared__ float sInv[3 * kI * kMaxR * P::kVec];  // [3][kI][kMaxR][kVec]: M, W, X
  __shared__ __align__(16) float sMu[kI][kDim];
  __shared__ __align__(16) float sD[kI][B];      // diagonal of T
  __shared__ __align__(16) float sE[kI][B];      // off-diagonal of T (e[k] couples k, k+1)
  __shared__ __align__(16) float sE2[kI][B];     // e[k - 1]^2 (0 for k = 0), Sturm counts
  __shared__ float sTau[kI][B];
  __shared__ __align__(16) float sV[kI][B];      // reflector broadcast
  __shared__ __align__(16) float sW[kI][B];      // update-vector broadcast
  __shared__ float sLam[kI][B];                  // eigenvalues, descending
  __shared__ float sFlip[kI][kMaxR];
  auto& sK = *reinterpret_cast<KT(*)[kI][B][kDim / P::kKeyParts]>(sBuf);
  auto& sA = *reinterpret_cast<float(*)[kI][B][P::kPad]>(sBuf);
  auto inv = [&](int which, int it, int l) -> float* {
    return sInv + ((which * kI + it) * kMaxR + l) * P::kVec;
  };

  const int lane = threadIdx.x;
  const int it = lane / B, i = lane % B;
  const long item = (long)blockIdx.x * kI + it;

  // ---- which (seq, page, KV head) this item builds
  bool active = false;
  int s = 0, j = 0, h = 0, e = 0;
  if (all_pages) {
    h = (int)(item % H_kv);
    const long t = item / H_kv;
    j = (int)(t % max_pages);
    s = (int)(t / max_pages);
    active = s < S && j < seq_lens[s] / B;
  } else {
    h = (int)(item % H_kv);
    e = (int)(item / H_kv);
    if (e < n_items) {
      s = build_list[2 * e];
      j = build_list[2 * e + 1];
      active = s >= 0 && s < S && j >= 0 && j < max_pages && j < seq_lens[s] / B;
    }
  }
  if (!__any(active)) return;
  const long blk = active ? (long)page_table[(long)s * max_pages + j] : 0;
  const KT* kpage = k_cache + (blk * H_kv + h) * (long)B * kDim;

  // ---- key rows, centroid and Gram in kParts column parts: the LDS holds one
  //      part of the item's key rows at a time (the squared norm of row i
  //      accumulates from the registers).  32-token pages take two parts, so the
  //      key rows need no more LDS than the Gram rows; at 64 tokens the Gram rows
  //      need more than all the key rows, and one part keeps the registers down.
  constexpr int kParts = P::kKeyParts;
  constexpr int kHalf = kDim / kParts;
  constexpr int kV = 16 / sizeof(KT);
  constexpr int kT = B / 16;
  constexpr int kTiles = kT * (kT + 1) / 2;
  float energy = 0.0f;
  f4 acc[kI][kTiles];
#pragma unroll
  for (int t = 0; t < kI; ++t)
#pragma unroll
    for (int tile = 0; tile < kTiles; ++tile) acc[t][tile] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int hf = 0; hf < kParts; ++hf) {
    {
      const uint4* src = reinterpret_cast<const uint4*>(kpage + (long)i * kDim + hf * kHalf);
      uint4 w[kHalf / kV];
#pragma unroll
      for (int u = 0; u < kHalf / kV; ++u) w[u] = active ? src[u] : make_uint4(0, 0, 0, 0);
      uint4* dst = reinterpret_cast<uint4*>(&sK[it][i][0]);
#pragma unroll
      for (int u = 0; u < kHalf / kV; ++u) dst[u] = w[u];
#pragma unroll
      for (int u = 0; u < kHalf / kV; ++u) {
        float x[kV];
        chunk_to_f<KT>(w[u], x);
#pragma unroll
        for (int e2 = 0; e2 < kV; ++e2) energy = fmaf(x[e2], x[e2], energy);
      }
      __syncthreads();
    }
    // centroid of the lane's kHC columns of the part: pairwise sum over the B rows
    // (exact when the rows are equal)
    {
      constexpr int kHC = kHalf / B;
      float v[B][kHC];
#pragma unroll
      for (int t = 0; t < B; ++t)
#pragma unroll
        for (int cc = 0; cc < kHC; ++cc) v[t][cc] = key_at(&sK[it][t][0], kHC * i + cc);
#pragma unroll
      for (int w = B / 2; w > 0; w >>= 1)
#pragma unroll
        for (int t = 0; t < w; ++t)
#pragma unroll
          for (int cc = 0; cc < kHC; ++cc) v[t][cc] = v[t][cc] + v[t + w][cc];
#pragma unroll
      for (int cc = 0; cc < kHC; ++cc) sMu[it][hf * kHalf + kHC * i + cc] = v[0][cc] * (1.0f / B);
    }
    __syncthreads();
    // Gram of the deviations on fp32 MFMA 16x16x4, one 16 x 16 tile at a time:
    // lane l supplies row 16 T + l % 16 (A) and 16 U + l % 16 (B) at columns
    // kGC (l / 16) + m, m < kGC, of the part; register jj then holds
    // G[16 T + 4 (l/16) + jj][16 U + l % 16].  Upper tiles only; the lower
    // triangle is mirrored.
    constexpr int kGC = kHalf / 4;
    {
      const int l16 = lane & 15, q4 = lane >> 4;
#pragma unroll
      for (int t = 0; t < kI; ++t) {
        int tile = 0;
#pragma unroll
        for (int T = 0; T < kT; ++T)
#pragma unroll
          for (int U = T; U < kT; ++U) {
            f4 a = acc[t][tile];
#pragma unroll
            for (int ch = 0; ch < kGC / kV; ++ch) {
              const int c0 = kGC * q4 + kV * ch;
              const uint4 wx = *reinterpret_cast<const uint4*>(&sK[t][16 * T + l16][c0]);
              const uint4 wy = *reinterpret_cast<const uint4*>(&sK[t][16 * U + l16][c0]);
              float xs[kV], ys[kV];
              chunk_to_f<KT>(wx, xs);
              chunk_to_f<KT>(wy, ys);
#pragma unroll
              for (int e2 = 0; e2 < kV; ++e2) {
                const float m2 = sMu[t][hf * kHalf + c0 + e2];
                a = __builtin_amdgcn_mfma_f32_16x16x4f32(xs[e2] - m2, ys[e2] - m2, a, 0, 0, 0);
              }
            }
            acc[t][tile++] = a;
          }
      }
    }
    __syncthreads();  // the next part (or the Gram rows) takes the key rows' LDS
  }
  energy = group_sum<B>(energy) * (1.0f / B);
  {
    const int l16 = lane & 15, q4 = lane >> 4;
#pragma unroll
    for (int t = 0; t < kI; ++t) {
      int tile = 0;
#pragma unroll
      for (int T = 0; T < kT; ++T)
#pragma unroll
        for (int U = T; U < kT; ++U) {
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const int row = 16 * T + 4 * q4 + jj, col = 16 * U + l16;
            if (row <= col) {
              sA[t][row][col] = acc[t][tile][jj];
              sA[t][col][row] = acc[t][tile][jj];
            }
          }
          ++tile;
        }
    }
  }
  __syncthreads();

  // ---- Householder reduction to tridiagonal form, rows in LDS.  Step k
  //      annihilates column k below the subdiagonal with H = I - tau v v^T (v[k+1]
  //      = 1) and updates the trailing block by the rank-2 form A - v w^T - w v^T;
  //      v is then kept in column k of the rows below k + 1 for the
  //      back-transformation.  Entries of v, p and w at indices <= k are zero, so
  //      every lane runs the same row loops over the 4-column groups from the one
  //      holding column k + 1 on (the skipped products are exact zeros).
  float* arow = &sA[it][i][0];
  for (int k = 0; k < B - 2; ++k) {
    const float x = arow[k];
    const float sig = group_sum<B>(i > k + 1 ? x * x : 0.0f);
    const float x0 = group_sum<B>(i == k + 1 ? x : 0.0f);
    float tau = 0.0f, v0 = 1.0f, beta = x0;
    if (sig > 0.0f) {
      const float mu = sqrtf(fmaf(x0, x0, sig));
      v0 = x0 <= 0.0f ? x0 - mu : -sig / (x0 + mu);
      tau = 2.0f * v0 * v0 / (sig + v0 * v0);
      beta = mu;
    }
    const float vi = i == k + 1 ? 1.0f : (i > k + 1 && sig > 0.0f ? x / v0 : 0.0f);
    if (i == k) {
      sD[it][k] = x;
      sE[it][k] = beta;
      sTau[it][k] = tau;
    }
    sV[it][i] = vi;
    __builtin_amdgcn_wave_barrier();
    // p = tau A v over the trailing block
    const int q0 = (k + 1) >> 2;
    float p = 0.0f;
#pragma unroll 4
    for (int q = q0; q < B / 4; ++q) {
      const float4 r4 = *reinterpret_cast<const float4*>(arow + 4 * q);
      const float4 v4 = *reinterpret_cast<const float4*>(&sV[it][4 * q]);
      p = fmaf(r4.x, v4.x, p);
      p = fmaf(r4.y, v4.y, p);
      p = fmaf(r4.z, v4.z, p);
      p = fmaf(r4.w, v4.w, p);
    }
    p = i > k ? tau * p : 0.0f;
    const float kc = 0.5f * tau * group_sum<B>(p * vi);
    const float wi = p - kc * vi;
    sW[it][i] = wi;
    __builtin_amdgcn_wave_barrier();
#pragma unroll 4
    for (int q = q0; q < B / 4; ++q) {
      float4 r4 = *reinterpret_cast<const float4*>(arow + 4 * q);
      const float4 v4 = *reinterpret_cast<const float4*>(&sV[it][4 * q]);
      const float4 w4 = *reinterpret_cast<const float4*>(&sW[it][4 * q]);
      r4.x = fmaf(-vi, w4.x, fmaf(-wi, v4.x, r4.x));
      r4.y = fmaf(-vi, w4.y, fmaf(-wi, v4.y, r4.y));
      r4.z = fmaf(-vi, w4.z, fmaf(-wi, v4.z, r4.z));
      r4.w = fmaf(-vi, w4.w, fmaf(-wi, v4.w, r4.w));
      *reinterpret_cast<float4*>(arow + 4 * q) = r4;
    }
    __builtin_amdgcn_wave_barrier();
    if (i > k + 1) arow[k] = vi;  // reflector component, for the back-transformation
    __builtin_amdgcn_wave_barrier();
  }
  if (i == B - 2) {
    sD[it][B - 2] = arow[B - 2];
    sE[it][B - 2] = arow[B - 1];
  }
  if (i == B - 1) {
    sD[it][B - 1] = arow[B - 1];
    sE[it][B - 1] = 0.0f;
  }
  __syncthreads();
  sE2[it][i] = i > 0 ? fmaf(sE[it][i - 1], sE[it][i - 1], 0x1p-126f) : 0.0f;
  __syncthreads();

  float lam;
  // ---- the wanted eigenvalues of T (the r largest; all B for the factor output)
  //      by multisection on Sturm counts: q = B / n lanes per eigenvalue, one
  //      point each per step, so a group cuts its interval into q + 1 parts and
  //      a wave ballot gives the part that holds the eigenvalue
  {
    float lo = INFINITY, hi = -INFINITY;
#pragma unroll
    for (int t = 0; t < B; ++t) {
      const float el = t > 0 ? fabsf(sE[it][t - 1]) : 0.0f;
      const float er = t < B - 1 ? fabsf(sE[it][t]) : 0.0f;
      const float dd = sD[it][t];
      lo = fminf(lo, dd - el - er);
      hi = fmaxf(hi, dd + el + er);
    }
    const int ne = kFactors ? B : r;
    const int q = B / ne;
    const int lq = i / q;
    const bool idle = lq >= ne;            // lanes past ne * q copy the last group
    const int le = idle ? ne - 1 : lq;     // the eigenvalue (0 = largest)
    const int pi = idle ? 0 : i - lq * q;  // this lane's point
    const int want = B - 1 - le;           // count(x) <= want  <=>  x <= lambda_le
    const uint64_t gmask = (q >= 64 ? ~0ull : ((1ull << q) - 1ull)) << (it * B + le * q);
    // the Sturm counts carry rounding of a few ulp of |T|: the interval is cut to
    // 2^-22 of its width (2^-24 for the factor output)
    int steps = 0;
    for (float w = 1.0f; w > (kFactors ? 0x1p-24f : 0x1p-22f); w /= (float)(q + 1)) ++steps;
    for (int st = 0; st < steps; ++st) {
      const float hstep = (hi - lo) / (float)(q + 1);
      const float x = fmaf((float)(pi + 1), hstep, lo);
      float qv = 1.0f;
      uint32_t cnt = 0;
#pragma unroll
      for (int qq = 0; qq < B / 4; ++qq) {
        const float4 d4 = *reinterpret_cast<const float4*>(&sD[it][4 * qq]);
        const float4 e4 = *reinterpret_cast<const float4*>(&sE2[it][4 * qq]);
        const float dd[4] = {d4.x, d4.y, d4.z, d4.w}, ee[4] = {e4.x, e4.y, e4.z, e4.w};
#pragma unroll
        for (int u2 = 0; u2 < 4; ++u2) {
          // q_t = (d_t - x) - e_{t-1}^2 / q_{t-1}, counted by sign bit: a zero
          // pivot makes the next one infinite with the opposite sign, and
          // e^2 >= FLT_MIN keeps 0 * inf out
          qv = fmaf(-ee[u2], __builtin_amdgcn_rcpf(qv), dd[u2] - x);
          cnt += __float_as_uint(qv) >> 31;
        }
      }
      const int nle = __popcll(__ballot((int)cnt <= want) & gmask);
      const float nlo = nle > 0 ? fmaf((float)nle, hstep, lo) : lo;
      const float nhi = nle < q ? fmaf((float)(nle + 1), hstep, lo) : hi;
      lo = nlo;
      hi = nhi;
    }
    const float lam_g = 0.5f * (lo + hi);
    lam = __shfl(lam_g, it * B + (i < ne ? i : ne - 1) * q, 64);
    sLam[it][i] = lam;
  }
  __syncthreads();
  const float top = fmaxf(sLam[it][0], 0.0f);
  const float floor_ = fmaxf(kZeroRel * top, kZeroAbs * energy);
  auto kept = [&](int l) { return l < r && sLam[it][l] > floor_ && sLam[it][l] > 0.0f; };

  // ---- eigenvectors of T for the kept modes: lane l < r runs inverse iteration
  //      for eigenvalue l on T - lambda_l I = L D L^T (no pivoting; a pivot below
  //      eps |T| is replaced by eps |T|), every round followed by modified
  //      Gram-Schmidt over the r vectors (lanes = components)
  float tn = 0.0f;
#pragma unroll
  for (int t = 0; t < B; ++t)
    tn = fmaxf(tn, fabsf(sD[it][t]) + fabsf(sE[it][t]) + (t > 0 ? fabsf(sE[it][t - 1]) : 0.0f));
  const float tiny = fmaxf(tn, 1e-30f) * 1.2e-7f;
  const int lv = i;  // the vector this lane solves for (when i < r)
  if (lv < r) {
    float* M = inv(0, it, lv);
    float* W = inv(1, it, lv);
    float* X = inv(2, it, lv);
    const float lv_lam = lam;
    float pv = sD[it][0] - lv_lam;
    if (fabsf(pv) < tiny) pv = pv < 0.0f ? -tiny : tiny;
    W[0] = pv;
    for (int t = 1; t < B; ++t) {
      const float el = sE[it][t - 1];
      const float m = el / pv;
      pv = (sD[it][t] - lv_lam) - m * el;
      if (fabsf(pv) < tiny) pv = pv < 0.0f ? -tiny : tiny;
      M[t] = m;
      W[t] = pv;
    }
    // start vector: a fixed pattern that differs between the r vectors
    for (int t = 0; t < B; ++t) X[t] = 1.0f + 0.25f * (float)((t * (2 * lv + 3) + lv) % 7);
  }
  for (int round = 0; round < kInvRounds; ++round) {
    if (lv < r) {
      const float* M = inv(0, it, lv);
      const float* W = inv(1, it, lv);
      float* X = inv(2, it, lv);
      // L y = x, then D z = y, then L^T x = z; scaled to unit max to stay finite
      float y = X[0];
      X[0] = y;
      for (int t = 1; t < B; ++t) {
        y = X[t] - M[t] * y;
        X[t] = y;
      }
      float xn = X[B - 1] / W[B - 1];
      X[B - 1] = xn;
      float amax = fabsf(xn);
      for (int t = B - 2; t >= 0; --t) {
        xn = X[t] / W[t] - M[t + 1] * xn;
        X[t] = xn;
        amax = fmaxf(amax, fabsf(xn));
      }
      const float sc = amax > 0.0f ? 1.0f / amax : 1.0f;
      for (int t = 0; t < B; ++t) X[t] *= sc;
    }
    __syncthreads();
    // modified Gram-Schmidt over the vectors in eigenvalue order; lane i holds
    // component i.  Vectors past r are zero and stay zero, so every loop runs at
    // the full width without a branch and the lane reductions can overlap.
    float xr[kMaxR];
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) xr[l] = l < r ? inv(2, it, l)[i] : 0.0f;
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) {
#pragma unroll
      for (int m = 0; m < l; ++m) {
        const float d = group_sum<B>(xr[l] * xr[m]);
        xr[l] = fmaf(-d, xr[m], xr[l]);
      }
      const float nn = group_sum<B>(xr[l] * xr[l]);
      xr[l] = nn > 0.0f ? xr[l] * __builtin_amdgcn_rsqf(nn) : 0.0f;
    }
#pragma unroll
    for (int l = 0; l < kMaxR; ++l)
      if (l < r) inv(2, it, l)[i] = xr[l];
    __syncthreads();
  }

  // ---- back-transformation: u_l = H_0 H_1 ... H_{B-3} x_l, lane i component i
  float u[kMaxR];
#pragma unroll
  for (int l = 0; l < kMaxR; ++l) u[l] = l < r ? inv(2, it, l)[i] : 0.0f;
  // (column k of row i holds v_k[i] for i > k + 1)
  // (vectors past r are zero and stay zero: no branch, the kMaxR reductions overlap)
  for (int k = B - 3; k >= 0; --k) {
    const float vi = i == k + 1 ? 1.0f : (i > k + 1 ? arow[k] : 0.0f);
    const float tau = sTau[it][k];
    float dd[kMaxR];
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) dd[l] = group_sum<B>(vi * u[l]);
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) u[l] = fmaf(-tau * dd[l], vi, u[l]);
  }
  __syncthreads();  // the reflectors are no longer read: U takes their LDS
  float* sU = reinterpret_cast<float*>(sBuf);  // [kI][B][kMaxR + 1]
  auto U_at = [&](int t, int row, int l) -> float& { return sU[(t * B + row) * (kMaxR + 1) + l]; };
#pragma unroll
  for (int l = 0; l < kMaxR; ++l)
    if (l < r) U_at(it, i, l) = u[l];
  __syncthreads();

  // ---- basis columns V[:, l] = D^T u_l / sigma_l over this lane's kCols columns;
  //      the key rows come back from global memory (cache-resident), every row's
  //      slice requested before the first is used
  constexpr int kC = P::kCols;
  constexpr int kW = kC * (int)sizeof(KT) / 4;  // 32-bit words of a row slice
  uint32_t ksl[B][kW];
  {
    const uint32_t* src = reinterpret_cast<const uint32_t*>(kpage + kC * i);
    constexpr int kRowW = kDim * (int)sizeof(KT) / 4;
#pragma unroll
    for (int t = 0; t < B; ++t) {
      if constexpr (kW == 4) {
        const uint4 w = active ? *reinterpret_cast<const uint4*>(src + t * kRowW) : make_uint4(0, 0, 0, 0);
        ksl[t][0] = w.x; ksl[t][1] = w.y; ksl[t][2] = w.z; ksl[t][3] = w.w;
      } else if constexpr (kW == 2) {
        const uint2 w = active ? *reinterpret_cast<const uint2*>(src + t * kRowW) : make_uint2(0, 0);
        ksl[t][0] = w.x; ksl[t][1] = w.y;
      } else {
        ksl[t][0] = active ? src[t * kRowW] : 0u;
      }
    }
  }
  float mu_c[kC];
#pragma unroll
  for (int cc = 0; cc < kC; ++cc) mu_c[cc] = sMu[it][kC * i + cc];
  float vcol[kMaxR][kC];
#pragma unroll
  for (int l = 0; l < kMaxR; ++l)
#pragma unroll
    for (int cc = 0; cc < kC; ++cc) vcol[l][cc] = 0.0f;
#pragma unroll
  for (int t = 0; t < B; ++t) {
    float kv[kC];
#pragma unroll
    for (int cc = 0; cc < kC; ++cc) {
      float x;
      if constexpr (sizeof(KT) == 2)
        x = __uint_as_float((cc & 1) ? (ksl[t][cc >> 1] & 0xffff0000u) : (ksl[t][cc >> 1] << 16));
      else
        x = __uint_as_float(ksl[t][cc]);
      kv[cc] = x - mu_c[cc];
    }
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) {
      if (l < r) {
        const float ul = U_at(it, t, l);
#pragma unroll
        for (int cc = 0; cc < kC; ++cc) vcol[l][cc] = fmaf(kv[cc], ul, vcol[l][cc]);
      }
    }
  }
  // sign convention: the largest |V[c][l]| (lowest c on ties) is made positive:
  // the largest magnitude over the item, then the lowest column holding it, its
  // sign in the low bit
  float best_abs[kMaxR];
#pragma unroll
  for (int l = 0; l < kMaxR; ++l) {
    best_abs[l] = 0.0f;
    if (l >= r) continue;
    const bool kl = kept(l);
    const float sig = kl ? sqrtf(sLam[it][l]) : 1.0f;
    float best = -1.0f, bval = 0.0f;
    int bidx = 0;
#pragma unroll
    for (int cc = 0; cc < kC; ++cc) {
      vcol[l][cc] = kl ? vcol[l][cc] / sig : 0.0f;
      const float av = fabsf(vcol[l][cc]);
      if (av > best) { best = av; bidx = kC * i + cc; bval = vcol[l][cc]; }
    }
    const float gbest = group_max<B>(best);
    const int key = group_min_int<B>(best == gbest ? 2 * bidx + (bval < 0.0f ? 1 : 0) : 0x7fffffff);
    best = gbest;
    const float flip = (key & 1) ? -1.0f : 1.0f;
    if (i == 0) sFlip[it][l] = flip;
#pragma unroll
    for (int cc = 0; cc < kC; ++cc) vcol[l][cc] *= flip;
    best_abs[l] = best;
  }
  __syncthreads();
  // coefficient row i: C[i][l] = flip_l u_l[i] sigma_l (0 for a dropped mode)
  float crow[kMaxR];
#pragma unroll
  for (int l = 0; l < kMaxR; ++l)
    crow[l] = (l < r && kept(l)) ? sFlip[it][l] * u[l] * sqrtf(sLam[it][l]) : 0.0f;

  if (kFactors) {
    if (!active) return;
    const long out_item = (long)e * H_kv + h;
#pragma unroll
    for (int cc = 0; cc < kC; ++cc) mu_out[out_item * kDim + kC * i + cc] = sMu[it][kC * i + cc];
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) {
      if (l >= r) continue;
#pragma unroll
      for (int cc = 0; cc < kC; ++cc)
        basis_out[(out_item * kDim + kC * i + cc) * r + l] = vcol[l][cc];
    }
#pragma unroll
    for (int l = 0; l < kMaxR; ++l)
      if (l < r) coef_out[(out_item * B + i) * r + l] = crow[l];
    sigma2_out[out_item * B + i] = fmaxf(sLam[it][i], 0.0f);
    return;
  }

  // ---- quantise and pack the record in LDS, then copy it out with 16-byte stores
  const int stride = rec_stride(r, basis, B);
  uint8_t* sRec = sBuf + it * stride;
  const int scale_off = rec_scale_off(r, basis, B);
#pragma unroll
  for (int l = 0; l < kMaxR; ++l) {
    if (l >= r) continue;
    if (basis == LOCKS_BASIS_INT4) {
      const float vs = f16_scale(best_abs[l], 7.0f);
      uint32_t word = 0;
#pragma unroll
      for (int cc = 0; cc < kC; ++cc) word |= (uint32_t)(quant(vcol[l][cc], vs, 7) + 8) << (4 * cc);
      uint8_t* dst = sRec + 64 * l + (kC / 2) * i;
#pragma unroll
      for (int bb = 0; bb < kC / 2; ++bb) dst[bb] = (uint8_t)(word >> (8 * bb));
      if (i == 0) *reinterpret_cast<uint16_t*>(sRec + scale_off + 2 * l) = f16_bits(vs);
    } else if (basis == LOCKS_BASIS_INT8) {
      const float vs = f16_scale(best_abs[l], 127.0f);
#pragma unroll
      for (int cc = 0; cc < kC; ++cc)
        sRec[128 * l + kC * i + cc] = (uint8_t)(quant(vcol[l][cc], vs, 127) + 128);
      if (i == 0) *reinterpret_cast<uint16_t*>(sRec + scale_off + 2 * l) = f16_bits(vs);
    } else {
#pragma unroll
      for (int cc = 0; cc < kC; ++cc)
        *reinterpret_cast<uint16_t*>(sRec + 256 * l + 2 * (kC * i + cc)) =
            (uint16_t)bf16_rne_bits(vcol[l][cc]);
      if (i == 0) *reinterpret_cast<uint16_t*>(sRec + scale_off + 2 * l) = f16_bits(1.0f);
    }
  }
  {
    float cabs = 0.0f;
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) cabs = fmaxf(cabs, fabsf(crow[l]));
    const float cs = f16_scale(cabs, 127.0f);
    const int coef_off = rec_coef_off(r, basis);
#pragma unroll
    for (int l = 0; l < kMaxR; ++l)
      if (l < r) sRec[coef_off + i * r + l] = (uint8_t)(quant(crow[l], cs, 127) + 128);
    *reinterpret_cast<uint16_t*>(sRec + scale_off + 2 * (r + i)) = f16_bits(cs);
  }
  {
    float m = 0.0f;
#pragma unroll
    for (int cc = 0; cc < kC; ++cc) m = fmaxf(m, fabsf(sMu[it][kC * i + cc]));
    m = group_max<B>(m);
    const float ms = f16_scale(m, 127.0f);
    const int mu_off = rec_mu_off(r, basis, B);
#pragma unroll
    for (int cc = 0; cc < kC; ++cc)
      sRec[mu_off + kC * i + cc] = (uint8_t)(quant(sMu[it][kC * i + cc], ms, 127) + 128);
    if (i == 0) *reinterpret_cast<uint16_t*>(sRec + scale_off + 2 * (r + B)) = f16_bits(ms);
  }
  for (int o = rec_payload(r, basis, B) + i; o < stride; o += B) sRec[o] = 0;
  __syncthreads();
  if (!active) return;
  uint8_t* rec = summaries + (blk * H_kv + h) * (long)stride;
  for (int o = 16 * i; o < stride; o += 16 * B)
    *reinterpret_cast<uint4*>(rec + o) = *reinterpret_cast<const uint4*>(sRec + o);
}

}  // namespace

hipError_t launch_build_page(const locks_cfg_t& c, const void* k_cache, const int32_t* page_table,
                             const int32_t* seq_lens, const int32_t* build_list, int32_t n_items,
                             bool all_pages, void* summaries, float* mu, float* basis,
                             float* coef, float* sigma2, hipStream_t st) {
  const long items = all_pages ? (long)c.num_seqs * c.max_pages_per_seq * c.num_kv_heads
                               : (long)n_items * c.num_kv_heads;
  if (items == 0) return hipSuccess;
  const bool factors = mu != nullptr;
  const int per = 64 / c.page_size;
  const long blocks = (items + per - 1) / per;
  if (blocks > 0x7fffffffL) return hipErrorInvalidConfiguration;
  const dim3 grid((unsigned)blocks), block(64);
  // ranks up to 8 take the instance whose rank-sized arrays (LDS and registers)
  // hold 8 vectors: its smaller LDS fits more waves per compute unit
#define LOCKS_BUILD_PAGE_R(KT, BP, F, MR)                                                      \
  hipLaunchKernelGGL((build_page_kernel<KT, BP, F, MR>), grid, block, 0, st, c.num_seqs,        \
                     c.num_kv_heads, c.max_pages_per_seq, c.rank, static_cast<const KT*>(k_cache), \
                     page_table, seq_lens, build_list, n_items, (int)all_pages,                \
                     (uint8_t*)summaries, mu, basis, coef, sigma2, c.basis)
#define LOCKS_BUILD_PAGE(KT, BP, F)                                                            \
  if (c.rank <= 8) LOCKS_BUILD_PAGE_R(KT, BP, F, 8); else LOCKS_BUILD_PAGE_R(KT, BP, F, kMaxRank)
#define LOCKS_BUILD_PAGE_B(KT)                                                                 \
  switch (c.page_size) {                                                                       \
    case 32: if (factors) LOCKS_BUILD_PAGE(KT, 32, true); else LOCKS_BUILD_PAGE(KT, 32, false); break; \
    case 64: if (factors) LOCKS_BUILD_PAGE(KT, 64, true); else LOCKS_BUILD_PAGE(KT, 64, false); break; \
    default: return hipErrorInvalidValue;                                                      \
  }
  if (c.kv_dtype == LOCKS_BF16) {
    LOCKS_BUILD_PAGE_B(uint16_t);
  } else {
    LOCKS_BUILD_PAGE_B(float);
  }
#undef LOCKS_BUILD_PAGE_B
#undef LOCKS_BUILD_PAGE
#undef LOCKS_BUILD_PAGE_R
  return hipGetLastError();
}

}  // namespace locks
