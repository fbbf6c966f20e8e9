// Symmetric 16 x 16 eigensolver on one 16-lane row of a wave, everything in
// registers (Sec. 4 "Build": the leading eigenpairs of a page's Gram).
//
// Lane i of the row owns row i of A.  Cross-lane traffic is DPP only: lane k's
// value reaches the whole row by a row broadcast, row sums take four DPP steps.
//  1. Householder reduction to tridiagonal T = Q^T A Q.  At step k every lane
//     receives row k (= column k) and forms the reflector v and its scale tau
//     itself; p = tau A v is formed per lane and broadcast; each lane updates its
//     row by A - v w^T - w v^T and keeps v_k[i] in a[k] for the back-transform.
//  2. Eigenvalues of T by multisection on Sturm counts: the 16 lanes are split
//     into groups of q = 16 / n lanes for the n eigenvalues wanted, each lane
//     tests one point per step, so a group cuts its interval into q + 1 parts;
//     a wave ballot gives the part that holds the eigenvalue.  Steps continue
//     until the Gershgorin width is cut by 2^22 (2^24 when all 16 are wanted).
//  3. Eigenvectors of T for the r leading eigenvalues by inverse iteration on
//     T - lambda I = L D L^T (lane l solves for vector l; a pivot below
//     1.2e-7 |T| is replaced by that value, which only scales the solution),
//     two rounds, each followed by modified Gram-Schmidt over the r vectors so
//     that a near-degenerate pair still spans its eigenspace.
//  4. Back-transformation u_l = H_0 H_1 ... H_13 x_l.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>
#include <utility>

namespace locks {
namespace tri16 {

constexpr int kN = 16;
constexpr int kXRow = 20;  // LDS stride (floats) of one vector in the scratch

template <int C>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), C, 0xF, 0xF, false));
}
// the value of lane K of this lane's 16-lane row
template <int K>
__device__ __forceinline__ float bcast(float v) {
  return dpp<0x150 + K>(v);
}
// sum over the 16 lanes of the row: quad xor 1, quad xor 2, half-row mirror, row mirror
__device__ __forceinline__ float row_sum(float v) {
  v += dpp<0xB1>(v);
  v += dpp<0x4E>(v);
  v += dpp<0x141>(v);
  v += dpp<0x140>(v);
  return v;
}
// N independent row sums, stage by stage (each DPP step waits on the previous
// write of its own operand only)
template <int N>
__device__ __forceinline__ void row_sums(float (&v)[N]) {
#pragma unroll
  for (int n = 0; n < N; ++n) v[n] += dpp<0xB1>(v[n]);
#pragma unroll
  for (int n = 0; n < N; ++n) v[n] += dpp<0x4E>(v[n]);
#pragma unroll
  for (int n = 0; n < N; ++n) v[n] += dpp<0x141>(v[n]);
#pragma unroll
  for (int n = 0; n < N; ++n) v[n] += dpp<0x140>(v[n]);
}

// f(std::integral_constant<int, N>) for the smallest N in {2, 4, 8, NMax} with
// r <= N: loops over the r leading vectors then run at a fixed width
template <int NMax, typename F>
__device__ __forceinline__ void with_width(int r, F&& f) {
  if (r <= 2) f(std::integral_constant<int, 2>{});
  else if (r <= 4) f(std::integral_constant<int, 4>{});
  else if (r <= 8) f(std::integral_constant<int, 8>{});
  else f(std::integral_constant<int, NMax>{});
}

template <typename F, int... Ks>
__device__ __forceinline__ void for_each_int(F& f, std::integer_sequence<int, Ks...>) {
  (f(std::integral_constant<int, Ks>{}), ...);
}
// f(std::integral_constant<int, k>) for k = 0 .. N - 1, in order
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  for_each_int(f, std::make_integer_sequence<int, N>{});
}

// a: row i of A (consumed: holds the reflectors afterwards).  kAll: all 16
// eigenvalues are wanted (else the r leading ones).  On return lam is the i-th
// largest eigenvalue (for i < r, or every i with kAll) and u[l] (l < r) is
// component i of the unit eigenvector of the l-th largest.  scratch: 16 x kXRow
// floats of LDS owned by this row; the caller's wave runs this code without
// divergence (every lane of the wave, DPP reads neighbouring lanes).
template <bool kAll, int kMaxR>
__device__ __forceinline__ void eig16(float (&a)[kN], const int i, const int r, float& lam,
                                      float (&u)[kMaxR], float* scratch) {
  float d[kN], e[kN], tau[kN - 2];

  // ---- 1. Householder reduction
  static_for<kN - 2>([&](auto kc) __attribute__((always_inline)) {
    constexpr int k = decltype(kc)::value;
    float x[kN];  // column k below the diagonal, from lane k's row
#pragma unroll
    for (int j = k; j < kN; ++j) x[j] = bcast<k>(a[j]);
    d[k] = x[k];
    float sig = 0.0f;
#pragma unroll
    for (int j = k + 2; j < kN; ++j) sig = fmaf(x[j], x[j], sig);
    const float x0 = x[k + 1];
    // (hardware square root and reciprocals: the reflector need only be
    // orthogonal to a few ulp, which its own tau guarantees)
    float t = 0.0f, v0 = 1.0f, beta = x0;
    if (sig > 0.0f) {
      const float mu = __builtin_amdgcn_sqrtf(fmaf(x0, x0, sig));
      v0 = x0 <= 0.0f ? x0 - mu : -sig * __builtin_amdgcn_rcpf(x0 + mu);
      t = 2.0f * v0 * v0 * __builtin_amdgcn_rcpf(fmaf(v0, v0, sig));
      beta = mu;
    }
    e[k] = beta;
    tau[k] = t;
    float v[kN];
    const float iv0 = sig > 0.0f ? __builtin_amdgcn_rcpf(v0) : 0.0f;
    v[k + 1] = 1.0f;
#pragma unroll
    for (int j = k + 2; j < kN; ++j) v[j] = x[j] * iv0;
    float vi = 0.0f, p = 0.0f;
#pragma unroll
    for (int j = k + 1; j < kN; ++j) {
      vi = i == j ? v[j] : vi;
      p = fmaf(a[j], v[j], p);
    }
    p = i > k ? t * p : 0.0f;
    float pj[kN];
    static_for<kN>([&](auto jc) __attribute__((always_inline)) {
      constexpr int j = decltype(jc)::value;
      if constexpr (j > k) pj[j] = bcast<j>(p);
    });
    float kv = 0.0f;
#pragma unroll
    for (int j = k + 1; j < kN; ++j) kv = fmaf(pj[j], v[j], kv);
    kv *= 0.5f * t;
    const float wi = p - kv * vi;
#pragma unroll
    for (int j = k + 1; j < kN; ++j) {
      const float wj = fmaf(-kv, v[j], pj[j]);
      a[j] = fmaf(-vi, wj, fmaf(-wi, v[j], a[j]));
    }
    a[k] = vi;  // 0 above row k + 1, 1 at row k + 1
  });
  d[kN - 2] = bcast<kN - 2>(a[kN - 2]);
  e[kN - 2] = bcast<kN - 1>(a[kN - 2]);
  d[kN - 1] = bcast<kN - 1>(a[kN - 1]);
  e[kN - 1] = 0.0f;

  // ---- 2. eigenvalues by multisection
  float lo = INFINITY, hi = -INFINITY, tn = 0.0f;
  float e2[kN];
#pragma unroll
  for (int t = 0; t < kN; ++t) {
    const float el = t > 0 ? fabsf(e[t - 1]) : 0.0f;
    const float er = fabsf(e[t]);
    lo = fminf(lo, d[t] - el - er);
    hi = fmaxf(hi, d[t] + el + er);
    tn = fmaxf(tn, fabsf(d[t]) + el + er);
    // (the floor moves eigenvalues by at most 1e-19; an all-zero T has a zero-width
    // interval, so its eigenvalues stay exactly 0)
    e2[t] = t > 0 ? fmaf(e[t - 1], e[t - 1], 0x1p-126f) : 0.0f;
  }
  const int ne = kAll ? kN : r;            // eigenvalues wanted: the ne largest
  const int q = kN / ne;                   // lanes per eigenvalue
  const int lq = i / q;
  const bool idle = lq >= ne;              // lanes past ne * q copy the last group
  const int le = idle ? ne - 1 : lq;       // the eigenvalue (0 = largest)
  const int pi = idle ? 0 : i - lq * q;    // this lane's first point is kPts * pi
  const int want = kN - 1 - le;            // count(x) <= want  <=>  x <= lambda_le
  constexpr int kPts = 1;                  // points per lane and step
  const int npts = kPts * q;
  const int row0 = threadIdx.x & 48;
  const uint64_t gmask = ((1ull << q) - 1ull) << (row0 + le * q);
  // the Sturm counts carry rounding of a few ulp of |T|, so the interval is cut to
  // 2^-22 of its width (2^-24 when every eigenvalue is reported)
  int steps = 0;
  for (float w = 1.0f; w > (kAll ? 0x1p-24f : 0x1p-22f); w /= (float)(npts + 1)) ++steps;
  for (int st = 0; st < steps; ++st) {
    const float h = (hi - lo) / (float)(npts + 1);
    float qv[kPts], xv[kPts];
    uint32_t cnt[kPts];
#pragma unroll
    for (int pp = 0; pp < kPts; ++pp) {
      xv[pp] = fmaf((float)(kPts * pi + pp + 1), h, lo);
      qv[pp] = 1.0f;
      cnt[pp] = 0;
    }
#pragma unroll
    for (int t = 0; t < kN; ++t) {
      // q_t = (d_t - x) - e_{t-1}^2 / q_{t-1}, counted by sign bit.  A zero pivot
      // makes the next one infinite with the opposite sign (one count either
      // way), and e^2 >= FLT_MIN keeps 0 * inf out.  The hardware reciprocal's
      // last-bit error moves only counts at x within rounding of an eigenvalue.
#pragma unroll
      for (int pp = 0; pp < kPts; ++pp) {
        qv[pp] = fmaf(-e2[t], __builtin_amdgcn_rcpf(qv[pp]), d[t] - xv[pp]);
        cnt[pp] += __float_as_uint(qv[pp]) >> 31;
      }
    }
    int nle = 0;
#pragma unroll
    for (int pp = 0; pp < kPts; ++pp) nle += __popcll(__ballot((int)cnt[pp] <= want) & gmask);
    const float nlo = nle > 0 ? fmaf((float)nle, h, lo) : lo;
    const float nhi = nle < npts ? fmaf((float)(nle + 1), h, lo) : hi;
    lo = nlo;
    hi = nhi;
  }
  const float lam_g = 0.5f * (lo + hi);
  lam = __shfl(lam_g, row0 + (i < ne ? i : ne - 1) * q, 64);

  // ---- 3. eigenvectors of T: lane l < r solves for vector l
  const float tiny = fmaxf(tn, 1e-30f) * 1.2e-7f;
  float M[kN], Wi[kN], X[kN];
  {
    float pv = d[0] - lam;
    if (fabsf(pv) < tiny) pv = pv < 0.0f ? -tiny : tiny;
    Wi[0] = __builtin_amdgcn_rcpf(pv);
    M[0] = 0.0f;
#pragma unroll
    for (int t = 1; t < kN; ++t) {
      const float m = e[t - 1] * Wi[t - 1];
      pv = (d[t] - lam) - m * e[t - 1];
      if (fabsf(pv) < tiny) pv = pv < 0.0f ? -tiny : tiny;
      M[t] = m;
      Wi[t] = __builtin_amdgcn_rcpf(pv);
    }
    // start vector: a fixed pattern that differs between the vectors
#pragma unroll
    for (int t = 0; t < kN; ++t) X[t] = 1.0f + 0.25f * (float)((t * (2 * i + 3) + i) % 7);
  }
#pragma unroll
  for (int round = 0; round < 2; ++round) {
    // L y = x, D z = y, L^T x = z, scaled to unit max
#pragma unroll
    for (int t = 1; t < kN; ++t) X[t] = fmaf(-M[t], X[t - 1], X[t]);
    X[kN - 1] *= Wi[kN - 1];
    float amax = fabsf(X[kN - 1]);
#pragma unroll
    for (int t = kN - 2; t >= 0; --t) {
      X[t] = fmaf(-M[t + 1], X[t + 1], X[t] * Wi[t]);
      amax = fmaxf(amax, fabsf(X[t]));
    }
    const float sc = amax > 0.0f ? __builtin_amdgcn_rcpf(amax) : 1.0f;
    // modified Gram-Schmidt over the vectors in eigenvalue order, lane i
    // holding component i (the transposition goes through LDS; one wave, so
    // its LDS accesses complete in issue order)
    if (i < r) {
#pragma unroll
      for (int c = 0; c < kN / 4; ++c)
        reinterpret_cast<float4*>(scratch + i * kXRow)[c] =
            make_float4(X[4 * c] * sc, X[4 * c + 1] * sc, X[4 * c + 2] * sc, X[4 * c + 3] * sc);
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int l = 0; l < kMaxR; ++l) u[l] = l < r ? scratch[l * kXRow + i] : 0.0f;
    // (right-looking: once u_m is final it is projected out of every later
    // vector at once; each vector sees the same operations in the same order
    // as in the left-looking loop; vectors past r are 0 and stay 0)
    with_width<kMaxR>(r, [&](auto nc) __attribute__((always_inline)) {
      constexpr int N = decltype(nc)::value;
      static_for<N>([&](auto mc) __attribute__((always_inline)) {
        constexpr int m = decltype(mc)::value;
        const float nn = row_sum(u[m] * u[m]);
        u[m] = nn > 0.0f ? u[m] * __builtin_amdgcn_rsqf(nn) : 0.0f;
        if constexpr (m + 1 < N) {
          float t[N - 1 - m];
#pragma unroll
          for (int l = m + 1; l < N; ++l) t[l - m - 1] = u[l] * u[m];
          row_sums(t);
#pragma unroll
          for (int l = m + 1; l < N; ++l) u[l] = fmaf(-t[l - m - 1], u[m], u[l]);
        }
      });
    });
    if (round == 0) {
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int l = 0; l < kMaxR; ++l)
        if (l < r) scratch[l * kXRow + i] = u[l];
      __builtin_amdgcn_wave_barrier();
      if (i < r) {
#pragma unroll
        for (int c = 0; c < kN / 4; ++c) {
          const float4 v = reinterpret_cast<const float4*>(scratch + i * kXRow)[c];
          X[4 * c] = v.x; X[4 * c + 1] = v.y; X[4 * c + 2] = v.z; X[4 * c + 3] = v.w;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }

  // ---- 4. back-transformation through the stored reflectors
  static_for<kN - 2>([&](auto kc) __attribute__((always_inline)) {
    constexpr int k = kN - 3 - decltype(kc)::value;
    const float vk = a[k];
    const float tk = tau[k];
    with_width<kMaxR>(r, [&](auto nc) __attribute__((always_inline)) {
      constexpr int N = decltype(nc)::value;
      float s[N];
#pragma unroll
      for (int l = 0; l < N; ++l) s[l] = vk * u[l];
      row_sums(s);
#pragma unroll
      for (int l = 0; l < N; ++l) u[l] = fmaf(-tk * s[l], vk, u[l]);
    });
  });
}

}  // namespace tri16
}  // namespace locks
