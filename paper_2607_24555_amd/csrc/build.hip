// Per-page summary construction (Sec. 4 "Build"): centre the page's 16 keys,
// eigendecompose the 16 x 16 Gram of the deviations, keep the r leading nonzero
// modes, form V = D^T U_r S_r^{-1} and C = U_r S_r, quantise and pack.
//
// Mapping: one 64-lane wave per block, four (page, KV head) items per wave, 16
// lanes per item with lane i owning row i of the page.  The Gram is formed on the
// matrix cores with the same summation order for (i, j) and (j, i), so it is
// exactly symmetric; its eigenpairs come from the register-resident tridiagonal
// solver of tridiag16.h (one 16-lane DPP row per item).  Everything is fp32.
#include "locks_internal.h"
#include "tridiag16.h"

namespace locks {
namespace {

constexpr int kItems = 4;         // items per block

typedef float f4 __attribute__((ext_vector_type(4)));
constexpr int kRow = 20;          // LDS row stride of A and U: 16-byte aligned, conflict-free
constexpr int kARows = kPage + 1; // rows per item of A and U: the spare row moves the four
                                  // items' rows to different banks
constexpr int kKPad = 16;         // bytes after each key row: consecutive rows start 4 banks apart
constexpr float kZeroRel = 1e-6f;
constexpr float kZeroAbs = 1e-10f;

// The block is a single wave, whose LDS operations complete in issue order: a
// barrier inside the rotation rounds only has to keep the compiler from moving
// LDS accesses across it.
__device__ __forceinline__ void wave_sync() { __builtin_amdgcn_wave_barrier(); }

__device__ __forceinline__ void ld_row(const float* p, float (&r)[kPage]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 v = reinterpret_cast<const float4*>(p)[q];
    r[4 * q] = v.x; r[4 * q + 1] = v.y; r[4 * q + 2] = v.z; r[4 * q + 3] = v.w;
  }
}

// sum / max over the 16 lanes of an item (one DPP row)
__device__ __forceinline__ float group16_sum(float v) { return tri16::row_sum(v); }
__device__ __forceinline__ float group16_max(float v) {
  v = fmaxf(v, tri16::dpp<0xB1>(v));
  v = fmaxf(v, tri16::dpp<0x4E>(v));
  v = fmaxf(v, tri16::dpp<0x141>(v));
  return fmaxf(v, tri16::dpp<0x140>(v));
}

__device__ __forceinline__ int group16_min_int(int v) {
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false));
  v = min(v, __builtin_amdgcn_update_dpp(0, v, 0x141, 0xF, 0xF, false));
  return min(v, __builtin_amdgcn_update_dpp(0, v, 0x140, 0xF, 0xF, false));
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

// 1 / s for a code scale s (0 when s is 0: every code is then 0)
__device__ __forceinline__ float inv_scale(float s) { return s > 0.0f ? 1.0f / s : 0.0f; }
// code of x at scale 1 / inv: nearest integer, clamped to +-qmax (x inv may differ
// from x / s in the last bit, which moves a code only at an exact half)
__device__ __forceinline__ int quant(float x, float inv, int qmax) {
  float c = rintf(x * inv);
  c = fminf(fmaxf(c, (float)-qmax), (float)qmax);
  return (int)c;
}

// Nearest bfloat16 (ties to even) of a finite float, as its 16-bit pattern.
__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint16_t f16_bits(float s) {
  _Float16 h = (_Float16)s;
  return *reinterpret_cast<uint16_t*>(&h);
}

// kMode (BuildMode): kBuildAll builds every listed (or complete) page; kBuildInner
// skips the pages that are the last complete page of their sequence, and its block 0
// instead prepares the scan of the step (scan lengths without those pages);
// kBuildLast builds only those pages and scores them for the step's query (Eq. 1
// on the decoded summary), writing their page scores and one extra (max, sum)
// partial per query head of their sequence.
template <typename KT, bool kFactors, int kMode>
__global__ __launch_bounds__(64) void build_kernel(
    int S, int H_kv, int max_pages, int r, const KT* __restrict__ k_cache,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ build_list, int n_items, int all_pages,
    uint8_t* __restrict__ summaries, float* __restrict__ mu_out, float* __restrict__ basis_out,
    float* __restrict__ coef_out, float* __restrict__ sigma2_out, BuildStep bs, int basis) {
  constexpr bool kScore = kMode == kBuildLast;  // (int4 bases only)
  // raw key rows (bf16 or fp32 as stored; deviations are formed on the fly as
  // float(k) - mu, the same fp32 value for every use) share LDS with the Gram A
  // and the eigenvectors U, which are written once the Gram is complete
  constexpr int kKRow = kDim + kKPad / (int)sizeof(KT);  // key row stride (elements)
  constexpr int kKBytes = kItems * kPage * kKRow * (int)sizeof(KT);
  constexpr int kJBytes = 2 * kItems * kARows * kRow * (int)sizeof(float);
  __shared__ __align__(16) uint8_t sBuf[kKBytes > kJBytes ? kKBytes : kJBytes];
  auto& sK = *reinterpret_cast<KT(*)[kItems][kPage][kKRow]>(sBuf);
  auto& sA = *reinterpret_cast<float(*)[kItems][kARows][kRow]>(sBuf);
  auto& sU = *reinterpret_cast<float(*)[kItems][kARows][kRow]>(sBuf + kJBytes / 2);
  __shared__ float sFlip[kItems][kMaxRank];
  __shared__ float sMu[kItems][kDim];
  __shared__ float sLam[kItems][kPage];
  // quantised basis columns (packed codes, scales) and projections of the scored pages
  __shared__ uint32_t sVw[kScore ? kItems : 1][kScore ? kMaxRank : 1][kScore ? kPage : 1];
  __shared__ float sVs[kScore ? kItems : 1][kScore ? kMaxRank : 1];
  __shared__ float sP[kScore ? kItems : 1][kScore ? kMaxRank : 1];

  if (kMode == kBuildInner && blockIdx.x == 0) {
    // scan lengths: a sequence whose last complete page is listed is scanned
    // without it (kBuildLast scores that page and writes its extra partials)
    for (int i = threadIdx.x; i < S; i += 64) bs.sl_scan[i] = seq_lens[i];
    __threadfence();  // the stores above complete before the ones below
    __syncthreads();
    for (int e = threadIdx.x; e < n_items; e += 64) {
      const int ss = build_list[2 * e], jj = build_list[2 * e + 1];
      if (ss < 0 || ss >= S) continue;
      const int L = seq_lens[ss];
      if (jj >= 0 && jj < max_pages && jj == L / kPage - 1) bs.sl_scan[ss] = L - kPage;
    }
    return;
  }

  const int grp = threadIdx.x >> 4;
  const int li = threadIdx.x & 15;
  const long item = (long)(kMode == kBuildInner ? blockIdx.x - 1 : blockIdx.x) * kItems + grp;

  // ---- which (seq, page, KV head) this group builds
  bool active = false;
  int s = 0, j = 0, h = 0, e = 0;
  if (all_pages) {
    h = (int)(item % H_kv);
    long t = item / H_kv;
    j = (int)(t % max_pages);
    s = (int)(t / max_pages);
    active = s < S && j < seq_lens[s] / kPage;
  } else {
    h = (int)(item % H_kv);
    e = (int)(item / H_kv);
    if (e < n_items) {
      s = build_list[2 * e];
      j = build_list[2 * e + 1];
      active = s >= 0 && s < S && j >= 0 && j < max_pages && j < seq_lens[s] / kPage;
      if (active && kMode != kBuildAll) {
        const bool last = j == seq_lens[s] / kPage - 1;
        active = kMode == kBuildLast ? last : !last;
      }
    }
  }
  if (!__any(active)) return;  // the block is one wave: nothing to build
  // the scored builds run beside the scan and lead the step's critical path:
  // their instructions go first on a shared SIMD
  if (kMode == kBuildLast) __builtin_amdgcn_s_setprio(3);
  const long blk = active ? (long)page_table[(long)s * max_pages + j] : 0;

  // ---- load row li of the page (16-byte loads), track its squared norm
  float energy = 0.0f;
  {
    constexpr int kVec = 16 / sizeof(KT);  // elements per 16-byte load
    const uint4* src = reinterpret_cast<const uint4*>(k_cache + ((blk * H_kv + h) * kPage + li) * kDim);
    uint4* dst = reinterpret_cast<uint4*>(&sK[grp][li][0]);
    uint4 w[kDim / kVec];
#pragma unroll
    for (int u = 0; u < kDim / kVec; ++u) w[u] = active ? src[u] : make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int u = 0; u < kDim / kVec; ++u) dst[u] = w[u];
#pragma unroll
    for (int u = 0; u < kDim / kVec; ++u) {
      float x[kVec];
      chunk_to_f<KT>(w[u], x);
#pragma unroll
      for (int c = 0; c < kVec; ++c) energy = fmaf(x[c], x[c], energy);
    }
    __syncthreads();
  }
  energy = group16_sum(energy) * (1.0f / kPage);

  // ---- centroid of the lane's 8 columns: pairwise sum over the 16 rows (exact
  //      for equal rows)
  {
    float v[kPage][8];
#pragma unroll
    for (int i = 0; i < kPage; ++i) {
      const uint4* row = reinterpret_cast<const uint4*>(&sK[grp][i][8 * li]);
#pragma unroll
      for (int u = 0; u < 8 / (16 / (int)sizeof(KT)); ++u)
        chunk_to_f<KT>(row[u], &v[i][u * (16 / (int)sizeof(KT))]);
    }
#pragma unroll
    for (int w = 8; w > 0; w >>= 1)
#pragma unroll
      for (int i = 0; i < w; ++i)
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) v[i][cc] = v[i][cc] + v[i + w][cc];
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) sMu[grp][8 * li + cc] = v[0][cc] * (1.0f / kPage);
  }
  __syncthreads();

  // ---- Gram of the deviations on the matrix cores, one item at a time: lane
  //      (grp, li) supplies deviation row li at columns 32 grp + m as both
  //      operands of 32 fp32 MFMAs 16x16x4, which leave G[4 grp + jj][li] in
  //      register jj; the upper triangle is then mirrored so A is exactly
  //      symmetric
  {
    f4 acc[kItems];
#pragma unroll
    for (int it = 0; it < kItems; ++it) {
      acc[it] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      constexpr int kVec = 16 / (int)sizeof(KT);
#pragma unroll
      for (int ch = 0; ch < 32 / kVec; ++ch) {
        const int c0 = 32 * grp + kVec * ch;
        float x[kVec];
        chunk_to_f<KT>(*reinterpret_cast<const uint4*>(&sK[it][li][c0]), x);
#pragma unroll
        for (int m = 0; m < kVec; ++m) {
          const float d = x[m] - sMu[it][c0 + m];
          acc[it] = __builtin_amdgcn_mfma_f32_16x16x4f32(d, d, acc[it], 0, 0, 0);
        }
      }
    }
    __syncthreads();  // every lane is done with the key rows: A and U reuse their LDS
#pragma unroll
    for (int it = 0; it < kItems; ++it)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) sA[it][4 * grp + jj][li] = acc[it][jj];
    __syncthreads();
#pragma unroll
    for (int jj = 0; jj < kPage; ++jj)
      if (jj < li) sA[grp][li][jj] = sA[grp][jj][li];
  }
  __syncthreads();

  // ---- eigenpairs of the Gram: Householder tridiagonalisation, multisection
  //      and inverse iteration in registers; the solver's LDS scratch is A's
  {
    float a[kPage];
    ld_row(&sA[grp][li][0], a);
    __syncthreads();
    float lam, u[kMaxRank];
    tri16::eig16<kFactors, kMaxRank>(a, li, r, lam, u, &sA[grp][0][0]);
    sLam[grp][li] = fmaxf(lam, 0.0f);
#pragma unroll
    for (int l = 0; l < kMaxRank; ++l)
      if (l < r) sU[grp][li][l] = u[l];
  }
  __syncthreads();
  const float top = sLam[grp][0];
  const float floor_ = fmaxf(kZeroRel * top, kZeroAbs * energy);

  const long out_item = all_pages ? 0 : (long)e * H_kv + h;
  uint8_t* rec = summaries + (blk * H_kv + h) * (long)rec_stride(r, basis);

  // ---- basis columns V[:, l] = D^T u_l / sigma_l.  This lane's 8 dimensions of
  //      the 16 key rows are re-read from global memory (the page was just
  //      loaded, so they come from cache) and held in registers.
  constexpr int kSliceVec = 8 * (int)sizeof(KT) / 16;  // 16-byte loads per 8-element slice
  uint4 ks[kPage][kSliceVec];
  {
    const uint4* kpage = reinterpret_cast<const uint4*>(k_cache + (blk * H_kv + h) * kPage * kDim);
#pragma unroll
    for (int i = 0; i < kPage; ++i)
#pragma unroll
      for (int u = 0; u < kSliceVec; ++u)
        ks[i][u] = active ? kpage[(i * kDim + 8 * li) / (16 / (int)sizeof(KT)) + u]
                          : make_uint4(0, 0, 0, 0);
  }
  float cabs = 0.0f;  // running max |C[li][:]| for the row scale
  float mu8[8];
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) mu8[cc] = sMu[grp][8 * li + cc];
  // four modes at a time: each key row is converted once per pass and
  // multiplies the four eigenvector components of that row (one LDS broadcast)
  constexpr int kMG = 4;
#pragma unroll 1
  for (int l0 = 0; l0 < r; l0 += kMG) {
    float vacc[kMG][8];
#pragma unroll
    for (int m = 0; m < kMG; ++m)
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) vacc[m][cc] = 0.0f;
#pragma unroll
    for (int i = 0; i < kPage; ++i) {
      const float4 ua = *reinterpret_cast<const float4*>(&sU[grp][i][l0]);
      const float ui[kMG] = {ua.x, ua.y, ua.z, ua.w};
      float x[8];
#pragma unroll
      for (int u = 0; u < kSliceVec; ++u) chunk_to_f<KT>(ks[i][u], &x[u * (16 / (int)sizeof(KT))]);
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const float dv = x[cc] - mu8[cc];
#pragma unroll
        for (int m = 0; m < kMG; ++m) vacc[m][cc] = fmaf(dv, ui[m], vacc[m][cc]);
      }
    }
#pragma unroll
    for (int m = 0; m < kMG; ++m) {
      const int l = l0 + m;
      if (l >= r) break;
      const float lam = sLam[grp][l];
      const bool kept = lam > floor_ && lam > 0.0f;
      const float isig = kept ? 1.0f / sqrtf(lam) : 0.0f;
      const float sig = kept ? sqrtf(lam) : 1.0f;
      float v[8];
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) v[cc] = vacc[m][cc] * isig;
      // sign convention: largest |v| (first index on ties) made positive: the
      // largest magnitude over the item, then the lowest index holding it, with
      // its sign in the low bit
      float best = -1.0f;
      int bidx = 0;
      float bval = 0.0f;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const float a = fabsf(v[cc]);
        if (a > best) { best = a; bidx = 8 * li + cc; bval = v[cc]; }
      }
      const float gbest = group16_max(best);
      const int key = group16_min_int(best == gbest ? 2 * bidx + (bval < 0.0f ? 1 : 0) : 0x7fffffff);
      best = gbest;
      bval = (key & 1) ? -1.0f : 1.0f;
      const float flip = (bval < 0.0f) ? -1.0f : 1.0f;
      const float cval = kept ? flip * sU[grp][li][l] * sig : 0.0f;
      if (li == 0) sFlip[grp][l] = flip;
      cabs = fmaxf(cabs, fabsf(cval));
      if (!active) continue;
      if (kFactors) {
        float* bo = basis_out + out_item * (kDim * (long)r);
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) bo[(8 * li + cc) * r + l] = flip * v[cc];
      } else {
        if (basis == 0) {  // int4, excess 8, two per byte
          const float vs = f16_scale(best, 7.0f);
          const float ivs = inv_scale(vs);
          uint32_t word = 0;
#pragma unroll
          for (int cc = 0; cc < 8; ++cc) {
            const int code = quant(flip * v[cc], ivs, 7);
            word |= (uint32_t)(code + 8) << (4 * cc);
          }
          *reinterpret_cast<uint32_t*>(rec + 64 * l + 4 * li) = word;
          if (li == 0) *reinterpret_cast<uint16_t*>(rec + rec_scale_off(r) + 2 * l) = f16_bits(vs);
          if (kScore) {
            sVw[grp][l][li] = word;
            if (li == 0) sVs[grp][l] = vs;
          }
        } else if (basis == 1) {  // int8, excess 128
          const float vs = f16_scale(best, 127.0f);
          const float ivs = inv_scale(vs);
          uint32_t w[2] = {0u, 0u};
#pragma unroll
          for (int cc = 0; cc < 8; ++cc)
            w[cc >> 2] |= (uint32_t)(quant(flip * v[cc], ivs, 127) + 128) << (8 * (cc & 3));
          *reinterpret_cast<uint2*>(rec + 128 * l + 8 * li) = make_uint2(w[0], w[1]);
          if (li == 0) *reinterpret_cast<uint16_t*>(rec + rec_scale_off(r, 1) + 2 * l) = f16_bits(vs);
        } else {  // bfloat16, round to nearest even; the column scale is 1
          uint32_t w[4];
#pragma unroll
          for (int e2 = 0; e2 < 4; ++e2)
            w[e2] = bf16_rne_bits(flip * v[2 * e2]) | (bf16_rne_bits(flip * v[2 * e2 + 1]) << 16);
          *reinterpret_cast<uint4*>(rec + 256 * l + 16 * li) = make_uint4(w[0], w[1], w[2], w[3]);
          if (li == 0) *reinterpret_cast<uint16_t*>(rec + rec_scale_off(r, 2) + 2 * l) = f16_bits(1.0f);
        }
      }
    }
  }
  __syncthreads();  // sFlip visible to the whole group
  if (!active) return;
  // C[li][l] = flip_l * U[li][l] * sigma_l (0 for a dropped mode)
  auto coef_value = [&](int l) {
    const float lam = sLam[grp][l];
    const bool kept = lam > floor_ && lam > 0.0f;
    return kept ? sFlip[grp][l] * sU[grp][li][l] * sqrtf(lam) : 0.0f;
  };

  if (kFactors) {
    float* mo = mu_out + out_item * kDim;
    for (int cc = 0; cc < 8; ++cc) mo[8 * li + cc] = sMu[grp][8 * li + cc];
    float* co = coef_out + out_item * (kPage * (long)r);
    for (int l = 0; l < r; ++l) co[li * r + l] = coef_value(l);
    sigma2_out[out_item * kPage + li] = sLam[grp][li];
    return;
  }

  // ---- coefficient row li: int8 with its own scale
  float chat[kScore ? kMaxRank : 1];  // decoded row (scored pages)
  {
    const float cs = f16_scale(cabs, 127.0f);
    const float ics = inv_scale(cs);
    for (int l = 0; l < r; ++l) {
      const int code = quant(coef_value(l), ics, 127);
      rec[rec_coef_off(r, basis) + li * r + l] = (uint8_t)(code + 128);
      if (kScore) {
#pragma unroll
        for (int u = 0; u < kMaxRank; ++u)
          if (u == l) chat[u] = (float)code * cs;
      }
    }
    *reinterpret_cast<uint16_t*>(rec + rec_scale_off(r, basis) + 2 * (r + li)) = f16_bits(cs);
  }
  // ---- centroid: int8 with one scale
  {
    float m = 0.0f;
    for (int cc = 0; cc < 8; ++cc) m = fmaxf(m, fabsf(sMu[grp][8 * li + cc]));
    m = group16_max(m);
    const float ms = f16_scale(m, 127.0f);
    const float ims = inv_scale(ms);
    float mhat[8];
    for (int cc = 0; cc < 8; ++cc) {
      const int code = quant(sMu[grp][8 * li + cc], ims, 127);
      rec[rec_mu_off(r, basis) + 8 * li + cc] = (uint8_t)(code + 128);
      mhat[cc] = (float)code * ms;
    }
    if (li == 0) *reinterpret_cast<uint16_t*>(rec + rec_scale_off(r, basis) + 2 * (r + kPage)) = f16_bits(ms);
    if (kScore) {
      // ---- page score for each query head of the group (Eq. 1 on the decoded
      //      summary): z_i = q^T (mu + sum_l c_il v_l) / sqrt d over the 16 tokens
      //      (token li on this lane), then their log-sum-exp
      const int G = bs.H_q / H_kv;
      const long qrow0 = (long)s * bs.H_q + (long)h * G;
      // this lane's 8 query elements of head g (the next head's are requested
      // before the current one is used)
      auto load_q = [&](int g, float (&qv)[8]) {
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) {
          const long qi = (qrow0 + g) * kDim + 8 * li + cc;
          qv[cc] = bs.q_bf16 ? bf16_bits_to_f32(static_cast<const uint16_t*>(bs.q)[qi])
                             : static_cast<const float*>(bs.q)[qi];
        }
      };
      float qn[8];
      load_q(0, qn);
      for (int g = 0; g < G; ++g) {
        float qv[8];
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) qv[cc] = qn[cc];
        if (g + 1 < G) load_q(g + 1, qn);
        float a = 0.0f;
#pragma unroll
        for (int cc = 0; cc < 8; ++cc) a = fmaf(qv[cc], mhat[cc], a);
        a = group16_sum(a);
        for (int l = 0; l < r; ++l) {
          const uint32_t word = sVw[grp][l][li];
          const float vs = sVs[grp][l];
          float pl = 0.0f;
#pragma unroll
          for (int cc = 0; cc < 8; ++cc)
            pl = fmaf(qv[cc], (float)((int)((word >> (4 * cc)) & 15u) - 8) * vs, pl);
          pl = group16_sum(pl);
          if (li == 0) sP[grp][l] = pl;
        }
        wave_sync();
        float z = a;
        for (int l = 0; l < r; ++l) {
          float cl = 0.0f;
#pragma unroll
          for (int u = 0; u < kMaxRank; ++u)
            if (u == l) cl = chat[u];
          z = fmaf(cl, sP[grp][l], z);
        }
        z *= 0.08838834764831845f;  // 1 / sqrt(128)
        const float mx = group16_max(z);
        const float sm = group16_sum(expf(z - mx));
        const float shat = mx + logf(sm);
        if (li == 0) {
          bs.s_hat[bs.lay.base(s, h) + (long)g * bs.lay.head + (long)j * bs.lay.page] = shat;
          bs.part_x[qrow0 + g] = make_float2(shat * 1.4426950408889634f, 1.0f);
        }
        wave_sync();
      }
    }
  }
  // ---- zero padding up to the record stride
  {
    const int pad0 = rec_payload(r, basis);
    if (pad0 + li < rec_stride(r, basis)) rec[pad0 + li] = 0;
  }
}

}  // namespace

hipError_t launch_build(const locks_cfg_t& c, const void* k_cache, const int32_t* page_table,
                        const int32_t* seq_lens, const int32_t* build_list, int32_t n_items,
                        bool all_pages, void* summaries, float* mu, float* basis, float* coef,
                        float* sigma2, hipStream_t st, BuildMode mode, const BuildStep* step) {
  const long items = all_pages ? (long)c.num_seqs * c.max_pages_per_seq * c.num_kv_heads
                               : (long)n_items * c.num_kv_heads;
  if (items == 0) return hipSuccess;
  const bool factors = mu != nullptr;
  if (mode != kBuildAll && (all_pages || factors || step == nullptr)) return hipErrorInvalidValue;
  const long blocks = (items + kItems - 1) / kItems + (mode == kBuildInner ? 1 : 0);
  if (blocks > 0x7fffffffL) return hipErrorInvalidConfiguration;
  const dim3 grid((unsigned)blocks), block(64);
  const BuildStep bs = step ? *step : BuildStep{};
#define LOCKS_BUILD(KT, F, M)                                                                  \
  hipLaunchKernelGGL((build_kernel<KT, F, M>), grid, block, 0, st, c.num_seqs, c.num_kv_heads,  \
                     c.max_pages_per_seq, c.rank, static_cast<const KT*>(k_cache), page_table,  \
                     seq_lens, build_list, n_items, (int)all_pages, (uint8_t*)summaries, mu,    \
                     basis, coef, sigma2, bs, c.basis)
#define LOCKS_BUILD_T(KT)                                     \
  if (factors) LOCKS_BUILD(KT, true, kBuildAll);              \
  else if (mode == kBuildInner) LOCKS_BUILD(KT, false, kBuildInner); \
  else if (mode == kBuildLast) LOCKS_BUILD(KT, false, kBuildLast);   \
  else LOCKS_BUILD(KT, false, kBuildAll)
  if (c.kv_dtype == LOCKS_BF16) {
    LOCKS_BUILD_T(uint16_t);
  } else {
    LOCKS_BUILD_T(float);
  }
#undef LOCKS_BUILD_T
#undef LOCKS_BUILD
  return hipGetLastError();
}

}  // namespace locks
