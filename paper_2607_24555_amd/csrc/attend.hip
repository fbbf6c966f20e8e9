// Paged decode attention over a page list (Sec. 2 "Decode-time attention";
// App. E "sparse decode over k pages"):
//   o_g = sum_{i in S} softmax_S(q_g^T k_i / sqrt d) v_i,
// renormalised over the tokens of the listed pages.  With page_ids == nullptr the
// list is every page of the sequence (the dense baseline).
//
// Split-K: block (split, KV head, seq) walks its slice of the page list with an
// online softmax for all G query heads of the KV head (the G heads share every K/V
// page load), then writes an unnormalised partial (o, max, sum).  merge_kernel
// combines the splits exactly: m = max m_s, l = sum l_s e^{m_s - m},
// o = sum o_s e^{m_s - m} / l, lse = m + log l.
//
// bf16 Q and KV take attend_mfma_kernel: each wave owns pages_per_split / 4
// consecutive list entries and handles one page (16 tokens) per step on the
// matrix cores; the block's four waves combine in LDS before the partial is
// written.  Other dtypes take the VALU kernel attend_kernel.  In the fused
// decode step (kSelect) every block first derives its (sequence, KV head)'s
// page table from the selection chunks' survivors -- all blocks of the unit
// compute the same table -- and writes the table entries it attends together
// with their estimated page LSEs.
#include "locks_internal.h"
#include "topk.h"

namespace locks {
namespace {

constexpr int kAttnBlock = 256;

template <typename T>
__device__ __forceinline__ float ld(const T* p, size_t i) { return load_elem(p, i); }

// Work is counted in 16-token sub-pages: unit t of the list is sub-page t % nsub
// of list entry t / nsub (nsub = B / 16 for pages of B tokens).
template <typename QT, typename KT>
__global__ __launch_bounds__(kAttnBlock) void attend_kernel(
    int H_q, int H_kv, int max_pages, int k_list, int pgsz, int lg_sub,
    const QT* __restrict__ q, const KT* __restrict__ k_cache, const KT* __restrict__ v_cache,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ page_ids, int pages_per_split, int n_splits,
    float* __restrict__ partial) {
  __shared__ float sq[kMaxGroup][kDim];
  __shared__ float sK[kPage][kDim + 1];
  __shared__ float sV[kPage][kDim];
  __shared__ float sP[kMaxGroup][kPage];
  __shared__ float sO[kMaxGroup][kDim];
  __shared__ float sM[kMaxGroup], sL[kMaxGroup], sScale[kMaxGroup];

  const int split = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int tid = threadIdx.x;
  const int G = H_q / H_kv;
  const int L = seq_lens[s];
  const int n = (L + pgsz - 1) / pgsz;
  const float zscale = 1.0f / sqrtf((float)kDim);

  for (int e = tid; e < G * kDim; e += kAttnBlock) {
    sq[e / kDim][e % kDim] = ld(q, ((long)s * H_q + h * G) * kDim + e);
    sO[e / kDim][e % kDim] = 0.0f;
  }
  for (int g = tid; g < G; g += kAttnBlock) { sM[g] = -INFINITY; sL[g] = 0.0f; }
  __syncthreads();

  const int t0 = split * pages_per_split;
  for (int t = t0; t < t0 + pages_per_split; ++t) {
    const int entry = t >> lg_sub, sub = t & ((1 << lg_sub) - 1);
    int id;
    if (page_ids) {
      id = entry < k_list ? page_ids[((long)s * H_kv + h) * k_list + entry] : -1;
    } else {
      id = entry;
    }
    if (id < 0 || id >= n) continue;  // uniform across the block
    const int tok0 = id * pgsz + sub * kPage;
    if (tok0 >= L) continue;
    const long blk = page_table[(long)s * max_pages + id];
    const int valid = min(kPage, L - tok0);
    const long base = ((blk * H_kv + h) * pgsz + sub * kPage) * kDim;
    for (int e = tid; e < kPage * kDim; e += kAttnBlock) {
      sK[e / kDim][e % kDim] = ld(k_cache, base + e);
      sV[e / kDim][e % kDim] = ld(v_cache, base + e);
    }
    __syncthreads();
    for (int e = tid; e < G * kPage; e += kAttnBlock) {
      const int g = e / kPage, i = e % kPage;
      float z = -INFINITY;
      if (i < valid) {
        float acc = 0.0f;
        for (int c = 0; c < kDim; ++c) acc = fmaf(sq[g][c], sK[i][c], acc);
        z = acc * zscale;
      }
      sP[g][i] = z;
    }
    __syncthreads();
    for (int g = tid; g < G; g += kAttnBlock) {
      float mx = sM[g];
      for (int i = 0; i < kPage; ++i) mx = fmaxf(mx, sP[g][i]);
      const float sc = (sM[g] == -INFINITY) ? 0.0f : __expf(sM[g] - mx);
      float l = sL[g] * sc;
      for (int i = 0; i < kPage; ++i) {
        const float w = (sP[g][i] == -INFINITY) ? 0.0f : __expf(sP[g][i] - mx);
        sP[g][i] = w;
        l += w;
      }
      sM[g] = mx;
      sL[g] = l;
      sScale[g] = sc;
    }
    __syncthreads();
    for (int e = tid; e < G * kDim; e += kAttnBlock) {
      const int g = e / kDim, c = e % kDim;
      float acc = sO[g][c] * sScale[g];
      for (int i = 0; i < kPage; ++i) acc = fmaf(sP[g][i], sV[i][c], acc);
      sO[g][c] = acc;
    }
    __syncthreads();
  }
  for (int e = tid; e < G * (kDim + 2); e += kAttnBlock) {
    const int g = e / (kDim + 2), c = e % (kDim + 2);
    const long row = (long)s * H_q + h * G + g;
    float v = c < kDim ? sO[g][c] : (c == kDim ? sM[g] : sL[g]);
    partial[(row * n_splits + split) * (kDim + 2) + c] = v;
  }
}


// ---------------------------------------------------------------- MFMA path
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));
typedef short s4v __attribute__((ext_vector_type(4)));
typedef float f4v __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ bf8v as_bf8(uint4 v) { return __builtin_bit_cast(bf8v, v); }

// Round-to-nearest-even float -> bf16 bits (finite inputs).
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Sum / max over the lanes {l, l^16, l^32, l^48} (the four 16-lane rows).
__device__ __forceinline__ float rows_max(float v) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(p[0]), __uint_as_float(p[1]));
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float rows_sum(float v) {
  auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// 16-bit element e (0..7) of a uint4.
__device__ __forceinline__ uint32_t half_of(const uint4& v, int e) {
  const uint32_t w = e < 2 ? v.x : (e < 4 ? v.y : (e < 6 ? v.z : v.w));
  return (e & 1) ? (w >> 16) : (w & 0xffffu);
}

// One page of K (16 tokens x 128) and V in the operand layouts below.
struct PageRegs {
  uint4 k[4];  // lane (t = l % 16, r = l / 16): K[t][32 r + 8 kb .. + 7], kb = 0..3
  uint4 v[4];  // lane (c = l % 16, r): V[4 r + j][8 c .. 8 c + 7], j = 0..3
};

__device__ __forceinline__ void load_page(PageRegs& P, const uint16_t* kp, const uint16_t* vp,
                                          int c16, int r4) {
  const uint4* k4 = reinterpret_cast<const uint4*>(kp + c16 * kDim + 32 * r4);
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) P.k[kb] = k4[kb];
#pragma unroll
  for (int j = 0; j < 4; ++j) P.v[j] = *reinterpret_cast<const uint4*>(vp + (4 * r4 + j) * kDim + 8 * c16);
}

// Lane layout (l = 16 r + c):
//   S^T = K Q^T  (mfma 16x16x32, M = token, N = head, K = dim with dim order
//                 32 r + 8 kb + e): lane holds S^T[4 r + j][c], j = 0..3, so head
//                 c's 16 logits are the j values of lanes c, c+16, c+32, c+48;
//   O^T += V^T P (mfma 16x16x16, M = dim, N = head, K = token; tile n covers
//                 dims 8 m + n, m = 0..15): P is the B operand exactly as S^T
//                 left it, and lane holds O^T for head c, dims 32 r + 8 j + n.
// P enters as bf16 hi + lo (two MFMAs) so the weights keep ~16 bits.
// Chunk survivors and outputs of the selection merged into the attention kernel.
struct SelTable {
  SelectBufs sb;
  int n_rows, width;
  const float* s_hat;
  SHatLayout lay;
  int32_t* out_ids;
  float* out_sel_lse;
};

// kPPW > 0: every wave owns exactly kPPW list entries and keeps up to four
// pages in flight (fully unrolled, so each wait covers one page); kPPW == 0: any
// count, one page in flight ahead of the one being used.
template <bool kSelect, int kPPW>
__global__ __launch_bounds__(256) void attend_mfma_kernel(
    int H_q, int H_kv, int max_pages, int k_list, int pgsz, int lg_sub,
    const uint16_t* __restrict__ q,
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ page_ids, int pages_per_split, int n_splits,
    float* __restrict__ partial, SelTable tb) {
  __shared__ float sO[4][kDim][kMaxGroup + 1];
  __shared__ float sM[4][kMaxGroup], sL[4][kMaxGroup];
  __shared__ int32_t s_tab[kSelect ? kFastK + 2 : 1], s_blk[kSelect ? kFastK + 2 : 1];
  __shared__ UnionLds<4> unionL;
  const int split = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c16 = lane & 15, r4 = lane >> 4;
  const int G = H_q / H_kv;
  // the selection survivors are requested before the sequence length is known
  UnionRegs<kUnionNK> UR;
  if constexpr (kSelect) {
    const long unit = (long)s * H_kv + h;
    const long rb = unit * tb.n_rows * tb.width;
    union_load<kUnionNK, 4>(UR, tb.n_rows, tb.width, tb.sb.cand_key + rb, tb.sb.cand_idx + rb,
                            tb.sb.cand_blk + rb, tb.sb.sat + unit * tb.n_rows);
  }
  const int L = seq_lens[s];
  const int n = (L + pgsz - 1) / pgsz;
  const float zs = kLog2e / sqrtf((float)kDim);
  const int sub_mask = (1 << lg_sub) - 1;

  uint4 qb[4];
  {
    const int g = c16 < G ? c16 : 0;
    const uint4* q4 = reinterpret_cast<const uint4*>(q + ((long)s * H_q + h * G + g) * kDim + 32 * r4);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qb[kb] = c16 < G ? q4[kb] : make_uint4(0, 0, 0, 0);
  }
  const int ppw = pages_per_split / 4;
  const int t_begin = split * pages_per_split + wave * ppw, t_end = t_begin + ppw;
  const int32_t* ids = page_ids ? page_ids + ((long)s * H_kv + h) * k_list : nullptr;
  if constexpr (kSelect) {
    const long unit = (long)s * H_kv + h;
    const int used = n > k_list ? (n - 2) / kFastChunk + 1 : 0;
    union_table_from<kUnionNK, 4>(UR, k_list, n, used, tb.width, tb.sb.keys + unit * max_pages,
                                  page_table + (long)s * max_pages, s_tab, s_blk, unionL);
    ids = s_tab;
  }
  // this block's table entries and their estimated page LSEs (NaN without a
  // summary): loaded now, written after the pages (at most 32 entries per block,
  // so at most 32 x 17 values over the 256 threads)
  constexpr int kSelPer = 3;
  const int epb = pages_per_split >> lg_sub;  // table entries per block
  float sel_v[kSelPer];
  int sel_e[kSelPer];
  if constexpr (kSelect) {
    const int t0 = split * epb, n_c = L / pgsz;
    const float* sb = tb.s_hat + tb.lay.base(s, h);
#pragma unroll
    for (int u = 0; u < kSelPer; ++u) {
      const int e = tid + 256 * u;
      const int t = t0 + e % epb, g = e / epb;
      sel_e[u] = (e < epb * (G + 1) && t < k_list) ? e : -1;
      sel_v[u] = 0.0f;
      if (sel_e[u] >= 0 && g < G) {
        const int id = s_tab[t];
        const bool ok = id >= 0 && id < n_c;
        const float v = sb[(long)(ok ? id : 0) * tb.lay.page + (long)(ok ? g : 0) * tb.lay.head];
        sel_v[u] = ok ? v : __int_as_float(0x7fc00000);
      }
    }
  }
  // unit t: sub-page t & sub_mask of list entry t >> lg_sub; returns the unit's
  // first token (-1: nothing to attend)
  auto page_at = [&](int t) -> int {
    int id = -1;
    const int entry = t >> lg_sub;
    if (t < t_end) id = ids ? (entry < k_list ? ids[entry] : -1) : entry;
    const int tok0 = (id >= 0 && id < n) ? id * pgsz + (t & sub_mask) * kPage : -1;
    return tok0 < L ? tok0 : -1;
  };
  const long kv_head = (long)h * pgsz * kDim;
  const long kv_blk = (long)H_kv * pgsz * kDim;
  // physical block of unit t starting at token tok0 (a valid block stands in for an
  // empty unit); the fused step knows the blocks from the selection
  auto blk_at = [&](int t, int tok0) -> long {
    if constexpr (kSelect) {
      const int entry = t >> lg_sub;
      const int b = entry < k_list ? s_blk[entry] : -1;
      return b >= 0 ? b : s_blk[0];
    } else {
      return page_table[(long)s * max_pages + (tok0 >= 0 ? tok0 / pgsz : 0)];
    }
  };
  auto page_ptr = [&](long blk, int t, const uint16_t* base) {
    return base + blk * kv_blk + kv_head + (long)(t & sub_mask) * kPage * kDim;
  };

  float m = -INFINITY, l = 0.0f;
  f4v o[8];
#pragma unroll
  for (int t = 0; t < 8; ++t) o[t] = f4v{0.0f, 0.0f, 0.0f, 0.0f};

  // one 16-token unit of the list (tok0 < 0: an empty unit, nothing to add)
  auto use_page = [&](const PageRegs& cur, int tok0) {
    if (tok0 >= 0) {
      const int valid = min(kPage, L - tok0);
      f4v st = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf8(cur.k[kb]), as_bf8(qb[kb]), st, 0, 0, 0);
      float z[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) z[j] = (4 * r4 + j < valid) ? st[j] * zs : -INFINITY;
      const float pm = rows_max(fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3])));
      const float mn = fmaxf(m, pm);
      const float sc = (m == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m - mn);
      float p[4], ps = 0.0f;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        p[j] = (z[j] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(z[j] - mn);
        ps += p[j];
      }
      l = l * sc + rows_sum(ps);
      m = mn;
      uint32_t hi[4], lo[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        hi[j] = bf16_rne(p[j]);
        lo[j] = bf16_rne(p[j] - __uint_as_float(hi[j] << 16));
      }
      const s4v bh = __builtin_bit_cast(s4v, make_uint2(hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16)));
      const s4v bl = __builtin_bit_cast(s4v, make_uint2(lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16)));
#pragma unroll
      for (int t8 = 0; t8 < 8; ++t8) {
        o[t8] *= sc;
        const uint32_t a01 = half_of(cur.v[0], t8) | (half_of(cur.v[1], t8) << 16);
        const uint32_t a23 = half_of(cur.v[2], t8) | (half_of(cur.v[3], t8) << 16);
        const s4v a = __builtin_bit_cast(s4v, make_uint2(a01, a23));
        o[t8] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, bh, o[t8], 0, 0, 0);
        o[t8] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, bl, o[t8], 0, 0, 0);
      }
    }
  };
  // loads unit t into P (a valid page stands in for an empty unit)
  auto load_entry = [&](PageRegs& P, int t) {
    const int tok0 = page_at(t);
    const long b = blk_at(t, tok0);
    load_page(P, page_ptr(b, t, k_cache), page_ptr(b, t, v_cache), c16, r4);
    return tok0;
  };

  if (n > 0) {
    if constexpr (kPPW > 0) {
      constexpr int D = kPPW < 4 ? kPPW : 4;
      PageRegs buf[D];
      int ids[D];
#pragma unroll
      for (int j = 0; j < D; ++j) ids[j] = load_entry(buf[j], t_begin + j);
#pragma unroll
      for (int i = 0; i < kPPW; ++i) {
        use_page(buf[i % D], ids[i % D]);
        if (i + D < kPPW) ids[i % D] = load_entry(buf[i % D], t_begin + i + D);
      }
    } else {
      int id = page_at(t_begin);
      PageRegs cur;
      {
        const long b = blk_at(t_begin, id);
        load_page(cur, page_ptr(b, t_begin, k_cache), page_ptr(b, t_begin, v_cache), c16, r4);
      }
      for (int t = t_begin; t < t_end; ++t) {
        // prefetch the next unit (a valid page stands in for an empty one)
        const int id_next = page_at(t + 1);
        PageRegs nxt;
        if (t + 1 < t_end) {
          const long b = blk_at(t + 1, id_next);
          load_page(nxt, page_ptr(b, t + 1, k_cache), page_ptr(b, t + 1, v_cache), c16, r4);
        }
        use_page(cur, id);
        id = id_next;
        cur = nxt;
      }
    }
  }
  if constexpr (kSelect) {
    const long unit = (long)s * H_kv + h;
    const int t0 = split * epb;
#pragma unroll
    for (int u = 0; u < kSelPer; ++u) {
      const int e = sel_e[u];
      if (e < 0) continue;
      const int t = t0 + e % epb, g = e / epb;
      if (g == G) tb.out_ids[unit * k_list + t] = s_tab[t];
      else tb.out_sel_lse[((long)s * H_q + h * G + g) * k_list + t] = sel_v[u];
    }
  }
  // combine the block's four waves; m is kept in log2 units until here.  sO is
  // [wave][d][17]: the odd row pitch keeps both the MFMA-layout writes and the
  // d-contiguous reads free of bank conflicts
  if (r4 == 0) { sM[wave][c16] = m; sL[wave][c16] = l; }
#pragma unroll
  for (int t8 = 0; t8 < 8; ++t8)
#pragma unroll
    for (int j = 0; j < 4; ++j) sO[wave][32 * r4 + 8 * j + t8][c16] = o[t8][j];
  __syncthreads();
  for (int e = tid; e < G * (kDim + 2); e += 256) {
    const int g = e / (kDim + 2), c = e % (kDim + 2);
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) mx = fmaxf(mx, sM[w][g]);
    float acc = 0.0f, ls = 0.0f;
    if (mx > -INFINITY) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float wt = sM[w][g] == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f(sM[w][g] - mx);
        ls += sL[w][g] * wt;
        if (c < kDim) acc += sO[w][c][g] * wt;
      }
    }
    const float v = c < kDim ? acc : (c == kDim ? (mx == -INFINITY ? mx : mx * kLn2) : ls);
    const long row = (long)s * H_q + h * G + g;
    partial[(row * n_splits + split) * (kDim + 2) + c] = v;
  }
}

__global__ __launch_bounds__(kDim) void merge_kernel(int H_q, int n_splits,
                                                     const float* __restrict__ partial,
                                                     float* __restrict__ out,
                                                     float* __restrict__ out_lse) {
  const int hq = blockIdx.x, s = blockIdx.y, c = threadIdx.x;
  const long row = (long)s * H_q + hq;
  const float* p = partial + row * n_splits * (kDim + 2);
  constexpr int kB = 32;  // splits per round trip (every split of a sparse step)
  float m = -INFINITY, l = 0.0f, o = 0.0f;
  for (int t0 = 0; t0 < n_splits; t0 += kB) {
    float mt[kB], lt[kB], ot[kB];
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      const float* pt = p + (long)min(t0 + u, n_splits - 1) * (kDim + 2);
      mt[u] = pt[kDim];
      lt[u] = pt[kDim + 1];
      ot[u] = pt[c];
    }
#pragma unroll
    for (int u = 0; u < kB; ++u) asm volatile("" : "+v"(mt[u]), "+v"(lt[u]), "+v"(ot[u]));
#pragma unroll
    for (int u = 0; u < kB; ++u) mt[u] = t0 + u < n_splits ? mt[u] : -INFINITY;
    float mm = m;
#pragma unroll
    for (int u = 0; u < kB; ++u) mm = fmaxf(mm, mt[u]);
    if (mm == -INFINITY) continue;
    const float sc = (m == -INFINITY) ? 0.0f : __expf(m - mm);
    l *= sc;
    o *= sc;
#pragma unroll
    for (int u = 0; u < kB; ++u) {
      const float w = (mt[u] == -INFINITY) ? 0.0f : __expf(mt[u] - mm);
      l += lt[u] * w;
      o += ot[u] * w;
    }
    m = mm;
  }
  out[row * kDim + c] = (l > 0.0f) ? o / l : 0.0f;
  if (out_lse && c == 0) out_lse[row] = (l > 0.0f) ? m + logf(l) : -INFINITY;
}

template <typename QT, typename KT>
void launch_typed(const locks_cfg_t& c, const void* q, const void* k_cache, const void* v_cache,
                  const int32_t* page_table, const int32_t* seq_lens, const int32_t* page_ids,
                  int pages_per_split, int n_splits, float* partial, hipStream_t st) {
  hipLaunchKernelGGL((attend_kernel<QT, KT>), dim3(n_splits, c.num_kv_heads, c.num_seqs),
                     dim3(kAttnBlock), 0, st, c.num_q_heads, c.num_kv_heads, c.max_pages_per_seq,
                     page_budget(c), c.page_size, sub_page_log2(c), static_cast<const QT*>(q),
                     static_cast<const KT*>(k_cache),
                     static_cast<const KT*>(v_cache), page_table, seq_lens, page_ids,
                     pages_per_split, n_splits, partial);
}

// bf16 MFMA kernel with the page count per wave fixed at compile time where the
// list is split into 1, 2, 4 or 8 entries per wave.
template <bool kSelect>
void launch_mfma(const locks_cfg_t& c, dim3 grid, hipStream_t st, const uint16_t* q,
                 const uint16_t* k_cache, const uint16_t* v_cache, const int32_t* page_table,
                 const int32_t* seq_lens, const int32_t* page_ids, int pages_per_split,
                 int n_splits, float* partial, SelTable tb) {
  const int ppw = pages_per_split % 4 == 0 ? pages_per_split / 4 : 0;
#define LOCKS_ATTEND_MFMA(P)                                                                   \
  hipLaunchKernelGGL((attend_mfma_kernel<kSelect, P>), grid, dim3(256), 0, st, c.num_q_heads,   \
                     c.num_kv_heads, c.max_pages_per_seq, page_budget(c), c.page_size,          \
                     sub_page_log2(c), q, k_cache, v_cache, page_table, seq_lens, page_ids,     \
                     pages_per_split, n_splits, partial, tb)
  switch (ppw) {
    case 1: LOCKS_ATTEND_MFMA(1); break;
    case 2: LOCKS_ATTEND_MFMA(2); break;
    case 4: LOCKS_ATTEND_MFMA(4); break;
    case 8: LOCKS_ATTEND_MFMA(8); break;
    default: LOCKS_ATTEND_MFMA(0); break;
  }
#undef LOCKS_ATTEND_MFMA
}

}  // namespace

hipError_t launch_attend(const locks_cfg_t& c, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                         const int32_t* page_ids, int pages_per_split, int n_splits,
                         float* partial, float* out, float* out_lse, hipStream_t st) {
  const bool qb = c.q_dtype == LOCKS_BF16, kb = c.kv_dtype == LOCKS_BF16;
  if (qb && kb)
    launch_mfma<false>(c, dim3(n_splits, c.num_kv_heads, c.num_seqs), st,
                       static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_cache),
                       static_cast<const uint16_t*>(v_cache), page_table, seq_lens, page_ids,
                       pages_per_split, n_splits, partial, SelTable{});
  else if (qb)
    launch_typed<uint16_t, float>(c, q, k_cache, v_cache, page_table, seq_lens, page_ids,
                                  pages_per_split, n_splits, partial, st);
  else if (kb)
    launch_typed<float, uint16_t>(c, q, k_cache, v_cache, page_table, seq_lens, page_ids,
                                  pages_per_split, n_splits, partial, st);
  else
    launch_typed<float, float>(c, q, k_cache, v_cache, page_table, seq_lens, page_ids,
                               pages_per_split, n_splits, partial, st);
  hipLaunchKernelGGL(merge_kernel, dim3(c.num_q_heads, c.num_seqs), dim3(kDim), 0, st,
                     c.num_q_heads, n_splits, partial, out, out_lse);
  return hipGetLastError();
}

bool attend_select_fused(const locks_cfg_t& c) {
  return c.q_dtype == LOCKS_BF16 && c.kv_dtype == LOCKS_BF16 && select_fast_path(c);
}

hipError_t launch_attend_select(const locks_cfg_t& c, const void* q, const void* k_cache,
                                const void* v_cache, const int32_t* page_table,
                                const int32_t* seq_lens, const SelectBufs& sb, const float* s_hat,
                                SHatLayout lay, int32_t* out_ids, float* out_sel_lse,
                                int pages_per_split, int n_splits, float* partial, float* out,
                                float* out_lse, hipStream_t st) {
  const SelTable tb{sb, select_fast_rows(c), select_fast_width(c), s_hat, lay, out_ids, out_sel_lse};
  launch_mfma<true>(c, dim3(n_splits, c.num_kv_heads, c.num_seqs), st,
                    static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k_cache),
                    static_cast<const uint16_t*>(v_cache), page_table, seq_lens, nullptr,
                    pages_per_split, n_splits, partial, tb);
  hipLaunchKernelGGL(merge_kernel, dim3(c.num_q_heads, c.num_seqs), dim3(kDim), 0, st,
                     c.num_q_heads, n_splits, partial, out, out_lse);
  return hipGetLastError();
}

}  // namespace locks
