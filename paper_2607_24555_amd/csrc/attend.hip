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
#include "locks_internal.h"

namespace locks {
namespace {

constexpr int kAttnBlock = 256;

template <typename T>
__device__ __forceinline__ float ld(const T* p, size_t i) { return load_elem(p, i); }

template <typename QT, typename KT>
__global__ __launch_bounds__(kAttnBlock) void attend_kernel(
    int H_q, int H_kv, int max_pages, int k_list, const QT* __restrict__ q,
    const KT* __restrict__ k_cache, const KT* __restrict__ v_cache,
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
  const int n = (L + kPage - 1) / kPage;
  const float zscale = 1.0f / sqrtf((float)kDim);

  for (int e = tid; e < G * kDim; e += kAttnBlock) {
    sq[e / kDim][e % kDim] = ld(q, ((long)s * H_q + h * G) * kDim + e);
    sO[e / kDim][e % kDim] = 0.0f;
  }
  for (int g = tid; g < G; g += kAttnBlock) { sM[g] = -INFINITY; sL[g] = 0.0f; }
  __syncthreads();

  const int t0 = split * pages_per_split;
  for (int t = t0; t < t0 + pages_per_split; ++t) {
    int id;
    if (page_ids) {
      id = t < k_list ? page_ids[((long)s * H_kv + h) * k_list + t] : -1;
    } else {
      id = t;
    }
    if (id < 0 || id >= n) continue;  // uniform across the block
    const long blk = page_table[(long)s * max_pages + id];
    const int valid = min(kPage, L - id * kPage);
    const long base = ((blk * H_kv + h) * kPage) * kDim;
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

__global__ __launch_bounds__(kDim) void merge_kernel(int H_q, int n_splits,
                                                     const float* __restrict__ partial,
                                                     float* __restrict__ out,
                                                     float* __restrict__ out_lse) {
  const int hq = blockIdx.x, s = blockIdx.y, c = threadIdx.x;
  const long row = (long)s * H_q + hq;
  const float* p = partial + row * n_splits * (kDim + 2);
  float m = -INFINITY;
  for (int t = 0; t < n_splits; ++t) m = fmaxf(m, p[t * (kDim + 2) + kDim]);
  float l = 0.0f, o = 0.0f;
  if (m > -INFINITY) {
    for (int t = 0; t < n_splits; ++t) {
      const float mt = p[t * (kDim + 2) + kDim];
      if (mt == -INFINITY) continue;
      const float w = __expf(mt - m);
      l += p[t * (kDim + 2) + kDim + 1] * w;
      o += p[t * (kDim + 2) + c] * w;
    }
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
                     page_budget(c), static_cast<const QT*>(q), static_cast<const KT*>(k_cache),
                     static_cast<const KT*>(v_cache), page_table, seq_lens, page_ids,
                     pages_per_split, n_splits, partial);
}

}  // namespace

hipError_t launch_attend(const locks_cfg_t& c, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                         const int32_t* page_ids, int pages_per_split, int n_splits,
                         float* partial, float* out, float* out_lse, hipStream_t st) {
  const bool qb = c.q_dtype == LOCKS_BF16, kb = c.kv_dtype == LOCKS_BF16;
  if (qb && kb)
    launch_typed<uint16_t, uint16_t>(c, q, k_cache, v_cache, page_table, seq_lens, page_ids,
                                     pages_per_split, n_splits, partial, st);
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

}  // namespace locks
