// KIVI fake quantisation of finalised pages, in place (Sec. 5 "KV-cache
// quantization under extreme sparsity"; App. C, protocol of the full KIVI grid):
// asymmetric min/max quantisation with 2^b levels followed by dequantisation back
// to bfloat16.  Keys are quantised per channel over the page's 16 tokens, values
// per token over groups of g consecutive channels.
//
// Every arithmetic step is one IEEE float32 rounding, in this order:
//   s = (max - min) / (2^b - 1),  code = min(rint((x - min) / s), 2^b - 1),
//   y = bf16(code * s + min)     (round to nearest even at both ends),
// and a slice with s = 0 keeps its values.  Contraction into fused multiply-adds
// is switched off for this file so that the product and the sum round separately.
#include "locks_internal.h"

#pragma clang fp contract(off)

namespace locks {
namespace {

constexpr int kKiviWaves = 4;  // one (page, KV head) per wave

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// float32 -> bfloat16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ float fake_quant(float x, float mn, float s, float levels) {
  const float code = fminf(rintf((x - mn) / s), levels);
  return code * s + mn;
}

// Lane layout of one 16 x 128 page: lane = 16 * tg + cg holds channels
// [8 cg, 8 cg + 8) of tokens 4 t + tg (t = 0..3), one 16-byte load per token, so
// each load instruction of the wave covers four whole token rows (1 KiB).  A
// channel's 16 tokens sit in lanes cg, cg + 16, cg + 32, cg + 48; a value group of
// g channels of one token in g / 8 neighbouring lanes (GL of them).
template <int GL>
__global__ __launch_bounds__(64 * kKiviWaves) void kivi_kernel(
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ page_table, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ page_list, long n_units, int all_pages, int num_seqs,
    int num_kv_heads, int max_pages, float levels, int which) {
  const long unit = (long)blockIdx.x * kKiviWaves + (threadIdx.x >> 6);
  if (unit >= n_units) return;
  const int lane = threadIdx.x & 63;
  const int h = (int)(unit % num_kv_heads);
  const long item = unit / num_kv_heads;
  int s, j;
  if (all_pages) {
    s = (int)(item / max_pages);
    j = (int)(item % max_pages);
  } else {
    s = page_list[2 * item];
    j = page_list[2 * item + 1];
    if (s < 0 || s >= num_seqs || j >= max_pages) return;
  }
  const int n_complete = seq_lens[s] / kPage;
  if (j < 0 || j >= n_complete) return;  // only complete pages are finalised
  if (which != kKiviAny && (j == n_complete - 1) != (which == kKiviLast)) return;
  const long blk = page_table[(long)s * max_pages + j];
  const size_t base = ((size_t)blk * num_kv_heads + h) * (kPage * kDim);
  const int cg = lane & 15, tg = lane >> 4;

  uint4 kr[4], vr[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const size_t off = base + (size_t)(4 * t + tg) * kDim + 8 * cg;
    kr[t] = *reinterpret_cast<const uint4*>(k_cache + off);
    vr[t] = *reinterpret_cast<const uint4*>(v_cache + off);
  }

  // ---- keys: one (min, max) per channel over the 16 tokens
  float x[4][8];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint32_t w[4] = {kr[t].x, kr[t].y, kr[t].z, kr[t].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      x[t][2 * e] = bf16_lo(w[e]);
      x[t][2 * e + 1] = bf16_hi(w[e]);
    }
  }
  float mn[8], mx[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    mn[c] = fminf(fminf(x[0][c], x[1][c]), fminf(x[2][c], x[3][c]));
    mx[c] = fmaxf(fmaxf(x[0][c], x[1][c]), fmaxf(x[2][c], x[3][c]));
    mn[c] = fminf(mn[c], __shfl_xor(mn[c], 16, 64));
    mx[c] = fmaxf(mx[c], __shfl_xor(mx[c], 16, 64));
    mn[c] = fminf(mn[c], __shfl_xor(mn[c], 32, 64));
    mx[c] = fmaxf(mx[c], __shfl_xor(mx[c], 32, 64));
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const float sc = (mx[c] - mn[c]) / levels;
    if (sc > 0.f) {
#pragma unroll
      for (int t = 0; t < 4; ++t) x[t][c] = fake_quant(x[t][c], mn[c], sc, levels);
    }
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = f32_to_bf16_rne(x[t][2 * e]) | (f32_to_bf16_rne(x[t][2 * e + 1]) << 16);
    kr[t] = make_uint4(w[0], w[1], w[2], w[3]);
  }

  // ---- values: one (min, max) per token and group of 8 * GL channels
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const uint32_t w[4] = {vr[t].x, vr[t].y, vr[t].z, vr[t].w};
    float y[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      y[2 * e] = bf16_lo(w[e]);
      y[2 * e + 1] = bf16_hi(w[e]);
    }
    float lo = y[0], hi = y[0];
#pragma unroll
    for (int c = 1; c < 8; ++c) {
      lo = fminf(lo, y[c]);
      hi = fmaxf(hi, y[c]);
    }
#pragma unroll
    for (int o = 1; o < GL; o <<= 1) {
      lo = fminf(lo, __shfl_xor(lo, o, 64));
      hi = fmaxf(hi, __shfl_xor(hi, o, 64));
    }
    const float sc = (hi - lo) / levels;
    if (sc > 0.f) {
#pragma unroll
      for (int c = 0; c < 8; ++c) y[c] = fake_quant(y[c], lo, sc, levels);
    }
    uint32_t o4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o4[e] = f32_to_bf16_rne(y[2 * e]) | (f32_to_bf16_rne(y[2 * e + 1]) << 16);
    vr[t] = make_uint4(o4[0], o4[1], o4[2], o4[3]);
  }

#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const size_t off = base + (size_t)(4 * t + tg) * kDim + 8 * cg;
    *reinterpret_cast<uint4*>(k_cache + off) = kr[t];
    *reinterpret_cast<uint4*>(v_cache + off) = vr[t];
  }
}

}  // namespace

bool kivi_valid(const locks_kivi_t& kv) {
  if (kv.bits < 1 || kv.bits > 8) return false;
  if (kv.stage != LOCKS_KIVI_POST && kv.stage != LOCKS_KIVI_PRE) return false;
  return kv.v_group == 8 || kv.v_group == 16 || kv.v_group == 32 || kv.v_group == 64 ||
         kv.v_group == 128;
}

hipError_t launch_kivi(const locks_cfg_t& c, const locks_kivi_t& kv, void* k_cache,
                       void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                       const int32_t* page_list, int32_t n_items, bool all_pages,
                       hipStream_t st, KiviPages which) {
  const long items = all_pages ? (long)c.num_seqs * c.max_pages_per_seq : (long)n_items;
  const long units = items * c.num_kv_heads;
  if (units <= 0) return hipSuccess;
  const dim3 grid((unsigned)((units + kKiviWaves - 1) / kKiviWaves)), block(64 * kKiviWaves);
  const float levels = (float)((1 << kv.bits) - 1);
  auto* kc = static_cast<uint16_t*>(k_cache);
  auto* vc = static_cast<uint16_t*>(v_cache);
  const int all = all_pages ? 1 : 0;
#define LOCKS_KIVI_LAUNCH(GL)                                                              \
  hipLaunchKernelGGL(kivi_kernel<GL>, grid, block, 0, st, kc, vc, page_table, seq_lens,    \
                     page_list, units, all, c.num_seqs, c.num_kv_heads, c.max_pages_per_seq, \
                     levels, (int)which)
  switch (kv.v_group) {
    case 8: LOCKS_KIVI_LAUNCH(1); break;
    case 16: LOCKS_KIVI_LAUNCH(2); break;
    case 32: LOCKS_KIVI_LAUNCH(4); break;
    case 64: LOCKS_KIVI_LAUNCH(8); break;
    default: LOCKS_KIVI_LAUNCH(16); break;
  }
#undef LOCKS_KIVI_LAUNCH
  return hipGetLastError();
}

}  // namespace locks
