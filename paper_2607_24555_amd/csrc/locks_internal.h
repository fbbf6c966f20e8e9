// Internal declarations shared by the HIP translation units of liblocks.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/locks.h"

namespace locks {

constexpr int kPage = 16;    // B
constexpr int kDim = 128;    // d
constexpr int kMaxRank = 15; // r <= B - 1 (rank of centred page deviations)
constexpr int kMaxGroup = 16;   // G = H_q / H_kv

// Byte offsets inside one summary record for rank r, basis precision b (0 int4,
// 1 int8, 2 bf16: 64 << b bytes per basis column; see locks_summary_stride_ex) and
// pages of P tokens (16, 32 or 64; P coefficient rows and P + r + 1 scales).
__host__ __device__ constexpr int rec_col_bytes(int b = 0) { return 64 << b; }
__host__ __device__ constexpr int rec_coef_off(int r, int b = 0) { return rec_col_bytes(b) * r; }
__host__ __device__ constexpr int rec_mu_off(int r, int b = 0, int P = kPage) {
  return rec_col_bytes(b) * r + P * r;
}
__host__ __device__ constexpr int rec_scale_off(int r, int b = 0, int P = kPage) {
  return rec_mu_off(r, b, P) + kDim;
}
__host__ __device__ constexpr int rec_payload(int r, int b = 0, int P = kPage) {
  return rec_scale_off(r, b, P) + 2 * (r + P + 1);
}
__host__ __device__ constexpr int rec_stride(int r, int b = 0, int P = kPage) {
  return (rec_payload(r, b, P) + 15) / 16 * 16;
}

// ---------------------------------------------------------------- device helpers

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b16) {
  return __uint_as_float(b16 << 16);
}

template <typename T>
__device__ __forceinline__ float load_elem(const T* p, size_t i);
template <>
__device__ __forceinline__ float load_elem<float>(const float* p, size_t i) {
  return p[i];
}
template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t* p, size_t i) {
  return bf16_bits_to_f32(p[i]);
}

// Float -> uint32 whose unsigned order matches the float order (NaN excluded).
__device__ __forceinline__ uint32_t f32_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float order_key_f32(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

__device__ __forceinline__ float warp_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float warp_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------- page-score layout

// Page scores hat s: element (seq s, KV head h, group head g, page j) lives at
// s * seq + h * kvh + g * head + j * page.  The API's out_all_lse is head-major
// ([S][H_q][max_pages]); the internal workspace copy is head-minor
// ([S][H_kv][max_pages][G]) so that one page's G scores are contiguous.
struct SHatLayout {
  long seq, kvh, head, page;
  __host__ __device__ long base(int s, int h) const { return s * seq + h * kvh; }
};
inline SHatLayout shat_head_major(const locks_cfg_t& c) {
  const long mp = c.max_pages_per_seq, G = c.num_q_heads / c.num_kv_heads;
  return SHatLayout{c.num_q_heads * mp, G * mp, mp, 1};
}
inline SHatLayout shat_head_minor(const locks_cfg_t& c) {
  const long mp = c.max_pages_per_seq, G = c.num_q_heads / c.num_kv_heads;
  return SHatLayout{c.num_kv_heads * mp * G, mp * G, 1, G};
}

// ---------------------------------------------------------------- workspace plan

struct WsPlan {
  size_t s_hat_off;   // float [S][H_kv][max_pages][G]    page scores (head-minor)
  size_t part_off;    // float2 [S][H_q][scan blocks]     (max, sum exp), log2 domain
  size_t ckey_off;    // uint32 [S][H_kv][rows][width]    per-chunk survivors (keys)
  size_t cidx_off;    // int32  [S][H_kv][rows][width]    per-chunk survivors (pages)
  size_t cblk_off;    // int32  [S][H_kv][rows][width]    per-chunk survivors (physical blocks)
  size_t sat_off;     // uint32 [S][H_kv][rows]           per-chunk truncation key
  size_t keys_off;    // uint32 [S][H_kv][max_pages]      every page's key (exact fallback)
  size_t attn_off;    // float [S][H_q][splits][d + 2]    split-K partials
  size_t slscan_off;  // int32 [S]                        scan lengths (overlapped builds)
  size_t partx_off;   // float2 [S][H_q]                  extra partials (overlapped builds)
  size_t chk_pt_off;  // int32 [S][max_pages]             checked page table (table checks)
  size_t chk_sl_off;  // int32 [S]                        checked sequence lengths
  size_t chk_err_off; // int32 [1 + S]                    error word, then one word per sequence
  size_t total;
  int n_chunks;       // select chunks per sequence (block-level path)
  int n_splits;       // attention splits per (seq, KV head)
};

constexpr int kScanPagesPerBlock = 256;  // 4 waves x 64 pages (generic scan kernels)
constexpr int kSelChunk = 1024;          // pages per selection chunk (block-level path)
constexpr int kFastChunk = 512;          // pages per selection chunk (fast path)
constexpr int kUnionCap = 2048;          // chunk survivors one table merge holds
constexpr int kUnionNK = kUnionCap / 256; // ... per lane of a 4-wave block
constexpr int kSparsePagesPerSplit = 4;   // one page per wave of a 4-wave block
constexpr int kDensePagesPerSplit = 256;

WsPlan plan_workspace(const locks_cfg_t& c);
// Bytes of the summary store (every block's records); below 2^32 for a valid
// configuration, so record offsets fit 32 bits.
inline size_t summary_store_bytes(const locks_cfg_t& c) {
  return (size_t)c.num_blocks * (size_t)c.num_kv_heads *
         (size_t)rec_stride(c.rank, c.basis, c.page_size);
}
int page_budget(const locks_cfg_t& c);  // k = ceil(b / B)
// Attention works on 16-token units: a page of B tokens is B / 16 of them.
inline int sub_page_log2(const locks_cfg_t& c) {
  return c.page_size == 64 ? 2 : (c.page_size == 32 ? 1 : 0);
}
int scan_pages_per_block(const locks_cfg_t& c);  // pages covered by one scan block
inline int scan_blocks(const locks_cfg_t& c) {
  const int ppb = scan_pages_per_block(c);
  return (c.max_pages_per_seq + ppb - 1) / ppb;
}

// ---------------------------------------------------------------- launchers
// Each returns hipError_t of the launch (hipSuccess on success).

// Builds of a decode step whose listed pages include the last complete page of
// their sequence: kBuildInner builds the other listed pages and prepares the scan
// (sl_scan = scan lengths without those last pages); kBuildLast builds the last
// pages and scores them for q (s_hat entries, and part_x [S][H_q] in the log2
// domain, valid for the sequences with sl_scan < seq_lens), so it may run beside
// the scan and needs nothing from kBuildInner.
enum BuildMode { kBuildAll = 0, kBuildInner = 1, kBuildLast = 2 };
struct BuildStep {
  int32_t* sl_scan;
  float2* part_x;
  const void* q;
  int q_bf16;
  int H_q;
  float* s_hat;
  SHatLayout lay;
};
hipError_t launch_build(const locks_cfg_t& c, const void* k_cache, const int32_t* page_table,
                        const int32_t* seq_lens, const int32_t* build_list, int32_t n_items,
                        bool all_pages, void* summaries, float* mu, float* basis, float* coef,
                        float* sigma2, hipStream_t st, BuildMode mode = kBuildAll,
                        const BuildStep* step = nullptr);

// The same build for pages of B = 16, 32 or 64 tokens (tridiagonal eigensolver);
// every listed or complete page, or the unquantised factors when mu != nullptr.
hipError_t launch_build_page(const locks_cfg_t& c, const void* k_cache, const int32_t* page_table,
                             const int32_t* seq_lens, const int32_t* build_list, int32_t n_items,
                             bool all_pages, void* summaries, float* mu, float* basis,
                             float* coef, float* sigma2, hipStream_t st);

hipError_t launch_scan(const locks_cfg_t& c, const void* q, const void* summaries,
                       const int32_t* page_table, const int32_t* seq_lens, float* s_hat,
                       SHatLayout lay, float2* partials, hipStream_t st);

struct SelectBufs {
  uint32_t* cand_key;
  int32_t* cand_idx;
  int32_t* cand_blk;
  uint32_t* sat;
  uint32_t* keys;
  int n_chunks;
};
// Fast selection: k - 2 <= kFastK and at most kUnionCap / 8 chunks of kFastChunk
// pages.  Each chunk keeps its top select_fast_width() keys; the table is the top k - 2
// of their union unless a chunk was truncated at or above the union's cut, in
// which case it is recomputed exactly from every page's key.
bool select_fast_path(const locks_cfg_t& c);
int select_fast_rows(const locks_cfg_t& c);
int select_fast_width(const locks_cfg_t& c);
// Fast path, first half: every page's key and each chunk's top keys (in sb).
// part_x (nullable): one more (max, sum) partial per query head, [S][H_q], valid
// for the sequences with sl_scan[s] < seq_lens[s].
hipError_t launch_select_chunks(const locks_cfg_t& c, const int32_t* page_table,
                                const int32_t* seq_lens, const float* s_hat, SHatLayout lay,
                                const float2* partials, const SelectBufs& sb, hipStream_t st,
                                const float2* part_x = nullptr, const int32_t* sl_scan = nullptr);
hipError_t launch_select(const locks_cfg_t& c, const int32_t* page_table, const int32_t* seq_lens,
                         const float* s_hat, SHatLayout lay, const float2* partials,
                         const SelectBufs& sb, int32_t* out_page_ids, float* out_sel_lse,
                         hipStream_t st);

hipError_t launch_attend(const locks_cfg_t& c, const void* q, const void* k_cache,
                         const void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                         const int32_t* page_ids, int pages_per_split, int n_splits,
                         float* partial, float* out, float* out_lse, hipStream_t st);

// Fused decode-step tail: the selection merge inside the attention kernel
// (bf16 Q and KV, fast selection path), then the split merge.
bool attend_select_fused(const locks_cfg_t& c);
hipError_t launch_attend_select(const locks_cfg_t& c, const void* q, const void* k_cache,
                                const void* v_cache, const int32_t* page_table,
                                const int32_t* seq_lens, const SelectBufs& sb, const float* s_hat,
                                SHatLayout lay, int32_t* out_ids, float* out_sel_lse,
                                int pages_per_split, int n_splits, float* partial, float* out,
                                float* out_lse, hipStream_t st);

// KIVI fake quantisation of the listed (seq, page) pairs' K and V, or of every
// complete page when all_pages (bf16 caches).  `which` narrows the pages to the
// last complete page of each sequence (kKiviLast) or to the others (kKiviInner),
// the split of a decode step's builds.
enum KiviPages { kKiviAny = 0, kKiviLast = 1, kKiviInner = 2 };
bool kivi_valid(const locks_kivi_t& kv);
hipError_t launch_kivi(const locks_cfg_t& c, const locks_kivi_t& kv, void* k_cache,
                       void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                       const int32_t* page_list, int32_t n_items, bool all_pages,
                       hipStream_t st, KiviPages which = kKiviAny);

// The newest token of every sequence (token seq_lens[s] - 1, skipped for an empty
// sequence) copied from k_new / v_new [S][H_kv][128] into the paged caches.
// Table checks: clamped copies of page_table and seq_lens, the per-sequence error
// words and their OR (LOCKS_TABLE_E_* bits).
hipError_t launch_check_tables(const locks_cfg_t& c, const int32_t* page_table,
                               const int32_t* seq_lens, int32_t* pt_out, int32_t* sl_out,
                               int32_t* err_word, int32_t* err_rows, hipStream_t st);
hipError_t launch_append(const locks_cfg_t& c, const void* k_new, const void* v_new,
                         void* k_cache, void* v_cache, const int32_t* page_table,
                         const int32_t* seq_lens, hipStream_t st);

}  // namespace locks
