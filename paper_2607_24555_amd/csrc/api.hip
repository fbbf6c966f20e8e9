// Host side of the C ABI declared in include/locks.h: argument validation,
// workspace planning and stream-ordered launches.  No allocation, no
// synchronisation, no exceptions.
#include <atomic>
#include <mutex>

#include "locks_internal.h"

namespace locks {

namespace {
thread_local int g_last_hip_error = 0;

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int validate(const locks_cfg_t* c) {
  if (!c) return LOCKS_E_INVAL;
  if (c->head_dim != kDim) return LOCKS_E_UNSUPPORTED;
  if (c->page_size != 16 && c->page_size != 32 && c->page_size != 64) return LOCKS_E_UNSUPPORTED;
  if ((c->kv_dtype != LOCKS_BF16 && c->kv_dtype != LOCKS_FP32) ||
      (c->q_dtype != LOCKS_BF16 && c->q_dtype != LOCKS_FP32))
    return LOCKS_E_UNSUPPORTED;
  if (c->num_seqs < 0 || c->num_kv_heads < 1 || c->num_q_heads < 1) return LOCKS_E_INVAL;
  if (c->num_q_heads % c->num_kv_heads) return LOCKS_E_INVAL;
  if (c->num_q_heads / c->num_kv_heads > kMaxGroup) return LOCKS_E_UNSUPPORTED;
  if (c->rank < 1 || c->rank > kMaxRank) return LOCKS_E_INVAL;
  if (c->basis < LOCKS_BASIS_INT4 || c->basis > LOCKS_BASIS_BF16) return LOCKS_E_INVAL;
  if (c->basis != LOCKS_BASIS_INT4 && c->rank != 2 && c->rank != 4 && c->rank != 8)
    return LOCKS_E_UNSUPPORTED;
  if (c->basis != LOCKS_BASIS_INT4 && c->page_size != kPage) return LOCKS_E_UNSUPPORTED;
  if (c->budget_tokens < 1 || (c->budget_tokens + c->page_size - 1) / c->page_size < 2)
    return LOCKS_E_INVAL;
  if (c->max_pages_per_seq < 1 || c->num_blocks < 1) return LOCKS_E_INVAL;
  if ((long)c->num_seqs * c->num_q_heads > 0x7fffffffL / kDim) return LOCKS_E_INVAL;
  // record offsets are 32-bit: the summary store must stay below 4 GiB
  if (summary_store_bytes(*c) > 0xffffffffull) return LOCKS_E_UNSUPPORTED;
  return LOCKS_OK;
}

int hip_status(hipError_t e) {
  if (e == hipSuccess) return LOCKS_OK;
  g_last_hip_error = (int)e;
  return LOCKS_E_HIP;
}

struct Ws {
  float* s_hat;
  float2* part;
  SelectBufs sel;
  float* attn;
  int32_t* sl_scan;
  float2* part_x;
};

Ws carve(void* ws, const WsPlan& p) {
  char* b = static_cast<char*>(ws);
  const SelectBufs sel{reinterpret_cast<uint32_t*>(b + p.ckey_off),
                       reinterpret_cast<int32_t*>(b + p.cidx_off),
                       reinterpret_cast<int32_t*>(b + p.cblk_off),
                       reinterpret_cast<uint32_t*>(b + p.sat_off),
                       reinterpret_cast<uint32_t*>(b + p.keys_off), p.n_chunks};
  return Ws{reinterpret_cast<float*>(b + p.s_hat_off), reinterpret_cast<float2*>(b + p.part_off),
            sel, reinterpret_cast<float*>(b + p.attn_off), reinterpret_cast<int32_t*>(b + p.slscan_off),
            reinterpret_cast<float2*>(b + p.partx_off)};
}

// The side stream of a decode step's overlapped build (one per device, with its
// fork and join events), created on first use and kept until the process ends.
struct SideStream {
  hipStream_t st = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
constexpr int kMaxDevices = 64;
std::mutex g_side_mu;  // also serialises the fork / join enqueues of one step
SideStream g_side[kMaxDevices];

// The current device's side stream, created here unless `create` is false (then
// *out is null when it does not exist yet).  Callers hold g_side_mu.
hipError_t side_stream(SideStream** out, bool create = true) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  SideStream& ss = g_side[dev];
  if (!ss.st || !ss.fork || !ss.join) {
    if (!create) return hipSuccess;
    if (!ss.st && (e = hipStreamCreateWithFlags(&ss.st, hipStreamNonBlocking)) != hipSuccess) return e;
    if (!ss.fork && (e = hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming)) != hipSuccess)
      return e;
    if (!ss.join && (e = hipEventCreateWithFlags(&ss.join, hipEventDisableTiming)) != hipSuccess)
      return e;
  }
  *out = &ss;
  return hipSuccess;
}

// Workspace of locks_decode_step_static: one array per device (each GPU the library
// runs on holds it until the process ends).  Host code never uses the array's name
// as an address: the device address comes from hipGetSymbolAddress, once per
// device with that device current, and is kept in g_scratch.
constexpr size_t kStaticScratchBytes = LOCKS_STATIC_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kStaticScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices];

// The current device's address of `scratch`, resolved on first use.
hipError_t scratch_ptr(void** out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

// Table checks (locks_set_table_checks), process-wide.
std::atomic<int> g_table_checks{0};

// With table checks on: validates page_table / seq_lens into the workspace's
// checked copies (clamping what is out of range, setting the error word) on `st`
// and points the two at the copies, which every later launch of the call reads.
int checked_tables(const locks_cfg_t& c, void* ws, const int32_t*& page_table,
                   const int32_t*& seq_lens, hipStream_t st) {
  if (!g_table_checks.load(std::memory_order_relaxed)) return LOCKS_OK;
  const WsPlan p = plan_workspace(c);
  char* b = static_cast<char*>(ws);
  int32_t* pt = reinterpret_cast<int32_t*>(b + p.chk_pt_off);
  int32_t* sl = reinterpret_cast<int32_t*>(b + p.chk_sl_off);
  int32_t* err = reinterpret_cast<int32_t*>(b + p.chk_err_off);
  const int rc = hip_status(launch_check_tables(c, page_table, seq_lens, pt, sl, err, err + 1, st));
  if (rc) return rc;
  page_table = pt;
  seq_lens = sl;
  return LOCKS_OK;
}

int check_ws(const locks_cfg_t* c, void* ws, size_t ws_bytes) {
  const WsPlan p = plan_workspace(*c);
  if (!ws || ws_bytes < p.total) return LOCKS_E_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(ws) & 255) return LOCKS_E_WORKSPACE;
  return LOCKS_OK;
}

// Table entries per attention block: 4 (one page per wave), doubled while the
// grid would exceed ~512 blocks, so large batches stream several pages per
// wave instead of paying per-block latency many times over.
// (Counted in 16-token units: a table entry of B tokens is B / 16 of them.)
int sparse_pages_per_split(const locks_cfg_t& c) {
  const long units = (long)c.num_seqs * c.num_kv_heads;
  const int k = page_budget(c) << sub_page_log2(c);
  int pps = kSparsePagesPerSplit;
  while (pps < 32 && units * ((k + pps - 1) / pps) > 512) pps *= 2;
  return pps;
}

int sparse_splits(const locks_cfg_t& c) {
  const int pps = sparse_pages_per_split(c);
  return ((page_budget(c) << sub_page_log2(c)) + pps - 1) / pps;
}

// Dense baseline: pages per split block, 256 (64 per wave), halved while the grid
// would hold fewer than 512 blocks -- two per compute unit -- so that short
// contexts and small batches still fill the chip.
int dense_pages_per_split(const locks_cfg_t& c) {
  const long units = (long)c.num_seqs * c.num_kv_heads;
  const long span = (long)c.max_pages_per_seq << sub_page_log2(c);
  int pps = kDensePagesPerSplit;
  while (pps > 4 && units * ((span + pps - 1) / pps) < 512) pps /= 2;
  return pps;
}

int dense_splits(const locks_cfg_t& c) {
  const int pps = dense_pages_per_split(c);
  return (int)((((long)c.max_pages_per_seq << sub_page_log2(c)) + pps - 1) / pps);
}

// The build for the configuration's page size: the register-resident kernel of
// build.hip for 16-token pages (which also serves a step's overlapped build), the
// LDS-resident one of build_page.hip for 32 and 64.
hipError_t build_pages(const locks_cfg_t& c, const void* k_cache, const int32_t* page_table,
                       const int32_t* seq_lens, const int32_t* build_list, int32_t n_items,
                       bool all_pages, void* summaries, float* mu, float* basis, float* coef,
                       float* sigma2, hipStream_t st) {
  if (c.page_size != kPage)
    return launch_build_page(c, k_cache, page_table, seq_lens, build_list, n_items, all_pages,
                             summaries, mu, basis, coef, sigma2, st);
  return launch_build(c, k_cache, page_table, seq_lens, build_list, n_items, all_pages, summaries,
                      mu, basis, coef, sigma2, st);
}

}  // namespace

int page_budget(const locks_cfg_t& c) { return (c.budget_tokens + c.page_size - 1) / c.page_size; }

WsPlan plan_workspace(const locks_cfg_t& c) {
  WsPlan p{};
  const size_t S = (size_t)c.num_seqs, Hq = (size_t)c.num_q_heads, Hkv = (size_t)c.num_kv_heads;
  const size_t mp = (size_t)c.max_pages_per_seq;
  const int k = page_budget(c);
  const size_t K = k > 2 ? (size_t)(k - 2) : 1;
  p.n_chunks = (int)((mp + kSelChunk - 1) / kSelChunk);
  const int sp = ((k << sub_page_log2(c)) + kSparsePagesPerSplit - 1) / kSparsePagesPerSplit;
  p.n_splits = sp > dense_splits(c) ? sp : dense_splits(c);
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t o = off; off = align256(off + bytes); return o; };
  p.s_hat_off = take(S * Hq * mp * sizeof(float));
  p.part_off = take(S * Hq * (size_t)scan_blocks(c) * sizeof(float2));
  // survivor rows: the block-level path keeps k - 2 per chunk, the fast path `width`
  const size_t rows = (size_t)select_fast_rows(c);
  size_t surv = (size_t)p.n_chunks * K;
  if (rows * (size_t)select_fast_width(c) > surv) surv = rows * (size_t)select_fast_width(c);
  p.ckey_off = take(S * Hkv * surv * sizeof(uint32_t));
  p.cidx_off = take(S * Hkv * surv * sizeof(int32_t));
  p.cblk_off = take(S * Hkv * surv * sizeof(int32_t));
  p.sat_off = take(S * Hkv * rows * sizeof(uint32_t));
  p.keys_off = take(S * Hkv * mp * sizeof(uint32_t));
  p.attn_off = take(S * Hq * (size_t)p.n_splits * (kDim + 2) * sizeof(float));
  p.slscan_off = take(S * sizeof(int32_t));
  p.partx_off = take(S * Hq * sizeof(float2));
  p.chk_pt_off = take(S * mp * sizeof(int32_t));
  p.chk_sl_off = take(S * sizeof(int32_t));
  p.chk_err_off = take((S + 1) * sizeof(int32_t));
  p.total = off;
  return p;
}

static int select_impl(const locks_cfg_t* c, const void* q, const void* summaries,
                       const int32_t* page_table, const int32_t* seq_lens, int32_t* out_page_ids,
                       float* out_sel_lse, float* out_all_lse, void* ws, hipStream_t st) {
  const WsPlan p = plan_workspace(*c);
  Ws w = carve(ws, p);
  float* s_hat = out_all_lse ? out_all_lse : w.s_hat;
  const SHatLayout lay = out_all_lse ? shat_head_major(*c) : shat_head_minor(*c);
  hipError_t e = launch_scan(*c, q, summaries, page_table, seq_lens, s_hat, lay, w.part, st);
  if (e != hipSuccess) return hip_status(e);
  e = launch_select(*c, page_table, seq_lens, s_hat, lay, w.part, w.sel, out_page_ids,
                    out_sel_lse, st);
  return hip_status(e);
}

}  // namespace locks

using namespace locks;

extern "C" {

size_t locks_summary_payload_bytes(int32_t rank) {
  return (rank < 1 || rank > kMaxRank) ? 0 : (size_t)rec_payload(rank);
}

size_t locks_summary_stride(int32_t rank) {
  return (rank < 1 || rank > kMaxRank) ? 0 : (size_t)rec_stride(rank);
}

size_t locks_summary_payload_bytes_ex(int32_t rank, int32_t basis) {
  if (rank < 1 || rank > kMaxRank || basis < LOCKS_BASIS_INT4 || basis > LOCKS_BASIS_BF16) return 0;
  return (size_t)rec_payload(rank, basis);
}

size_t locks_summary_stride_ex(int32_t rank, int32_t basis) {
  if (rank < 1 || rank > kMaxRank || basis < LOCKS_BASIS_INT4 || basis > LOCKS_BASIS_BF16) return 0;
  return (size_t)rec_stride(rank, basis);
}

size_t locks_summary_payload_bytes_page(int32_t rank, int32_t basis, int32_t page_size) {
  if (rank < 1 || rank > kMaxRank || basis < LOCKS_BASIS_INT4 || basis > LOCKS_BASIS_BF16) return 0;
  if (page_size != 16 && page_size != 32 && page_size != 64) return 0;
  return (size_t)rec_payload(rank, basis, page_size);
}

size_t locks_summary_stride_page(int32_t rank, int32_t basis, int32_t page_size) {
  if (rank < 1 || rank > kMaxRank || basis < LOCKS_BASIS_INT4 || basis > LOCKS_BASIS_BF16) return 0;
  if (page_size != 16 && page_size != 32 && page_size != 64) return 0;
  return (size_t)rec_stride(rank, basis, page_size);
}

size_t locks_workspace_bytes(const locks_cfg_t* cfg) {
  if (validate(cfg) != LOCKS_OK) return 0;
  return plan_workspace(*cfg).total;
}

int locks_build_summaries(const locks_cfg_t* cfg, const void* k_cache, const int32_t* page_table,
                          const int32_t* seq_lens, const int32_t* build_list, int32_t n_build,
                          void* summaries, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!k_cache || !page_table || !seq_lens || !summaries || n_build < 0) return LOCKS_E_INVAL;
  if (build_list == nullptr && n_build > 0) return LOCKS_E_INVAL;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  const bool all = build_list == nullptr;
  return hip_status(build_pages(*cfg, k_cache, page_table, seq_lens, build_list, n_build, all,
                                summaries, nullptr, nullptr, nullptr, nullptr,
                                static_cast<hipStream_t>(stream)));
}

int locks_build_factors(const locks_cfg_t* cfg, const void* k_cache, const int32_t* page_table,
                        const int32_t* seq_lens, const int32_t* build_list, int32_t n_build,
                        float* mu, float* basis, float* coef, float* sigma2, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!k_cache || !page_table || !seq_lens || !build_list || n_build < 0 || !mu || !basis ||
      !coef || !sigma2)
    return LOCKS_E_INVAL;
  if (cfg->num_seqs == 0 || n_build == 0) return LOCKS_OK;
  return hip_status(build_pages(*cfg, k_cache, page_table, seq_lens, build_list, n_build, false,
                                nullptr, mu, basis, coef, sigma2, static_cast<hipStream_t>(stream)));
}

int locks_select(const locks_cfg_t* cfg, const void* q, const void* summaries,
                 const int32_t* page_table, const int32_t* seq_lens, int32_t* out_page_ids,
                 float* out_sel_lse, float* out_all_lse, void* ws, size_t ws_bytes, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!q || !summaries || !page_table || !seq_lens || !out_page_ids || !out_sel_lse)
    return LOCKS_E_INVAL;
  if ((rc = check_ws(cfg, ws, ws_bytes))) return rc;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((rc = checked_tables(*cfg, ws, page_table, seq_lens, st))) return rc;
  return select_impl(cfg, q, summaries, page_table, seq_lens, out_page_ids, out_sel_lse,
                     out_all_lse, ws, st);
}

int locks_score_pages(const locks_cfg_t* cfg, const void* q, const void* summaries,
                      const int32_t* page_table, const int32_t* seq_lens, float* out_all_lse,
                      void* ws, size_t ws_bytes, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!q || !summaries || !page_table || !seq_lens || !out_all_lse) return LOCKS_E_INVAL;
  if ((rc = check_ws(cfg, ws, ws_bytes))) return rc;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((rc = checked_tables(*cfg, ws, page_table, seq_lens, st))) return rc;
  const WsPlan p = plan_workspace(*cfg);
  const Ws w = carve(ws, p);
  return hip_status(launch_scan(*cfg, q, summaries, page_table, seq_lens, out_all_lse,
                                shat_head_major(*cfg), w.part, st));
}

int locks_sparse_attend(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                        const int32_t* page_ids, float* out, float* out_lse, void* ws,
                        size_t ws_bytes, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!q || !k_cache || !v_cache || !page_table || !seq_lens || !page_ids || !out)
    return LOCKS_E_INVAL;
  if ((rc = check_ws(cfg, ws, ws_bytes))) return rc;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((rc = checked_tables(*cfg, ws, page_table, seq_lens, st))) return rc;
  const WsPlan p = plan_workspace(*cfg);
  const int pps = sparse_pages_per_split(*cfg);
  const int splits = sparse_splits(*cfg);
  return hip_status(launch_attend(*cfg, q, k_cache, v_cache, page_table, seq_lens, page_ids,
                                  pps, splits, carve(ws, p).attn, out, out_lse, st));
}

int locks_dense_attend(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                       const void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                       float* out, float* out_lse, void* ws, size_t ws_bytes, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!q || !k_cache || !v_cache || !page_table || !seq_lens || !out) return LOCKS_E_INVAL;
  if ((rc = check_ws(cfg, ws, ws_bytes))) return rc;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((rc = checked_tables(*cfg, ws, page_table, seq_lens, st))) return rc;
  const WsPlan p = plan_workspace(*cfg);
  return hip_status(launch_attend(*cfg, q, k_cache, v_cache, page_table, seq_lens, nullptr,
                                  dense_pages_per_split(*cfg), dense_splits(*cfg), carve(ws, p).attn, out,
                                  out_lse, st));
}

int locks_kivi_quantize(const locks_cfg_t* cfg, const locks_kivi_t* kivi, void* k_cache,
                        void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                        const int32_t* page_list, int32_t n_pages, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (cfg->kv_dtype != LOCKS_BF16 || cfg->page_size != kPage) return LOCKS_E_UNSUPPORTED;
  if (!kivi || !kivi_valid(*kivi) || !k_cache || !v_cache || !page_table || !seq_lens ||
      n_pages < 0 || (n_pages > 0 && !page_list))
    return LOCKS_E_INVAL;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  return hip_status(launch_kivi(*cfg, *kivi, k_cache, v_cache, page_table, seq_lens, page_list,
                                n_pages, page_list == nullptr, static_cast<hipStream_t>(stream)));
}

int locks_append_kv(const locks_cfg_t* cfg, const void* k_new, const void* v_new, void* k_cache,
                    void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                    void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!k_new || !v_new || !k_cache || !v_cache || !page_table || !seq_lens) return LOCKS_E_INVAL;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  return hip_status(launch_append(*cfg, k_new, v_new, k_cache, v_cache, page_table, seq_lens,
                                  static_cast<hipStream_t>(stream)));
}

// create_side: the overlapped build may create the device's side stream; without
// it (the allocation-free entry point) a missing side stream means the listed pages
// are built before the scan on `stream`.
static int decode_step_impl(const locks_cfg_t* cfg, const locks_step_opts_t* opts, const void* q,
                            const void* k_cache, const void* v_cache, const int32_t* page_table,
                            const int32_t* seq_lens, void* summaries, const int32_t* build_list,
                            int32_t n_build, int32_t* out_page_ids, float* out_sel_lse,
                            float* out, float* out_lse, void* ws, size_t ws_bytes, void* stream,
                            bool create_side = true) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (!q || !k_cache || !v_cache || !page_table || !seq_lens || !summaries || !out_page_ids ||
      !out_sel_lse || !out || n_build < 0 || (n_build > 0 && !build_list))
    return LOCKS_E_INVAL;
  const locks_kivi_t* kivi = opts ? opts->kivi : nullptr;
  const void* k_new = opts ? opts->k_new : nullptr;
  const void* v_new = opts ? opts->v_new : nullptr;
  if ((k_new == nullptr) != (v_new == nullptr)) return LOCKS_E_INVAL;
  if (kivi && (cfg->kv_dtype != LOCKS_BF16 || cfg->page_size != kPage)) return LOCKS_E_UNSUPPORTED;
  if (kivi && !kivi_valid(*kivi)) return LOCKS_E_INVAL;
  if ((rc = check_ws(cfg, ws, ws_bytes))) return rc;
  if (cfg->num_seqs == 0) return LOCKS_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if ((rc = checked_tables(*cfg, ws, page_table, seq_lens, st))) return rc;
  // KIVI finalisation of the listed pages, always on the stream that builds them:
  // PRE right before their build, POST right after it; either way before the
  // attention reads them.
  if (!kivi || n_build == 0) kivi = nullptr;
  void* kq = const_cast<void*>(k_cache);
  void* vq = const_cast<void*>(v_cache);
  auto kivi_at = [&](int stage, hipStream_t on, KiviPages which) -> hipError_t {
    if (!kivi || kivi->stage != stage) return hipSuccess;
    return launch_kivi(*cfg, *kivi, kq, vq, page_table, seq_lens, build_list, n_build, false, on,
                       which);
  };
  // the new token's KV write: beside the scan when the step forks it, else first
  auto append = [&]() -> hipError_t {
    if (!k_new) return hipSuccess;
    return launch_append(*cfg, k_new, v_new, kq, vq, page_table, seq_lens, st);
  };
  // The pages that just filled are built beside the scan on a side stream (bf16 q
  // and KV, int4 basis); the lock also serialises the fork / join enqueues.
  std::unique_lock<std::mutex> side_lock;
  SideStream* side = nullptr;
  if (attend_select_fused(*cfg) && n_build > 0 && cfg->basis == LOCKS_BASIS_INT4 &&
      cfg->page_size == kPage) {
    side_lock = std::unique_lock<std::mutex>(g_side_mu);
    if ((rc = hip_status(side_stream(&side, create_side)))) return rc;
  }
  const bool forked = side != nullptr;
  if (!forked && (rc = hip_status(append()))) return rc;
  if (!forked && (rc = hip_status(kivi_at(LOCKS_KIVI_PRE, st, kKiviAny)))) return rc;
  auto post_kivi = [&]() -> int { return hip_status(kivi_at(LOCKS_KIVI_POST, st, kKiviAny)); };
  const WsPlan p = plan_workspace(*cfg);
  const Ws w = carve(ws, p);
  const int pps = sparse_pages_per_split(*cfg);
  const int splits = sparse_splits(*cfg);
  if (attend_select_fused(*cfg)) {
    // scan -> per-chunk selection -> attention whose blocks merge the table
    const SHatLayout lay = shat_head_minor(*cfg);
    const float2* part_x = nullptr;
    if (n_build > 0 && !forked) {
      rc = hip_status(build_pages(*cfg, k_cache, page_table, seq_lens, build_list, n_build, false,
                                   summaries, nullptr, nullptr, nullptr, nullptr, st));
      if (rc) return rc;
      if ((rc = post_kivi())) return rc;
      rc = hip_status(launch_scan(*cfg, q, summaries, page_table, seq_lens, w.s_hat, lay, w.part,
                                  st));
      if (rc) return rc;
    } else if (n_build > 0) {
      // Listed pages that are the last complete page of their sequence (the
      // pages that just filled) are built and scored on `stream` while a side
      // stream, forked before them, builds the other listed pages and then scans
      // everything but those last pages.  The builds' few blocks are dispatched
      // first and stay resident beside the scan (the fork costs the side stream
      // a few microseconds); `stream` joins the side stream before the selection.
      const BuildStep bs{w.sl_scan, w.part_x, q, cfg->q_dtype == LOCKS_BF16, cfg->num_q_heads,
                         w.s_hat, lay};
      hipError_t e = hipEventRecord(side->fork, st);
      if (e == hipSuccess) e = hipStreamWaitEvent(side->st, side->fork, 0);
      if (e == hipSuccess) e = append();
      if (e == hipSuccess) e = kivi_at(LOCKS_KIVI_PRE, st, kKiviLast);
      if (e == hipSuccess)
        e = launch_build(*cfg, k_cache, page_table, seq_lens, build_list, n_build, false, summaries,
                         nullptr, nullptr, nullptr, nullptr, st, kBuildLast, &bs);
      if (e == hipSuccess) e = kivi_at(LOCKS_KIVI_POST, st, kKiviLast);
      if (e == hipSuccess) e = kivi_at(LOCKS_KIVI_PRE, side->st, kKiviInner);
      if (e == hipSuccess)
        e = launch_build(*cfg, k_cache, page_table, seq_lens, build_list, n_build, false, summaries,
                         nullptr, nullptr, nullptr, nullptr, side->st, kBuildInner, &bs);
      if (e == hipSuccess) e = kivi_at(LOCKS_KIVI_POST, side->st, kKiviInner);
      if (e == hipSuccess)
        e = launch_scan(*cfg, q, summaries, page_table, w.sl_scan, w.s_hat, lay, w.part, side->st);
      if (e == hipSuccess) e = hipEventRecord(side->join, side->st);
      if (e == hipSuccess) e = hipStreamWaitEvent(st, side->join, 0);
      if ((rc = hip_status(e))) return rc;
      part_x = w.part_x;
    } else {
      rc = hip_status(launch_scan(*cfg, q, summaries, page_table, seq_lens, w.s_hat, lay, w.part,
                                  st));
      if (rc) return rc;
    }
    rc = hip_status(launch_select_chunks(*cfg, page_table, seq_lens, w.s_hat, lay, w.part, w.sel,
                                         st, part_x, w.sl_scan));
    if (rc) return rc;
    return hip_status(launch_attend_select(*cfg, q, k_cache, v_cache, page_table, seq_lens, w.sel,
                                           w.s_hat, lay, out_page_ids, out_sel_lse,
                                           pps, splits, w.attn, out, out_lse, st));
  }
  if (n_build > 0) {
    rc = hip_status(build_pages(*cfg, k_cache, page_table, seq_lens, build_list, n_build, false,
                                 summaries, nullptr, nullptr, nullptr, nullptr, st));
    if (rc) return rc;
    if ((rc = post_kivi())) return rc;
  }
  rc = select_impl(cfg, q, summaries, page_table, seq_lens, out_page_ids, out_sel_lse, nullptr, ws,
                   st);
  if (rc) return rc;
  return hip_status(launch_attend(*cfg, q, k_cache, v_cache, page_table, seq_lens, out_page_ids,
                                  pps, splits, w.attn, out, out_lse, st));
}

int locks_decode_step(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                      const void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                      void* summaries, const int32_t* build_list, int32_t n_build,
                      int32_t* out_page_ids, float* out_sel_lse, float* out, float* out_lse,
                      void* ws, size_t ws_bytes, void* stream) {
  return decode_step_impl(cfg, nullptr, q, k_cache, v_cache, page_table, seq_lens, summaries,
                          build_list, n_build, out_page_ids, out_sel_lse, out, out_lse, ws,
                          ws_bytes, stream);
}

int locks_decode_step_ex(const locks_cfg_t* cfg, const locks_step_opts_t* opts, const void* q,
                         void* k_cache, void* v_cache, const int32_t* page_table,
                         const int32_t* seq_lens, void* summaries, const int32_t* build_list,
                         int32_t n_build, int32_t* out_page_ids, float* out_sel_lse, float* out,
                         float* out_lse, void* ws, size_t ws_bytes, void* stream) {
  return decode_step_impl(cfg, opts, q, k_cache, v_cache, page_table, seq_lens, summaries,
                          build_list, n_build, out_page_ids, out_sel_lse, out, out_lse, ws,
                          ws_bytes, stream);
}

int locks_decode_step_static(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                             const void* v_cache, const int32_t* page_table,
                             const int32_t* seq_lens, void* summaries,
                             const int32_t* build_list, int32_t n_build, int32_t* out_page_ids,
                             float* out_sel_lse, float* out, float* out_lse, void* stream) {
  int rc = validate(cfg);
  if (rc) return rc;
  if (plan_workspace(*cfg).total > kStaticScratchBytes) return LOCKS_E_WORKSPACE;
  void* ws = nullptr;
  if ((rc = hip_status(scratch_ptr(&ws)))) return rc;
  return decode_step_impl(cfg, nullptr, q, k_cache, v_cache, page_table, seq_lens, summaries,
                          build_list, n_build, out_page_ids, out_sel_lse, out, out_lse, ws,
                          kStaticScratchBytes, stream, /*create_side=*/false);
}

int locks_init(void) {
  void* ws = nullptr;
  int rc = hip_status(scratch_ptr(&ws));
  if (rc) return rc;
  std::lock_guard<std::mutex> lock(g_side_mu);
  SideStream* side = nullptr;
  return hip_status(side_stream(&side));
}

int locks_set_table_checks(int32_t enable) {
  return g_table_checks.exchange(enable ? 1 : 0);
}

size_t locks_table_error_offset(const locks_cfg_t* cfg) {
  if (validate(cfg) != LOCKS_OK) return (size_t)-1;
  return plan_workspace(*cfg).chk_err_off;
}

const char* locks_strerror(int status) {
  switch (status) {
    case LOCKS_OK: return "ok";
    case LOCKS_E_INVAL: return "invalid argument";
    case LOCKS_E_UNSUPPORTED: return "unsupported configuration";
    case LOCKS_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case LOCKS_E_HIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

int locks_last_hip_error(void) { return g_last_hip_error; }

}  // extern "C"
