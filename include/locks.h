/*
 * locks.h -- C ABI of the Locks per-step sparse decode attention for AMD
 * Instinct MI355X (gfx950).
 *
 * The method (arXiv 2607.24555): every KV page of B tokens (B = 16; 32 and 64 are
 * the page sizes of App. D.3) keeps a resident rank-r spectral summary of its keys
 * (Sec. 4 "Build"); every decode step rebuilds each page's B logits from its
 * summary and takes their log-sum-exp (Sec. 4 "Score",
 * Eq. (1)), averages the normalised page shares over the GQA group, keeps the
 * sink page, the most recent page and the top (k-2) other pages (Sec. 4, Cor.
 * "Group-shared selection"), and runs exact attention over those pages only
 * (Sec. 2 "Decode-time attention"; App. E).
 *
 * Conventions shared by every call
 *  - All tensor arguments are DEVICE pointers owned by the caller; the library
 *    never allocates device memory, frees, synchronises or throws.  Every call
 *    enqueues its kernels on `stream` (a hipStream_t; NULL = the default stream;
 *    locks_decode_step may fork part of its work to a side stream, see there)
 *    and returns a status immediately.
 *  - Host-side checks (configuration, null pointers, workspace size) run before
 *    any launch; a failing check returns an error and launches nothing.
 *    Device-resident values (page-table entries, sequence lengths) are trusted:
 *    page_table[s][j] must be a valid block for every j < ceil(seq_lens[s]/B),
 *    and seq_lens[s] <= B * max_pages_per_seq (B = page_size).  Entries past a
 *    sequence's last page are never read.  With table checks on
 *    (locks_set_table_checks) every call that takes a workspace checks them on
 *    the device instead, clamps what is out of range and reports it in an error
 *    word inside the workspace.
 *  - Layouts (row-major, innermost last):
 *      q           [num_seqs][num_q_heads][128]          (q_dtype)
 *      k/v cache   [num_blocks][num_kv_heads][B][128]    (kv_dtype, B = page_size)
 *      page_table  int32 [num_seqs][max_pages_per_seq]   logical page -> block
 *      seq_lens    int32 [num_seqs]                      tokens per sequence
 *      summaries   uint8 [num_blocks][num_kv_heads][stride]
 *                  stride = locks_summary_stride_page(rank, basis, page_size)
 *    Query head h belongs to KV head h / (num_q_heads / num_kv_heads).
 *  - Page ids returned and accepted by this API are LOGICAL page indices within
 *    their sequence.  Page j holds tokens [Bj, Bj+B); page 0 is the sink and
 *    page ceil(L/B)-1 is the most recent page.  A page has a summary only once
 *    it is complete (B tokens).
 *  - The workspace `ws` (caller-allocated, >= locks_workspace_bytes(cfg) bytes,
 *    256-byte aligned) holds per-call scratch; its content need not be
 *    initialised and is meaningless after the call.  No call clears memory, so a
 *    captured step replays without extra nodes.  Calls that share one workspace
 *    must be ordered on one stream.
 *  - Calls with no launches (num_seqs == 0) return LOCKS_OK.
 */
#ifndef LOCKS_H
#define LOCKS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
  LOCKS_OK = 0,
  LOCKS_E_INVAL = -1,        /* bad configuration value or null pointer          */
  LOCKS_E_UNSUPPORTED = -2,  /* head_dim != 128, page_size not 16, 32 or 64, an
                                int8 / bf16 basis or KIVI with page_size != 16,
                                G > 16, dtype unknown, or a summary store of
                                4 GiB or more (num_blocks * num_kv_heads * stride) */
  LOCKS_E_WORKSPACE = -3,    /* ws null or smaller than locks_workspace_bytes    */
  LOCKS_E_HIP = -4           /* a HIP launch failed; see locks_last_hip_error    */
};

/* Element types of q and of the KV cache. */
enum { LOCKS_BF16 = 0, LOCKS_FP32 = 1 };

/* Precision of the stored basis V (Sec. 5 "Ablations"; the r8fp control of the
 * retention remark): int4 (the deployed summary), int8, or bfloat16.
 * Coefficients and centroid are int8 in all three. */
enum { LOCKS_BASIS_INT4 = 0, LOCKS_BASIS_INT8 = 1, LOCKS_BASIS_BF16 = 2 };

/* Fixed-shape configuration of one decode step (Sec. 4 "Implementation": r, B and
 * b fixed, hence fixed shapes). */
typedef struct locks_cfg {
  int32_t num_seqs;          /* S >= 0                                          */
  int32_t num_q_heads;       /* H_q, a multiple of H_kv; G = H_q / H_kv <= 16   */
  int32_t num_kv_heads;      /* H_kv >= 1                                       */
  int32_t head_dim;          /* d, must be 128                                  */
  int32_t page_size;         /* B: 16, or 32 / 64 (App. D.3 "Page size")        */
  int32_t rank;              /* r in [1, 15]                                    */
  int32_t budget_tokens;     /* b; the page budget k = ceil(b / B) must be >= 2
                                (sink and most recent page take two slots,
                                Sec. 2 and App. C.1 "Budget counting")          */
  int32_t max_pages_per_seq; /* row stride of page_table, >= 1                  */
  int32_t num_blocks;        /* physical blocks in the caches, >= 1             */
  int32_t kv_dtype;          /* LOCKS_BF16 or LOCKS_FP32                        */
  int32_t q_dtype;           /* LOCKS_BF16 or LOCKS_FP32                        */
  int32_t basis;             /* LOCKS_BASIS_INT4 (0), _INT8 or _BF16; the int8
                                and bf16 bases take r in {2, 4, 8}              */
} locks_cfg_t;

/* Stored payload of one page summary (Sec. 4 "Build"; App. C.1 table):
 * d*r/2 int4 basis bytes + B*r int8 coefficient bytes + d int8 centroid bytes +
 * 2*(r + B + 1) bytes of float16 scales = 818 / 490 / 326 bytes at r = 8 / 4 / 2.
 * Returns 0 for r outside [1, 15]. */
size_t locks_summary_payload_bytes(int32_t rank);

/* Record stride in the summary store: the payload rounded up to 16 bytes
 * (832 / 496 / 336 at r = 8 / 4 / 2).  Record layout, byte offsets:
 *   [0, 64r)          basis V (d x r): column l at 64*l, 128 excess-8 nibbles,
 *                     element c in byte c/2, low nibble for even c; code in [-7, 7]
 *   [64r, 80r)        coefficients C (16 x r) row-major, excess-128 bytes
 *   [80r, 80r+128)    centroid mu, excess-128 bytes
 *   [80r+128, +2(r+17)) float16 scales: r basis columns, 16 coefficient rows,
 *                     1 centroid; value = code * scale
 *   rest              zero padding
 * Returns 0 for r outside [1, 15]. */
size_t locks_summary_stride(int32_t rank);

/* Payload and record stride for any basis precision.  The record keeps the field
 * order above with the basis columns widened: column l at (64 << basis) * l,
 * holding 128 excess-128 int8 codes (LOCKS_BASIS_INT8, one float16 scale per
 * column as for int4) or 128 little-endian bfloat16 values (LOCKS_BASIS_BF16,
 * round to nearest even; the column scales hold 1.0); the coefficients, centroid
 * and scales follow at the same relative offsets.  Payload = (64 << basis) r +
 * 16 r + 128 + 2 (r + 17): 818 / 1330 / 2354 bytes at r = 8.  Returns 0 for an
 * unknown basis or r outside [1, 15]. */
size_t locks_summary_payload_bytes_ex(int32_t rank, int32_t basis);
size_t locks_summary_stride_ex(int32_t rank, int32_t basis);

/* Payload and record stride for pages of page_size = B tokens (16, 32 or 64;
 * App. D.3 "Page size"): the coefficient block holds B rows and the scales
 * r + B + 1 entries, so for the int4 basis payload = 64 r + B r + 128 + 2 (r + B + 1)
 * (978 and 1298 bytes at r = 8 for B = 32 and 64), the fields in the order above.
 * Returns 0 for an unknown basis or page size or r outside [1, 15]. */
size_t locks_summary_payload_bytes_page(int32_t rank, int32_t basis, int32_t page_size);
size_t locks_summary_stride_page(int32_t rank, int32_t basis, int32_t page_size);

/* Bytes of workspace the select / attend / decode-step calls need for cfg
 * (0 if cfg is invalid). */
size_t locks_workspace_bytes(const locks_cfg_t* cfg);

/* Build the summaries of complete pages (Sec. 4 "Build"): per (page, KV head)
 * centre the B keys, eigendecompose the B x B Gram of the deviations, keep the
 * r leading nonzero modes (a mode counts as zero when its eigenvalue is at most
 * max(1e-6 * leading eigenvalue, 1e-10 * mean squared key norm)), form the
 * orthonormal basis V = D^T U_r S_r^{-1} and coefficients C = U_r S_r, make each
 * basis column's largest-magnitude entry positive, quantise (basis int4 per
 * column, coefficients int8 per row, centroid int8; scale = f16(max|x|/qmax),
 * code = round-half-even(x / scale)) and write the record of every KV head of
 * that page into summaries[block].
 *   build_list  NULL: every complete page of every sequence.  Otherwise n_build
 *               int32 pairs (seq, logical page) in device memory; pairs that do
 *               not name a complete page are skipped.
 * Returns LOCKS_E_INVAL for n_build < 0 or a null k_cache / page_table /
 * seq_lens / summaries. */
int locks_build_summaries(const locks_cfg_t* cfg, const void* k_cache,
                          const int32_t* page_table, const int32_t* seq_lens,
                          const int32_t* build_list, int32_t n_build,
                          void* summaries, void* stream);

/* The same build without quantisation (the float basis variant): for each of the
 * n_build listed (seq, page) pairs (build_list required) and each KV head, write
 *   mu     float [n_build][H_kv][128]
 *   basis  float [n_build][H_kv][128][r]   (sign convention as above)
 *   coef   float [n_build][H_kv][B][r]
 *   sigma2 float [n_build][H_kv][B]        all Gram eigenvalues, descending, >= 0
 * Dropped modes have zero basis and coefficient columns.  Listed pairs that are
 * not complete pages leave their rows untouched. */
int locks_build_factors(const locks_cfg_t* cfg, const void* k_cache,
                        const int32_t* page_table, const int32_t* seq_lens,
                        const int32_t* build_list, int32_t n_build,
                        float* mu, float* basis, float* coef, float* sigma2,
                        void* stream);

/* Score every complete page from its summary (Sec. 4 "Score", Eq. (1)):
 *   out_all_lse[s][h][j] = hat s_j(q_h) for every complete page j of sequence s
 *   (float [S][H_q][max_pages_per_seq]; entries of other pages are not written).
 * This is the scan that locks_select runs first, exposed on its own. */
int locks_score_pages(const locks_cfg_t* cfg, const void* q, const void* summaries,
                      const int32_t* page_table, const int32_t* seq_lens, float* out_all_lse,
                      void* ws, size_t ws_bytes, void* stream);

/* Score every complete page from its summary and select the shared page table
 * (Sec. 4 "Score", Eq. (1) and the share-average combine; Cor. "Group-shared
 * selection"; App. E "union table"):
 *   hat s_j(q_g) = log sum_i exp[(q_g^T mu_j + (V_j^T q_g)^T c_i) / sqrt(128)],
 *   mbar_j = (1/G) sum_g exp(hat s_j(q_g)) / sum_{j'} exp(hat s_j'(q_g)),
 * the normaliser summing every complete page of the sequence.  The table of each
 * (seq, KV head) holds page 0, the most recent page and the k-2 other pages of
 * largest mbar (lower index first on ties), in ascending order; a sequence with at
 * most k pages selects all of them.
 *   out_page_ids  int32 [S][H_kv][k], ascending, padded with -1
 *   out_sel_lse   float [S][H_q][k], hat s of each selected page (natural log,
 *                 1/sqrt(d) included); NaN for padding and for a page without
 *                 summary (the partial last page)
 *   out_all_lse   nullable float [S][H_q][max_pages_per_seq]: hat s of every
 *                 complete page (entries of other pages are not written). */
int locks_select(const locks_cfg_t* cfg, const void* q, const void* summaries,
                 const int32_t* page_table, const int32_t* seq_lens,
                 int32_t* out_page_ids, float* out_sel_lse, float* out_all_lse,
                 void* ws, size_t ws_bytes, void* stream);

/* Exact attention of every query head over the tokens of its KV head's selected
 * pages, softmax renormalised over that set (Sec. 2; App. E "sparse decode"):
 *   o_g = sum_{i in S} softmax_S(q_g^T k_i / sqrt(128)) v_i.
 * The partial last page contributes its valid tokens only; -1 entries of
 * page_ids are skipped; ids must be < ceil(seq_lens[s]/B).
 *   page_ids  int32 [S][H_kv][k] (k from cfg->budget_tokens)
 *   out       float [S][H_q][128]
 *   out_lse   nullable float [S][H_q], log of the softmax denominator
 * A query with no token to attend gets out = 0 and out_lse = -inf. */
int locks_sparse_attend(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* page_table,
                        const int32_t* seq_lens, const int32_t* page_ids,
                        float* out, float* out_lse, void* ws, size_t ws_bytes,
                        void* stream);

/* Dense paged decode attention over every token of each sequence (Sec. 2,
 * decode-time attention): the same-GPU baseline, with locks_sparse_attend's
 * arguments minus page_ids. */
int locks_dense_attend(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                       const void* v_cache, const int32_t* page_table,
                       const int32_t* seq_lens, float* out, float* out_lse,
                       void* ws, size_t ws_bytes, void* stream);

/* One fused decode step (App. E critical path, allocation-free and fixed-shape):
 * first the summaries of the n_build listed (seq, page) pairs are built (pages
 * that completed this step; n_build = 0 builds nothing, build_list may then be
 * NULL), then locks_select, then locks_sparse_attend over the selected table, all
 * ordered after earlier work on `stream` and before later work on it.  With bf16
 * q and KV and a listed page that is the last complete page of its sequence, the
 * build of those pages runs on `stream` beside the scan of the others, which the
 * library enqueues on a side stream of its own (one per device, created by
 * locks_init or else on first use -- a call that creates it cannot be captured --
 * and kept until the process ends), forked from and joined back to `stream` by
 * events, so a captured step records the fork and join too; such calls on one
 * device are serialised on the host.  Outputs as in those calls. */
int locks_decode_step(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                      const void* v_cache, const int32_t* page_table,
                      const int32_t* seq_lens, void* summaries,
                      const int32_t* build_list, int32_t n_build,
                      int32_t* out_page_ids, float* out_sel_lse, float* out,
                      float* out_lse, void* ws, size_t ws_bytes, void* stream);

/* KV-cache quantisation of finalised pages (Sec. 5 "KV-cache quantization under
 * extreme sparsity"; App. C, protocol of the full KIVI grid): KIVI's asymmetric
 * min/max quantiser applied as fake quantisation -- quantise, then dequantise back
 * to bfloat16 in place -- to complete pages only (the partial last page stays as
 * written).  Keys share one scale and zero point per channel over the page's 16
 * tokens; values one per token and group of v_group consecutive channels.  Each
 * slice x with min m and max M: s = (M - m) / (2^bits - 1) and
 *   x' = bf16(min(rint((x - m) / s), 2^bits - 1) * s + m),
 * every operation one IEEE float32 rounding (rint and the final bfloat16 rounding
 * to nearest even); a slice with s = 0 keeps its values.
 * The stage orders the quantiser against the summary build in the fused step:
 * POST builds a page's summary from the keys as written and then quantises the
 * page, so selection sees unquantised keys and attention quantised KV; PRE
 * quantises first and builds the summary from the quantised keys. */
enum { LOCKS_KIVI_POST = 0, LOCKS_KIVI_PRE = 1 };
typedef struct locks_kivi {
  int32_t bits;     /* b in [1, 8], 2^b levels (the paper's grid: 4 and 2)     */
  int32_t v_group;  /* channels per value scale: 8, 16, 32, 64 or 128          */
  int32_t stage;    /* LOCKS_KIVI_POST or LOCKS_KIVI_PRE                       */
} locks_kivi_t;

/* Fake-quantise, in place, the K and V of complete pages: every complete page of
 * every sequence (page_list NULL, n_pages 0) or the n_pages listed (seq, logical
 * page) int32 pairs in device memory (pairs that name no complete page are
 * skipped; a page may be listed once per call -- duplicates race).  All KV heads of
 * a page are quantised; kivi->stage is not used here.  Quantising a page twice is
 * not the identity in general, so each page should be finalised once.
 * Returns LOCKS_E_UNSUPPORTED unless kv_dtype is LOCKS_BF16 and page_size is 16,
 * LOCKS_E_INVAL for a
 * null kivi / cache / page_table / seq_lens, bits or v_group out of range,
 * n_pages < 0, or n_pages > 0 with a null page_list. */
int locks_kivi_quantize(const locks_cfg_t* cfg, const locks_kivi_t* kivi, void* k_cache,
                        void* v_cache, const int32_t* page_table, const int32_t* seq_lens,
                        const int32_t* page_list, int32_t n_pages, void* stream);

/* The caller's KV write of a decode step (App. E: the new token's KV write is
 * scheduled beside the selection): for every sequence s with seq_lens[s] >= 1,
 * the key and value rows k_new[s][h], v_new[s][h] ([num_seqs][num_kv_heads][128],
 * kv_dtype) are copied into the slot of token seq_lens[s] - 1, i.e. logical page
 * (seq_lens[s] - 1) / B (its block must be in page_table), row (seq_lens[s] - 1)
 * % B, of every KV head.  seq_lens already counts the new token; nothing else is
 * written.  Returns LOCKS_E_INVAL for a null argument. */
int locks_append_kv(const locks_cfg_t* cfg, const void* k_new, const void* v_new,
                    void* k_cache, void* v_cache, const int32_t* page_table,
                    const int32_t* seq_lens, void* stream);

/* Options of locks_decode_step_ex; all fields NULL is locks_decode_step. */
typedef struct locks_step_opts {
  const locks_kivi_t* kivi;  /* NULL, or KIVI fake quantisation of the listed pages */
  const void* k_new;         /* NULL, or this step's new key and value rows, as     */
  const void* v_new;         /* locks_append_kv takes them (both or neither)        */
} locks_step_opts_t;

/* locks_decode_step with the new token's KV write and KV-cache quantisation folded
 * in.  With k_new / v_new the step first writes each sequence's newest token as
 * locks_append_kv does (seq_lens already counting it); when the step builds the
 * last complete pages beside the scan, this write runs beside the scan too, on
 * `stream` before those builds.  With kivi the n_build listed pages (the pages
 * finalised this step) are fake-quantised as locks_kivi_quantize does, before
 * their summary build (kivi->stage == LOCKS_KIVI_PRE) or after it
 * (LOCKS_KIVI_POST), each on the stream that builds it, and before the attention
 * reads them (kivi requires bf16 caches and 16-token pages, else
 * LOCKS_E_UNSUPPORTED).  The rest of
 * the step is locks_decode_step's; opts == NULL is locks_decode_step itself.
 * Returns LOCKS_E_INVAL when exactly one of k_new, v_new is given. */
int locks_decode_step_ex(const locks_cfg_t* cfg, const locks_step_opts_t* opts, const void* q,
                         void* k_cache, void* v_cache, const int32_t* page_table,
                         const int32_t* seq_lens, void* summaries,
                         const int32_t* build_list, int32_t n_build,
                         int32_t* out_page_ids, float* out_sel_lse, float* out,
                         float* out_lse, void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes that locks_decode_step_static holds per device: 64 MiB, enough
 * for every configuration whose locks_workspace_bytes is at most that (the 1M-token
 * single-sequence step needs about 13 MiB, 8 x 128K about 16 MiB, 64 sequences of
 * up to 64K tokens about 57 MiB). */
#define LOCKS_STATIC_SCRATCH_BYTES ((size_t)64 << 20)

/* locks_decode_step without a caller workspace, for callers that cannot allocate
 * device memory at all: code under stream capture, tight serving loops, harnesses
 * that forbid hipMalloc.  The step's scratch lives in a static device array of
 * LOCKS_STATIC_SCRATCH_BYTES inside the library (one per device, held until the
 * process ends); the call itself allocates nothing -- no device memory, and no
 * stream or event either: when the overlapped build of the last pages (see
 * locks_decode_step) would need the device's side stream and locks_init has not
 * created it, the listed pages are built before the scan on `stream` instead
 * (the same step; those pages' scores come out of the scan rather than the build,
 * equal up to float rounding).  Every call on a device shares that device's array
 * and leaves its contents behind; no call needs it cleared, but calls that overlap
 * on one device (two streams, two threads, two graphs in flight) race on it and
 * must be ordered by the caller.  Arguments, outputs and errors as in
 * locks_decode_step, plus LOCKS_E_WORKSPACE when locks_workspace_bytes(cfg)
 * exceeds LOCKS_STATIC_SCRATCH_BYTES (nothing is launched). */
int locks_decode_step_static(const locks_cfg_t* cfg, const void* q, const void* k_cache,
                             const void* v_cache, const int32_t* page_table,
                             const int32_t* seq_lens, void* summaries,
                             const int32_t* build_list, int32_t n_build, int32_t* out_page_ids,
                             float* out_sel_lse, float* out, float* out_lse, void* stream);

/* Set-up for the current device (App. E: the step replays from a captured graph):
 * creates the device's side stream and its two events that locks_decode_step
 * forks to, so that no later call creates them -- in particular none under stream
 * capture -- and looks up the device address of locks_decode_step_static's
 * scratch array.  Call it once per device, with that device current, before the first
 * step that may be captured; calling it again is a no-op.  Returns LOCKS_E_HIP
 * if the stream or an event cannot be created. */
int locks_init(void);

/* Bits of the table-check error word. */
enum {
  LOCKS_TABLE_E_LENGTH = 1,  /* some seq_lens[s] < 0 or > B * max_pages_per_seq    */
  LOCKS_TABLE_E_BLOCK = 2    /* some page_table[s][j], j < ceil(L / B), outside
                                [0, num_blocks)                                   */
};

/* Table checks, the device-side guard of the tables' reads, for debugging a
 * caller's page tables (process-wide; off by default; returns the previous
 * setting).  While on, every call that takes a workspace (locks_select,
 * locks_score_pages, locks_sparse_attend, locks_dense_attend and the decode
 * steps) first runs two small kernels on its stream that copy seq_lens and the
 * page-table rows into the workspace, clamping each length to
 * [0, B * max_pages_per_seq] and replacing each out-of-range entry of a sequence's
 * pages by block 0; the call's other kernels read those copies.  The OR of the
 * LOCKS_TABLE_E_* bits over the sequences is written to the int32 at byte offset
 * locks_table_error_offset(cfg) of the workspace, followed by one int32 per
 * sequence; it holds the last checked call's result until the next call that
 * uses the workspace (read it after that call completes).  Outputs of a call
 * with a nonzero word are computed on the clamped tables and are not
 * meaningful.  The calls without a workspace (builds, KV write, KIVI pass)
 * are not checked. */
int locks_set_table_checks(int32_t enable);

/* Byte offset of the table-check error word in the workspace of `cfg`; (size_t)-1
 * for an invalid configuration. */
size_t locks_table_error_offset(const locks_cfg_t* cfg);

/* Static description of a status code. */
const char* locks_strerror(int status);

/* The hipError_t of the last failed launch on the calling thread (0 if none). */
int locks_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LOCKS_H */
