// Checked tables: the device-side guard of the step's page-table and
// sequence-length reads.  Every call that takes a workspace can run it first;
// the other kernels then read the checked copies, so an out-of-range value is
// clamped and reported instead of being dereferenced.
//
// Per sequence s: L = seq_lens[s] is clamped to [0, B * max_pages] (bit
// LOCKS_TABLE_E_LENGTH when it was outside); every entry j < ceil(L_clamped / B)
// of its page-table row must lie in [0, num_blocks), else it becomes block 0 (bit
// LOCKS_TABLE_E_BLOCK).  Entries past the last page are not read; their copies
// are 0.  A second kernel ORs the per-sequence words into the call's error word.
#include "locks_internal.h"

namespace locks {
namespace {

__global__ __launch_bounds__(256) void check_rows_kernel(const int32_t* __restrict__ page_table,
                                                         const int32_t* __restrict__ seq_lens,
                                                         int max_pages, int pgsz, int num_blocks,
                                                         int32_t* __restrict__ pt_out,
                                                         int32_t* __restrict__ sl_out,
                                                         int32_t* __restrict__ err_rows) {
  const int s = blockIdx.x;
  const int L = seq_lens[s];
  const long cap = (long)pgsz * max_pages;
  const int Lc = L < 0 ? 0 : (L > cap ? (int)cap : L);
  const int n = (Lc + pgsz - 1) / pgsz;
  const int32_t* row = page_table + (long)s * max_pages;
  int32_t* out = pt_out + (long)s * max_pages;
  int bad = 0;
  for (int j = threadIdx.x; j < max_pages; j += blockDim.x) {
    int32_t b = 0;
    if (j < n) {
      b = row[j];
      if (b < 0 || b >= num_blocks) {
        bad = 1;
        b = 0;
      }
    }
    out[j] = b;
  }
  bad = __syncthreads_or(bad);
  if (threadIdx.x == 0) {
    sl_out[s] = Lc;
    err_rows[s] = (Lc != L ? LOCKS_TABLE_E_LENGTH : 0) | (bad ? LOCKS_TABLE_E_BLOCK : 0);
  }
}

__global__ __launch_bounds__(256) void check_or_kernel(const int32_t* __restrict__ err_rows, int S,
                                                       int32_t* __restrict__ err_word) {
  int w = 0;
  for (int s = threadIdx.x; s < S; s += blockDim.x) w |= err_rows[s];
  // OR over the block: every bit is set by some thread or by none
  int out = 0;
#pragma unroll
  for (int bit = 0; bit < 2; ++bit) out |= __syncthreads_or(w & (1 << bit)) ? (1 << bit) : 0;
  if (threadIdx.x == 0) *err_word = out;
}

}  // namespace

hipError_t launch_check_tables(const locks_cfg_t& c, const int32_t* page_table,
                               const int32_t* seq_lens, int32_t* pt_out, int32_t* sl_out,
                               int32_t* err_word, int32_t* err_rows, hipStream_t st) {
  if (c.num_seqs <= 0) return hipSuccess;
  hipLaunchKernelGGL(check_rows_kernel, dim3(c.num_seqs), dim3(256), 0, st, page_table, seq_lens,
                     c.max_pages_per_seq, c.page_size, c.num_blocks, pt_out, sl_out, err_rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(check_or_kernel, dim3(1), dim3(256), 0, st, err_rows, c.num_seqs, err_word);
  return hipGetLastError();
}

}  // namespace locks
