// Cache compaction (sections 1 and 3.1: each layer keeps B entries, plus the always-kept tail).
//
// One workgroup per (problem, kv head): the B_p admitted positions (B_p = the problem's own budget,
// or the uniform B) are sorted in LDS (bitonic sort over the next power of two, padded with
// INT_MAX), then the kept rows of K and V are copied with 16-byte vector loads and stores into rows
// 0 .. B_p + keep_tail - 1 of the unit's block of out_rows rows (compact_rows.h).  Rows are opaque
// bytes, so the copy is exact for every dtype.
#include <limits.h>

#include "common.h"
#include "compact_rows.h"
#include "kernels.h"

namespace kv {

namespace {
constexpr int kThreads = 256;
constexpr int kMaxSortedBudget = 8192;
}  // namespace

__global__ __launch_bounds__(kThreads) void compact_kernel(
    const uint4* __restrict__ k, const uint4* __restrict__ v, const int32_t* __restrict__ sel_idx,
    const int32_t* __restrict__ lens, const int64_t* __restrict__ tok_off, int h_kv,
    int row_vecs, int budget, const int32_t* __restrict__ budgets, int keep_tail, int out_rows,
    uint4* __restrict__ k_out, uint4* __restrict__ v_out) {
  __shared__ int32_t srt[kMaxSortedBudget];
  const int g = blockIdx.x % h_kv, p = blockIdx.x / h_kv;
  const int L = lens[p];
  const int bp = budgets ? budgets[p] : budget;
  int n2 = 1;
  while (n2 < bp) n2 <<= 1;
  const int32_t* sel = sel_idx + ((size_t)p * h_kv + g) * budget;
  for (int i = threadIdx.x; i < n2; i += kThreads) srt[i] = i < bp ? sel[i] : INT_MAX;
  __syncthreads();
  sort_positions(srt, n2, threadIdx.x, kThreads);
  copy_kept_rows(k, v, srt, bp, keep_tail, L, row_vecs,
                 ((size_t)tok_off[p] * h_kv + (size_t)g * L) * row_vecs,
                 ((size_t)p * h_kv + g) * out_rows * row_vecs, k_out, v_out, threadIdx.x, kThreads);
}

hipError_t launch_compact(const Shape& s, const void* k, const void* v, const int32_t* sel_idx,
                          int budget, const int32_t* budgets, int keep_tail, int out_rows,
                          void* k_out, void* v_out, hipStream_t stream) {
  if (budget > kMaxSortedBudget) return hipErrorInvalidValue;
  const int elem = s.dtype == kDtBf16 ? 2 : 4;
  const int row_vecs = s.d * elem / 16;
  compact_kernel<<<dim3((unsigned)(s.n_prob * s.h_kv)), kThreads, 0, stream>>>(
      static_cast<const uint4*>(k), static_cast<const uint4*>(v), sel_idx, s.lens, s.tok_off,
      s.h_kv, row_vecs, budget, budgets, keep_tail, out_rows, static_cast<uint4*>(k_out),
      static_cast<uint4*>(v_out));
  return hipGetLastError();
}

}  // namespace kv
