// Cache compaction steps shared by the compaction kernel (compact.hip) and the selection kernel's
// optional compaction epilogue (select.hip): the B_p admitted positions of a unit sorted in LDS,
// then the kept rows of K and V, followed by the always-kept tail, copied with 16-byte vectors
// (sections 1 and 3.1: each layer keeps B entries plus the window).
#pragma once

#include <limits.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

namespace kv {

// Ascending bitonic sort of srt[0, n2) (n2 a power of two) by the nt threads of the workgroup;
// the caller has filled srt (padding with INT_MAX) and synchronised.  Ends synchronised.
__device__ __forceinline__ void sort_positions(int32_t* srt, int n2, int tid, int nt) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < n2; i += nt) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const int a = srt[i], b = srt[j];
          if ((a > b) == up) {
            srt[i] = b;
            srt[j] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

// Rows 0 .. bp + keep_tail - 1 of the unit's output block: the sorted positions srt[0, bp), then
// the last keep_tail positions of the unit.  src / dst are the unit's first 16-byte vectors.
__device__ __forceinline__ void copy_kept_rows(const uint4* __restrict__ k, const uint4* __restrict__ v,
                                               const int32_t* srt, int bp, int keep_tail, int L,
                                               int row_vecs, size_t src, size_t dst,
                                               uint4* __restrict__ k_out, uint4* __restrict__ v_out,
                                               int tid, int nt) {
  const int rows = bp + keep_tail;
  for (int e = tid; e < rows * row_vecs; e += nt) {
    const int r = e / row_vecs, c = e % row_vecs;
    const int pos = r < bp ? srt[r] : L - keep_tail + (r - bp);
    if (pos < 0 || pos >= L) continue;  // invalid selection: leave the row unwritten
    const size_t s = src + (size_t)pos * row_vecs + c;
    k_out[dst + e] = k[s];
    v_out[dst + e] = v[s];
  }
}

}  // namespace kv
