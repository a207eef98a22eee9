// Attention of one generated token per (sequence, layer) over its compacted cache (section 4.3:
// after eviction the model generates against the kept B + W rows of every layer).
//
// decode_kernel: one workgroup of 256 threads per (split of the rows, kv head, problem).  A row of
//   d elements is CH 16-byte chunks; thread t takes chunk t % CH of rows t / CH, t / CH + RPP, ...
//   (RPP = 256 / CH rows per pass), so a pass reads RPP whole consecutive rows of K and of V.  The
//   G query heads of the kv head share every loaded row.  Per row, the chunk dot products are summed
//   over the CH lanes of the row with butterfly shuffles, and every lane keeps a base-2 online
//   softmax (running max, sum, and the weighted sum of its value chunk) per head.  At the end the
//   row groups of a wave are merged with shuffles and the four waves through LDS.  With one split
//   the normalised output is written; with several, a partial (max, sum, weighted values) per
//   (head, split) goes to the workspace and decode_combine_kernel merges the splits.
//   If the token's own key / value are given, the split that holds row `len` attends to them from
//   the inputs and also writes them into row `len` of the cache block.
#include <math.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kUnroll = 4;  // rows per thread loaded before any of them is used

__device__ __forceinline__ void chunk_to_f32(const uint4& u, float (&f)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void chunk_to_f32(const uint4& u, float (&f)[4]) {
  f[0] = __uint_as_float(u.x);
  f[1] = __uint_as_float(u.y);
  f[2] = __uint_as_float(u.z);
  f[3] = __uint_as_float(u.w);
}

}  // namespace

template <int DT, int D, int GM>
__global__ __launch_bounds__(kThreads) void decode_kernel(DecodeArgs a) {
  using T = typename Elem<DT>::T;
  constexpr int EPT = 16 / (int)sizeof(T);  // elements of a 16-byte chunk
  constexpr int CH = D / EPT;               // chunks of a row
  constexpr int RPP = kThreads / CH;        // rows per pass
  static_assert(CH <= 64 && 64 % CH == 0, "a row's chunks sit in one wave");
  __shared__ float sh_m[kWaves][GM];
  __shared__ float sh_s[kWaves][GM];
  __shared__ float sh_acc[kWaves][GM][D];

  const int split = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int G = a.h_q / a.h_kv;
  const int len = a.lens[p];
  const bool append = a.k_new != nullptr;
  const int total = len + (append ? 1 : 0);
  const int r0 = split * a.split_rows;
  const int r1 = min(total, r0 + a.split_rows);
  const int rc = min(len, r1);  // rows of this split that come from the cache
  const int tid = threadIdx.x, rg = tid / CH, c = tid % CH, wave = tid / 64, lane = tid % 64;

  const size_t unit = (size_t)p * a.h_kv + g;
  const uint4* kc = static_cast<const uint4*>(a.k) + unit * a.row_stride * CH + c;
  const uint4* vc = static_cast<const uint4*>(a.v) + unit * a.row_stride * CH + c;
  const uint4* kn = append ? static_cast<const uint4*>(a.k_new) + unit * CH + c : nullptr;
  const uint4* vn = append ? static_cast<const uint4*>(a.v_new) + unit * CH + c : nullptr;

  // the query chunks of the group's heads, scaled so that logits come out in base 2
  float qf[GM][EPT];
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    uint4 u = make_uint4(0u, 0u, 0u, 0u);
    if (h < G) u = static_cast<const uint4*>(a.q)[((size_t)p * a.h_q + (size_t)g * G + h) * CH + c];
    chunk_to_f32(u, qf[h]);
#pragma unroll
    for (int e = 0; e < EPT; ++e) qf[h][e] *= a.c;
  }
  if (append && len >= r0 && len < r1 && rg == 0) {  // the new row joins the cache
    static_cast<uint4*>(a.k)[(unit * a.row_stride + len) * CH + c] = *kn;
    static_cast<uint4*>(a.v)[(unit * a.row_stride + len) * CH + c] = *vn;
  }

  float m[GM], s[GM], acc[GM][EPT];
#pragma unroll
  for (int h = 0; h < GM; ++h) {
    m[h] = -INFINITY;
    s[h] = 0.f;
#pragma unroll
    for (int e = 0; e < EPT; ++e) acc[h][e] = 0.f;
  }

  // the same trip count on every lane: the row sums shuffle within each row's lanes
  for (int rb = r0; rb < r1; rb += kUnroll * RPP) {
    uint4 ku[kUnroll], vu[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int r = rb + u * RPP + rg;
      ku[u] = vu[u] = make_uint4(0u, 0u, 0u, 0u);
      if (r < rc) {
        ku[u] = kc[(size_t)r * CH];
        vu[u] = vc[(size_t)r * CH];
      } else if (r < r1) {  // r == len: the appended row
        ku[u] = *kn;
        vu[u] = *vn;
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int r = rb + u * RPP + rg;
      float kf[EPT], vf[EPT];
      chunk_to_f32(ku[u], kf);
      chunk_to_f32(vu[u], vf);
#pragma unroll
      for (int h = 0; h < GM; ++h) {
        float t = 0.f;
#pragma unroll
        for (int e = 0; e < EPT; ++e) t = fmaf(qf[h][e], kf[e], t);
#pragma unroll
        for (int off = CH / 2; off > 0; off >>= 1) t += __shfl_xor(t, off);
        if (r < r1 && h < G) {
          const float mn = fmaxf(m[h], t);
          const float al = __builtin_amdgcn_exp2f(m[h] - mn);  // 0 while m = -inf
          const float be = __builtin_amdgcn_exp2f(t - mn);
          s[h] = fmaf(s[h], al, be);
#pragma unroll
          for (int e = 0; e < EPT; ++e) acc[h][e] = fmaf(acc[h][e], al, be * vf[e]);
          m[h] = mn;
        }
      }
    }
  }

  // merge the row groups of each wave (lanes c, c + CH, c + 2 CH, ... hold the same chunk)
#pragma unroll
  for (int off = CH; off < 64; off <<= 1) {
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      const float mo = __shfl_xor(m[h], off), so = __shfl_xor(s[h], off);
      const float mn = fmaxf(m[h], mo);
      const float f = m[h] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m[h] - mn);
      const float fo = mo == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mo - mn);
      s[h] = s[h] * f + so * fo;
#pragma unroll
      for (int e = 0; e < EPT; ++e) acc[h][e] = acc[h][e] * f + __shfl_xor(acc[h][e], off) * fo;
      m[h] = mn;
    }
  }
  if (lane < CH) {
#pragma unroll
    for (int h = 0; h < GM; ++h) {
      if (c == 0) {
        sh_m[wave][h] = m[h];
        sh_s[wave][h] = s[h];
      }
#pragma unroll
      for (int e = 0; e < EPT; ++e) sh_acc[wave][h][c * EPT + e] = acc[h][e];
    }
  }
  __syncthreads();
  for (int idx = tid; idx < G * D; idx += kThreads) {
    const int h = idx / D, e = idx % D;
    float M = -INFINITY;
    for (int i = 0; i < kWaves; ++i) M = fmaxf(M, sh_m[i][h]);
    float S = 0.f, A = 0.f;
    for (int i = 0; i < kWaves; ++i) {
      const float mi = sh_m[i][h];
      const float f = mi == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mi - M);
      S = fmaf(sh_s[i][h], f, S);
      A = fmaf(sh_acc[i][h][e], f, A);
    }
    const size_t row = (size_t)p * a.h_q + (size_t)g * G + h;
    if (a.n_split == 1) {
      a.out[row * D + e] = A / S;
    } else {
      float* pt = a.part + (row * a.n_split + split) * (D + 2);
      if (e == 0) {
        pt[0] = M;
        pt[1] = S;
      }
      pt[2 + e] = A;
    }
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void decode_combine_kernel(const float* __restrict__ part,
                                                                  int rows, int n_split,
                                                                  float* __restrict__ out) {
  const int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (idx >= (int64_t)rows * D) return;
  const int64_t row = idx / D;
  const int e = (int)(idx % D);
  const float* pt = part + row * n_split * (D + 2);
  float M = -INFINITY;
  for (int i = 0; i < n_split; ++i) M = fmaxf(M, pt[i * (D + 2)]);
  float S = 0.f, A = 0.f;
  for (int i = 0; i < n_split; ++i) {
    const float mi = pt[i * (D + 2)];
    const float f = mi == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mi - M);
    S = fmaf(pt[i * (D + 2) + 1], f, S);
    A = fmaf(pt[i * (D + 2) + 2 + e], f, A);
  }
  out[idx] = A / S;
}

namespace {

template <int DT, int D>
hipError_t decode_dispatch(const DecodeArgs& a, int n_prob, hipStream_t st) {
  const dim3 grid((unsigned)a.n_split, (unsigned)a.h_kv, (unsigned)n_prob);
  const int G = a.h_q / a.h_kv;
  if (G == 1) decode_kernel<DT, D, 1><<<grid, kThreads, 0, st>>>(a);
  else if (G == 2) decode_kernel<DT, D, 2><<<grid, kThreads, 0, st>>>(a);
  else if (G <= 4) decode_kernel<DT, D, 4><<<grid, kThreads, 0, st>>>(a);
  else decode_kernel<DT, D, 8><<<grid, kThreads, 0, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_split == 1) return e;
  const int rows = n_prob * a.h_q;
  const int64_t n = (int64_t)rows * D;
  decode_combine_kernel<D><<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, st>>>(
      a.part, rows, a.n_split, a.out);
  return hipGetLastError();
}

}  // namespace

DecodePlan decode_plan(int n_prob, int h_kv, int max_len) {
  // one workgroup per unit while there are enough units or the rows are few; otherwise split the
  // rows so that a launch has about 1024 workgroups, in multiples of 256 rows
  constexpr int64_t kTarget = 1024, kStep = 256;
  const int64_t units = (int64_t)n_prob * h_kv;
  const int64_t rows = (int64_t)max_len + 1;  // room for an appended row
  int64_t n_split = 1;
  if (units < kTarget && rows > 2 * kStep) {
    n_split = std::min<int64_t>((kTarget + units - 1) / units, (rows + kStep - 1) / kStep);
  }
  int64_t split_rows = (rows + n_split - 1) / n_split;
  split_rows = (split_rows + kStep - 1) / kStep * kStep;
  n_split = (rows + split_rows - 1) / split_rows;
  DecodePlan plan;
  plan.n_split = (int)n_split;
  plan.split_rows = (int)split_rows;
  return plan;
}

size_t decode_ws_bytes(int n_prob, int h_q, int d, const DecodePlan& plan) {
  if (plan.n_split == 1) return 0;
  return (size_t)n_prob * h_q * plan.n_split * (d + 2) * sizeof(float);
}

hipError_t launch_decode(int dtype, int d, int n_prob, const DecodeArgs& a, hipStream_t stream) {
  if (dtype == kDtBf16)
    return d == 64 ? decode_dispatch<kDtBf16, 64>(a, n_prob, stream)
                   : decode_dispatch<kDtBf16, 128>(a, n_prob, stream);
  return d == 64 ? decode_dispatch<kDtF32, 64>(a, n_prob, stream)
                 : decode_dispatch<kDtF32, 128>(a, n_prob, stream);
}

}  // namespace kv
