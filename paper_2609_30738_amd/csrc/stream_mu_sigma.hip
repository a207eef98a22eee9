// Streaming window statistics, pass 2 (section 3.1 Eq. (1), section 3.2 Eq. (3)): the row
// normalisers of a unit from the pass-1 partials, then per key the group-mean attention of the
// window rows, its mean mu and sample standard deviation sigma.  The design shared with pass 1 is
// described in stream_common.h.
#include "stream_passes.h"

namespace kv {
namespace stream {
namespace {

// ------------------------------------------------------------------------------------------------
// Pass 2
// ------------------------------------------------------------------------------------------------
template <int D, int NB, bool ALL, int NW, int S>
__global__ __launch_bounds__(NW * 64, 1) void mu_sigma_stream_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS, NT = NW * 64;
  __shared__ __align__(16) uint16_t ring[NW][S * Gm::TE];
  __shared__ __align__(16) float bsh[R];
  __shared__ float2 mz_part[NT / R][R];

  const int seg = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int L = a.lens[p];
  const int k0 = seg * a.seg_keys;
  if (k0 >= L) return;
  const int k1 = min(k0 + a.seg_keys, L);
  const int G = a.h_q / a.h_kv;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float c = a.c;
  const float inv_g = 1.f / (float)G;

  KeyStream<D, NB, NW, S> ks{ring[wave], a.k + ((size_t)a.tok_off[p] * a.h_kv + (size_t)g * L) * D,
                             k0, k1, wave, lane};
  const int n_tiles = (k1 - k0 + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + NW - 1) / NW : 0;
  // the query loads go first: vector memory operations complete in issue order, so the waits on
  // key tiles below also cover them
  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  ks.prologue(my_tiles);
  hold_until_loaded<D, NB>(q);

  // Normalisers of the unit's rows.  From segment partials: thread (row, part) merges segments
  // part, part + P, ... of its row (four loads in flight), then one thread per row merges the P
  // results in a fixed order.
  constexpr int P = NT / R;
  const size_t ri0 = ((size_t)p * a.h_q + (size_t)g * G) * 32;
  if (a.part) {
    const int n_seg = (L + a.seg_keys - 1) / a.seg_keys;
    const int row = threadIdx.x % R, pt = threadIdx.x / R;
    const float2* src = a.part + ((size_t)p * a.h_kv + g) * a.max_segs * R + row;
    float M = -INFINITY, Z = 0.f;
    for (int q0 = pt; q0 < n_seg; q0 += 4 * P) {
      float2 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int qq = q0 + u * P;
        v[u] = qq < n_seg ? src[(size_t)qq * R] : make_float2(-INFINITY, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) merge_mz(M, Z, v[u].x, v[u].y);
    }
    mz_part[pt][row] = make_float2(M, Z);
  }
  __syncthreads();
  if (threadIdx.x < R) {
    const size_t ri = ri0 + threadIdx.x;
    float bv;
    if (a.part) {
      float M = mz_part[0][threadIdx.x].x, Z = mz_part[0][threadIdx.x].y;
#pragma unroll
      for (int pt = 1; pt < P; ++pt) merge_mz(M, Z, mz_part[pt][threadIdx.x].x, mz_part[pt][threadIdx.x].y);
      bv = M + __builtin_log2f(Z);
      if (seg == 0) {
        a.row_max_out[ri] = M * kLn2;
        a.row_sum_out[ri] = Z;
      }
    } else {
      bv = a.row_max[ri] * kLog2e + __builtin_log2f(a.row_sum[ri]);
    }
    bsh[threadIdx.x] = bv;
  }
  __syncthreads();
  const size_t stat_base = (size_t)a.tok_off[p] * a.h_kv + (size_t)g * L;
  mu_sigma_tiles<D, NB, ALL, NW, S>(ks, q, bsh, my_tiles, k1, L, c, inv_g, a.mu + stat_base,
                                    a.sigma + stat_base, l32, half);
  wait_vmem<0>();  // no load into the ring may outlive the workgroup
}

template <int D, int NB> struct MuSigmaLaunch {
  static hipError_t run(const Shape& s, const StreamArgs& args, hipStream_t st) {
    // eight waves (two per SIMD), two-tile rings (measured: one wave per SIMD with four-tile rings
    // runs this pass 20 % slower)
    const dim3 grid(args.max_segs, s.h_kv, s.n_prob);
    if (args.sigma_all) mu_sigma_stream_kernel<D, NB, true, kWaves, 2><<<grid, kThreads, 0, st>>>(args);
    else mu_sigma_stream_kernel<D, NB, false, kWaves, 2><<<grid, kThreads, 0, st>>>(args);
    return hipGetLastError();
  }
};

}  // namespace
}  // namespace stream

hipError_t launch_stream_mu_sigma(const Shape& s, const StreamPlan& plan, const void* q_win,
                                  const void* k, float scale, const void* ws,
                                  const float* row_max_in, const float* row_sum_in,
                                  float* row_max_out, float* row_sum_out, float* mu, float* sigma,
                                  bool sigma_all, hipStream_t stream) {
  stream::StreamArgs a = stream::base_args(s, plan, q_win, k, scale);
  a.part = const_cast<float2*>(static_cast<const float2*>(ws));
  a.row_max = row_max_in;
  a.row_sum = row_sum_in;
  a.row_max_out = row_max_out;
  a.row_sum_out = row_sum_out;
  a.mu = mu;
  a.sigma = sigma;
  a.sigma_all = sigma_all ? 1 : 0;
  return stream::launch_for_shape<stream::MuSigmaLaunch>(s, a, stream);
}

}  // namespace kv