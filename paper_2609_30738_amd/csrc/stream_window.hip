// Both streaming passes over one whole unit in one workgroup (section 3.1, Eq. (1); section 3.2,
// Eq. (3)), for launches in which every (problem, kv head) unit is a single segment.  The unit's
// row statistics are complete when its own pass 1 ends, so its pass 2 follows at once, with the
// queries still in registers and the first key tiles of pass 2 loaded while the waves' statistics
// are merged; no workgroup waits for any other.  The per-segment loops are in stream_passes.h.
//
// In base-score mode (OUT = kOutScore) pass 2 keeps mu and sigma in registers and stores only
// each key's base score (section 3.2, Eq. (5)): half the bytes, which trickle out between the key
// loads of a stream that keeps HBM busy, and the selection reads one array instead of two.  The
// candidate mode, which stores nothing per key, has its own kernel (stream_prune.hip).
#include "stream_passes.h"

namespace kv {
namespace stream {
namespace {

template <int D, int NB, bool ALL, int NW, int S, int OUT>
__global__ __launch_bounds__(NW * 64, 1) void window_stream_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS;
  static_assert(OUT != kOutCand, "candidate mode: stream_prune.hip");
  __shared__ __align__(16) uint16_t ring[NW][S * Gm::TE];
  __shared__ float2 red[NW][R];
  __shared__ __align__(16) float bsh[R];

  const int g = blockIdx.y, p = blockIdx.z;
  const int L = a.lens[p];
  const int G = a.h_q / a.h_kv;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float c = a.c;
  const float inv_g = 1.f / (float)G;
  const size_t stat_base = (size_t)a.tok_off[p] * a.h_kv + (size_t)g * L;

  KeyStream<D, NB, NW, S> ks{ring[wave], a.k + stat_base * D, 0, L, wave, lane};
  const int n_tiles = (L + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + NW - 1) / NW : 0;
  // the query loads go first: vector memory operations complete in issue order, so the waits on
  // key tiles below also cover them
  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  ks.prologue(my_tiles);
  hold_until_loaded<D, NB>(q);

  float m_run[NB], z_run[NB];
  stats_tiles<D, NB, NW, S>(ks, q, my_tiles, L, L, c, l32, half, m_run, z_run);
  // every load of pass 1 has landed and been read (its last wait is vmcnt(0)): the ring takes the
  // first tiles of pass 2 while the statistics are merged
  ks.prologue(my_tiles);
  stats_to_lds<NB>(m_run, z_run, red[wave], l32, half);
  __syncthreads();
  if (threadIdx.x < R) {
    const float2 v = merge_waves<NW, R>(&red[0][0], threadIdx.x);
    bsh[threadIdx.x] = v.x + __builtin_log2f(v.y);  // b = M + log2 Z, base 2
  }
  __syncthreads();
  if constexpr (OUT == kOutScore) {
    const ScoreOut so{a.score + stat_base, a.lambda1[p], a.w_mu};
    mu_sigma_tiles<D, NB, ALL, NW, S, kOutScore>(ks, q, bsh, my_tiles, L, L, c, inv_g, nullptr,
                                                 nullptr, l32, half, so);
  } else {
    mu_sigma_tiles<D, NB, ALL, NW, S>(ks, q, bsh, my_tiles, L, L, c, inv_g, a.mu + stat_base,
                                      a.sigma + stat_base, l32, half);
  }
  wait_vmem<0>();  // no load into the ring may outlive the workgroup
  // the row statistics, merged again from the same entries in the same order
  if (threadIdx.x < R) {
    const float2 v = merge_waves<NW, R>(&red[0][0], threadIdx.x);
    const size_t ri = ((size_t)p * a.h_q + (size_t)g * G) * 32 + threadIdx.x;
    a.row_max_out[ri] = v.x * kLn2;
    a.row_sum_out[ri] = v.y;
  }
}

template <int D, int NB> struct WindowLaunch {
  static hipError_t run(const Shape& s, const StreamArgs& args, hipStream_t st) {
    const dim3 grid(1, s.h_kv, s.n_prob);
    if (args.score) {
      if (args.sigma_all) window_stream_kernel<D, NB, true, kWaves, 2, kOutScore><<<grid, kThreads, 0, st>>>(args);
      else window_stream_kernel<D, NB, false, kWaves, 2, kOutScore><<<grid, kThreads, 0, st>>>(args);
    } else {
      if (args.sigma_all) window_stream_kernel<D, NB, true, kWaves, 2, kOutMuSigma><<<grid, kThreads, 0, st>>>(args);
      else window_stream_kernel<D, NB, false, kWaves, 2, kOutMuSigma><<<grid, kThreads, 0, st>>>(args);
    }
    return hipGetLastError();
  }
};

}  // namespace
}  // namespace stream

hipError_t launch_stream_window(const Shape& s, const StreamPlan& plan, const void* q_win,
                                const void* k, float scale, float* row_max, float* row_sum,
                                float* mu, float* sigma, bool sigma_all, hipStream_t stream) {
  if (plan.max_segs != 1) return hipErrorInvalidValue;  // a unit must be one segment
  stream::StreamArgs a = stream::base_args(s, plan, q_win, k, scale);
  a.row_max_out = row_max;
  a.row_sum_out = row_sum;
  a.mu = mu;
  a.sigma = sigma;
  a.sigma_all = sigma_all ? 1 : 0;
  return stream::launch_for_shape<stream::WindowLaunch>(s, a, stream);
}

hipError_t launch_stream_window_scores(const Shape& s, const StreamPlan& plan, const void* q_win,
                                       const void* k, float scale, const float* lambda1,
                                       float w_mu, float* row_max, float* row_sum, float* score,
                                       bool sigma_all, hipStream_t stream) {
  if (plan.max_segs != 1 || !score) return hipErrorInvalidValue;
  stream::StreamArgs a = stream::base_args(s, plan, q_win, k, scale);
  a.row_max_out = row_max;
  a.row_sum_out = row_sum;
  a.sigma_all = sigma_all ? 1 : 0;
  a.score = score;
  a.lambda1 = lambda1;
  a.w_mu = w_mu;
  return stream::launch_for_shape<stream::WindowLaunch>(s, a, stream);
}

}  // namespace kv
