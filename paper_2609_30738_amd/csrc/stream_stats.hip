// Streaming window statistics, pass 1 (section 3.1): per segment of a unit's keys, the running
// maximum and the sum of exponentials of every window row's logits.  The design shared with pass 2
// is described in stream_common.h.
#include "stream_passes.h"

namespace kv {
namespace stream {
namespace {

// ------------------------------------------------------------------------------------------------
// Pass 1
// ------------------------------------------------------------------------------------------------
template <int D, int NB, int NW, int S>
__global__ __launch_bounds__(NW * 64, 1) void stats_stream_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS;
  __shared__ __align__(16) uint16_t ring[NW][S * Gm::TE];
  __shared__ float2 red[NW][R];

  const int seg = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int L = a.lens[p];
  const int k0 = seg * a.seg_keys;
  if (k0 >= L) return;
  const int k1 = min(k0 + a.seg_keys, L);
  const int G = a.h_q / a.h_kv;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float c = a.c;

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

  float m_run[NB], z_run[NB];
  stats_tiles<D, NB, NW, S>(ks, q, my_tiles, k1, L, c, l32, half, m_run, z_run);
  wait_vmem<0>();  // no load into the ring may outlive the workgroup

  stats_to_lds<NB>(m_run, z_run, red[wave], l32, half);
  __syncthreads();
  if (threadIdx.x < R) {
    const float2 v = merge_waves<NW, R>(&red[0][0], threadIdx.x);
    if (a.part) {
      a.part[(((size_t)p * a.h_kv + g) * a.max_segs + seg) * R + threadIdx.x] = v;
    } else {  // every unit is one segment: the row statistics themselves
      const size_t ri = ((size_t)p * a.h_q + (size_t)g * G) * 32 + threadIdx.x;
      a.row_max_out[ri] = v.x * kLn2;
      a.row_sum_out[ri] = v.y;
    }
  }
}

template <int D, int NB> struct StatsLaunch {
  static hipError_t run(const Shape& s, const StreamArgs& args, hipStream_t st) {
    const dim3 grid(args.max_segs, s.h_kv, s.n_prob);
    stats_stream_kernel<D, NB, kWaves, 2><<<grid, kThreads, 0, st>>>(args);
    return hipGetLastError();
  }
};

}  // namespace
}  // namespace stream

hipError_t launch_stream_stats(const Shape& s, const StreamPlan& plan, const void* q_win,
                               const void* k, float scale, void* ws, float* row_max,
                               float* row_sum, hipStream_t stream) {
  stream::StreamArgs a = stream::base_args(s, plan, q_win, k, scale);
  a.part = static_cast<float2*>(ws);
  a.row_max_out = row_max;
  a.row_sum_out = row_sum;
  return stream::launch_for_shape<stream::StatsLaunch>(s, a, stream);
}

}  // namespace kv
