// Streaming window statistics, pass 1 (section 3.1): per segment of a unit's keys, the running
// maximum and the sum of exponentials of every window row's logits.  The design shared with pass 2
// is described in stream_common.h.
#include "stream_common.h"

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
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    m_run[b] = -INFINITY;
    z_run[b] = 0.f;
  }
  // a tile is interior when none of its keys is masked: t0 + 31 < min(k1, L - 31)
  const int kedge = min(k1, L - 31);
  for (int j = 0; j < my_tiles; ++j) {
    bf16x8_t kt[NS];
    ks.template next<0>(kt, j, my_tiles, l32, half);
    const int t0 = ks.tile_key(j);
    if (t0 + 31 < kedge) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16_t d = chain<NS>(kt, q[b]);
        float mx = fmax3(fmax3(fmax3(d[0], d[1], d[2]), d[3], d[4]), d[5], d[6]);
        mx = fmax3(fmax3(mx, d[7], d[8]), d[9], d[10]);
        mx = fmax3(fmax3(mx, d[11], d[12]), d[13], d[14]);
        const float mn = __builtin_elementwise_maximum(m_run[b], __builtin_elementwise_maximum(mx, d[15]) * c);
        const float keep = __builtin_amdgcn_exp2f(m_run[b] - mn);  // 0 on the lane's first tile
        float ex[16];
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) ex[jj] = __builtin_amdgcn_exp2f(fmaf(d[jj], c, -mn));
        float zs[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) zs[u] = (ex[4 * u] + ex[4 * u + 1]) + (ex[4 * u + 2] + ex[4 * u + 3]);
        z_run[b] = fmaf(z_run[b], keep, (zs[0] + zs[1]) + (zs[2] + zs[3]));
        m_run[b] = mn;
      }
    } else {
      // window row l32 of every head sees keys <= L - 32 + l32; keys >= k1 belong to the next
      // segment.  The key of register jj is t0 + 4 half + 8 (jj / 4) + (jj % 4).
      const int thr = min(k1 - 1, L - 32 + l32) - t0 - 4 * half;
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        f32x16_t d = chain<NS>(kt, q[b]);
#pragma unroll
        for (int jj = 0; jj < 16; ++jj)
          if (8 * (jj >> 2) + (jj & 3) > thr) d[jj] = -INFINITY;
        float mx = d[0];
#pragma unroll
        for (int jj = 1; jj < 16; ++jj) mx = fmaxf(mx, d[jj]);
        const float mn = fmaxf(m_run[b], mx * c);
        if (mn != -INFINITY) {
          const float keep = m_run[b] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run[b] - mn);
          float z = z_run[b] * keep;
#pragma unroll
          for (int jj = 0; jj < 16; ++jj) z += __builtin_amdgcn_exp2f(fmaf(d[jj], c, -mn));
          z_run[b] = z;
          m_run[b] = mn;
        }
      }
    }
  }
  wait_vmem<0>();  // no load into the ring may outlive the workgroup

  // lanes l and l ^ 32 hold the same rows (different keys); then the waves
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float m = m_run[b], z = z_run[b];
    merge_mz(m, z, swap_halves(m), swap_halves(z));
    if (half == 0) red[wave][b * 32 + l32] = make_float2(m, z);
  }
  __syncthreads();
  if (threadIdx.x < R) {
    float2 v = red[0][threadIdx.x];
#pragma unroll
    for (int w = 1; w < NW; ++w) merge_mz(v.x, v.y, red[w][threadIdx.x].x, red[w][threadIdx.x].y);
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

bool stream_shape_ok(const Shape& s, float scale) {
  const int G = s.group();
  // pass 1 takes a tile's maximum logit as the scaled maximum of the raw dot products
  return s.dtype == kDtBf16 && s.w == 32 && (s.d == 64 || s.d == 128) &&
         (G == 1 || G == 2 || G == 4) && scale > 0.f;
}

StreamPlan stream_plan(const Shape& s, int64_t total_keys) {
  // about one segment per compute unit (256 on MI355X), whole 256-key steps of the eight waves
  constexpr int64_t kTarget = 256, kStep = stream::kWaves * stream::kTileKeys, kMinSeg = 1024;
  int64_t seg = (total_keys + kTarget - 1) / kTarget;
  seg = std::max<int64_t>(kMinSeg, (seg + kStep - 1) / kStep * kStep);
  seg = std::min<int64_t>(seg, ((int64_t)s.max_len + kStep - 1) / kStep * kStep);
  StreamPlan plan;
  plan.seg_keys = (int)seg;
  plan.max_segs = (int)(((int64_t)s.max_len + seg - 1) / seg);
  return plan;
}

size_t stream_ws_bytes(const Shape& s, const StreamPlan& plan) {
  return (size_t)s.n_prob * s.h_kv * plan.max_segs * s.group() * 32 * sizeof(float2);
}

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
