// Both streaming passes in one launch when units span several segments (section 3.1, Eq. (1);
// section 3.2, Eq. (3)).  The per-segment loops are in stream_passes.h, the key stream in
// stream_common.h.
#include "stream_passes.h"

namespace kv {
namespace stream {
namespace {

// ------------------------------------------------------------------------------------------------
// Units split over several segments, one launch: every workgroup runs pass 1 over its segment,
// publishes the segment's (m, z) per row and raises its unit's arrival counter, issues pass 2's
// first tile loads, and waits (a bounded poll) until every segment of the unit has arrived; then it
// merges the unit's partials into the normalisers and runs pass 2 over the same segment, with the
// queries still in registers.  Nothing assumes that all workgroups are resident at once: a
// workgroup whose poll runs out computes the partials of the unit's other segments itself (the
// same code over the same keys, hence the same values, written to the same slots) and goes on,
// so a launch that shares the chip with other work is slower, never wrong or stuck.
// ------------------------------------------------------------------------------------------------
__device__ __forceinline__ void store_partial(float2* dst, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(dst), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_partial(const float2* src) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const uint64_t*>(src),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

// In base-score mode (SC) pass 2 stores each key's base score instead of mu and sigma (see
// stream_window.hip).
template <int D, int NB, bool ALL, int NW, int S, bool SC>
__global__ __launch_bounds__(NW * 64, 1) void window_coop_kernel(StreamArgs a, uint32_t* arrive,
                                                                 uint32_t spin_limit) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS, NT = NW * 64, P = NT / R;
  __shared__ __align__(16) uint16_t ring[NW][S * Gm::TE];
  __shared__ float2 red[NW][R];
  __shared__ float2 mz_part[P][R];
  __shared__ __align__(16) float bsh[R];
  __shared__ uint32_t all_arrived;

  const int seg = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int L = a.lens[p];
  const int k0 = seg * a.seg_keys;
  if (k0 >= L) return;  // not one of this unit's segments (it never counts as one)
  const int k1 = min(k0 + a.seg_keys, L);
  const int n_seg = (L + a.seg_keys - 1) / a.seg_keys;
  const int G = a.h_q / a.h_kv;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float c = a.c;
  const float inv_g = 1.f / (float)G;
  const size_t unit = (size_t)p * a.h_kv + g;
  const size_t stat_base = (size_t)a.tok_off[p] * a.h_kv + (size_t)g * L;
  const uint16_t* kg = a.k + stat_base * D;
  float2* part_u = a.part + unit * a.max_segs * R;
  auto tiles_of = [&](int s0, int s1) {
    const int n_tiles = (s1 - s0 + kTileKeys - 1) / kTileKeys;
    return n_tiles > wave ? (n_tiles - wave + NW - 1) / NW : 0;
  };

  KeyStream<D, NB, NW, S> ks{ring[wave], kg, k0, k1, wave, lane};
  const int my_tiles = tiles_of(k0, k1);

  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  ks.prologue(my_tiles);
  hold_until_loaded<D, NB>(q);

  // pass 1 over segment `sg` (keys [s0, s1)) by the whole workgroup; its partial goes to its slot
  // with device-coherent stores, complete before the workgroup leaves the final barrier
  auto pass1 = [&](const KeyStream<D, NB, NW, S>& st, int sg, int s1, int n_my) {
    float m_run[NB], z_run[NB];
    stats_tiles<D, NB, NW, S>(st, q, n_my, s1, L, c, l32, half, m_run, z_run);
    stats_to_lds<NB>(m_run, z_run, red[wave], l32, half);
    __syncthreads();
    if (threadIdx.x < R) store_partial(part_u + (size_t)sg * R + threadIdx.x, merge_waves<NW, R>(&red[0][0], threadIdx.x));
    wait_vmem<0>();
    __syncthreads();  // red is free again, every partial store has completed
  };
  pass1(ks, seg, k1, my_tiles);
  // The partials and the counter are device-coherent atomics (no cache-wide write-back or
  // invalidation, which would disturb every workgroup streaming keys through the same L2).
  if (threadIdx.x == 0)
    __hip_atomic_fetch_add(arrive + unit, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // the ring is free (pass 1's last wait covered all its loads): pass 2's first tiles load while
  // the other segments arrive
  ks.prologue(my_tiles);
  if (threadIdx.x == 0) {
    uint32_t spins = 0, n = 0;
    while ((n = __hip_atomic_load(arrive + unit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) < (uint32_t)n_seg &&
           spins < spin_limit) {
      __builtin_amdgcn_s_sleep(1);
      ++spins;
    }
    all_arrived = n >= (uint32_t)n_seg ? 1u : 0u;
  }
  __syncthreads();
  if (!all_arrived) {
    // Not every segment arrived in time: the other segments' partials are computed here.
    wait_vmem<0>();  // pass 2's prologue loads own the ring until they land
    for (int sg = 0; sg < n_seg; ++sg) {
      if (sg == seg) continue;
      const int s0 = sg * a.seg_keys, s1 = min(s0 + a.seg_keys, L);
      KeyStream<D, NB, NW, S> other{ring[wave], kg, s0, s1, wave, lane};
      const int n_my = tiles_of(s0, s1);
      other.prologue(n_my);
      pass1(other, sg, s1, n_my);
    }
    ks.prologue(my_tiles);
  }
  // normalisers: thread (row, part) merges segments part, part + P, ... of its row (partials read
  // with device-coherent loads), then one thread per row merges the P results in a fixed order
  // (the same order as the two-launch path)
  {
    const int row = threadIdx.x % R, pt = threadIdx.x / R;
    float M = -INFINITY, Z = 0.f;
    for (int q0 = pt; q0 < n_seg; q0 += 4 * P) {
      float2 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int qq = q0 + u * P;
        v[u] = qq < n_seg ? load_partial(part_u + (size_t)qq * R + row) : make_float2(-INFINITY, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) merge_mz(M, Z, v[u].x, v[u].y);
    }
    mz_part[pt][row] = make_float2(M, Z);
  }
  __syncthreads();
  if (threadIdx.x < R) {
    float M = mz_part[0][threadIdx.x].x, Z = mz_part[0][threadIdx.x].y;
#pragma unroll
    for (int pt = 1; pt < P; ++pt) merge_mz(M, Z, mz_part[pt][threadIdx.x].x, mz_part[pt][threadIdx.x].y);
    bsh[threadIdx.x] = M + __builtin_log2f(Z);
    if (seg == 0) {
      const size_t ri = ((size_t)p * a.h_q + (size_t)g * G) * 32 + threadIdx.x;
      a.row_max_out[ri] = M * kLn2;
      a.row_sum_out[ri] = Z;
    }
  }
  __syncthreads();
  if constexpr (SC) {
    const ScoreOut so{a.score + stat_base, a.lambda1[p], a.w_mu};
    mu_sigma_tiles<D, NB, ALL, NW, S, kOutScore>(ks, q, bsh, my_tiles, k1, L, c, inv_g, nullptr, nullptr,
                                            l32, half, so);
  } else {
    mu_sigma_tiles<D, NB, ALL, NW, S>(ks, q, bsh, my_tiles, k1, L, c, inv_g, a.mu + stat_base,
                                      a.sigma + stat_base, l32, half);
  }
  wait_vmem<0>();  // no load into the ring may outlive the workgroup
}

__global__ void zero_words_kernel(uint32_t* w, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) w[i] = 0u;
}

// One launch of window_coop_kernel after its counters are cleared.  Used when the whole grid fits
// the chip at once (then no workgroup normally waits long); `launched` tells the caller whether it
// ran.
template <int D, int NB> struct CoopLaunch {
  template <bool ALL, bool SC> static const void* kernel() {
    return reinterpret_cast<const void*>(window_coop_kernel<D, NB, ALL, kWaves, 2, SC>);
  }
  static hipError_t run(const Shape& s, StreamArgs args, uint32_t* arrive, uint32_t spin_limit,
                        hipStream_t st, bool* launched) {
    const bool sc = args.score != nullptr;
    const void* kern = args.sigma_all ? (sc ? kernel<true, true>() : kernel<true, false>())
                                      : (sc ? kernel<false, true>() : kernel<false, false>());
    int dev = 0, n_cu = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, kThreads, 0);
    if (e != hipSuccess) return e;
    const dim3 grid(args.max_segs, s.h_kv, s.n_prob);
    if ((int64_t)grid.x * grid.y * grid.z > (int64_t)per_cu * n_cu) {
      *launched = false;
      return hipSuccess;
    }
    const int n_units = s.n_prob * s.h_kv;
    zero_words_kernel<<<(n_units + 255) / 256, 256, 0, st>>>(arrive, n_units);
    if (args.sigma_all) {
      if (sc) window_coop_kernel<D, NB, true, kWaves, 2, true><<<grid, kThreads, 0, st>>>(args, arrive, spin_limit);
      else window_coop_kernel<D, NB, true, kWaves, 2, false><<<grid, kThreads, 0, st>>>(args, arrive, spin_limit);
    } else {
      if (sc) window_coop_kernel<D, NB, false, kWaves, 2, true><<<grid, kThreads, 0, st>>>(args, arrive, spin_limit);
      else window_coop_kernel<D, NB, false, kWaves, 2, false><<<grid, kThreads, 0, st>>>(args, arrive, spin_limit);
    }
    e = hipGetLastError();
    *launched = e == hipSuccess;
    return e;
  }
};

}  // namespace
}  // namespace stream

hipError_t launch_stream_window_coop(const Shape& s, const StreamPlan& plan, const void* q_win,
                                     const void* k, float scale, void* ws, float* row_max,
                                     float* row_sum, float* mu, float* sigma, bool sigma_all,
                                     uint32_t spin_limit, hipStream_t stream, bool* launched,
                                     const ScoreMode* sm) {
  *launched = false;
  stream::StreamArgs a = stream::base_args(s, plan, q_win, k, scale);
  a.part = static_cast<float2*>(ws);
  a.row_max_out = row_max;
  a.row_sum_out = row_sum;
  a.mu = mu;
  a.sigma = sigma;
  a.sigma_all = sigma_all ? 1 : 0;
  if (sm) {
    a.score = sm->score;
    a.lambda1 = sm->lambda1;
    a.w_mu = sm->w_mu;
  }
  uint32_t* arrive = reinterpret_cast<uint32_t*>(static_cast<char*>(ws) + stream_counter_offset(s, plan));
  const int G = s.group();
  using namespace stream;
  if (s.d == 128) {
    if (G == 4) return CoopLaunch<128, 4>::run(s, a, arrive, spin_limit, stream, launched);
    if (G == 2) return CoopLaunch<128, 2>::run(s, a, arrive, spin_limit, stream, launched);
    return CoopLaunch<128, 1>::run(s, a, arrive, spin_limit, stream, launched);
  }
  if (G == 4) return CoopLaunch<64, 4>::run(s, a, arrive, spin_limit, stream, launched);
  if (G == 2) return CoopLaunch<64, 2>::run(s, a, arrive, spin_limit, stream, launched);
  return CoopLaunch<64, 1>::run(s, a, arrive, spin_limit, stream, launched);
}

}  // namespace kv
