// Streaming window statistics, pass 2 (section 3.1 Eq. (1), section 3.2 Eq. (3)): the row
// normalisers of a unit from the pass-1 partials, then per key the group-mean attention of the
// window rows, its mean mu and sample standard deviation sigma.  The design shared with pass 1 is
// described in stream_common.h.
#include "stream_common.h"

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
  auto tile = [&](const bf16x8_t (&kt)[NS], int t0, auto masked) __attribute__((always_inline)) {
    const int key = t0 + l32;
    // window row r = 4 half + 8 (j / 4) + (j % 4) of every head sees the key iff key <= L - 32 + r
    const int thr = key - (L - 32) - 4 * half;
    float ab[16];
    float h_mean = 0.f, h_m2 = 0.f;  // ALL: running mean and squared deviations of the heads so far
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      float eb[16];
      const f32x16_t d = chain<NS>(q[b], kt);
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        // window rows 8 qq + 4 half + 0..3 of query head b (read per tile: the registers hold
        // the queries, the tile and the logit blocks)
        const float4 bv = *reinterpret_cast<const float4*>(bsh + b * 32 + 8 * qq + 4 * half);
        const float bb[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int j = 4 * qq + u;
          float e = __builtin_amdgcn_exp2f(fmaf(d[j], c, -bb[u]));
          if (decltype(masked)::value && 8 * qq + u < thr) e = 0.f;
          ab[j] = b == 0 ? e : ab[j] + e;
          eb[j] = e;
        }
      }
      if constexpr (ALL) {
        float hs[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 16; ++j) hs[j & 3] += eb[j];
        const float mb = sum_halves((hs[0] + hs[1]) + (hs[2] + hs[3])) * (1.f / 32.f);
        float hv[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const float dl = eb[j] - mb;
          hv[j & 3] = fmaf(dl, dl, hv[j & 3]);
        }
        const float m2b = sum_halves((hv[0] + hv[1]) + (hv[2] + hv[3]));
        if (b == 0) {
          h_mean = mb;
          h_m2 = m2b;
        } else {  // b heads of 32 rows merged with one more
          const float dl = mb - h_mean;
          h_mean = fmaf(dl, 1.f / (float)(b + 1), h_mean);
          h_m2 += fmaf(dl * dl, 32.f * (float)b / (float)(b + 1), m2b);
        }
      }
    }
    // ab[j] = G a[r][key] for the window rows r = acc_row(j, lane); the other 16 are in lane ^ 32
    float sp[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) sp[u] = (ab[u] + ab[u + 4]) + (ab[u + 8] + ab[u + 12]);
    const float mean = sum_halves((sp[0] + sp[1]) + (sp[2] + sp[3])) * (inv_g * (1.f / 32.f));
    float var;
    if constexpr (ALL) {
      var = h_m2 * (1.f / (float)(NB * 32 - 1));
    } else {
      float vp[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float dl = fmaf(ab[j], inv_g, -mean);
        vp[j & 3] = fmaf(dl, dl, vp[j & 3]);
      }
      var = sum_halves((vp[0] + vp[1]) + (vp[2] + vp[3])) * (1.f / 31.f);
    }
    if (key < k1) (half == 0 ? a.mu : a.sigma)[stat_base + key] = half == 0 ? mean : __builtin_amdgcn_sqrtf(var);
  };

  for (int j = 0; j < my_tiles; ++j) {
    bf16x8_t kt[NS];
    ks.template next<1>(kt, j, my_tiles, l32, half);  // one mu / sigma store per tile
    const int t0 = ks.tile_key(j);
    if (t0 + 31 > L - 32) tile(kt, t0, std::true_type{});
    else tile(kt, t0, std::false_type{});
  }
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