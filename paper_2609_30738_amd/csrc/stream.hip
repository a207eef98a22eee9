// Streaming window statistics for bf16 caches with w = 32 (section 3.1, Eq. (1), Eq. (3)): two
// passes over the keys, each a plain stream from HBM with no communication between workgroups.
//
//   Work item: one segment of `seg_keys` consecutive keys of one (problem, kv head) unit, 512
//   threads = 8 waves.  The unit's R = 32 G window rows are staged in LDS once; every wave streams
//   32-key tiles (tile j of the segment goes to wave j % 8) straight from HBM into MFMA operand
//   registers, two tiles ahead of the one it computes.
//
//   stats_stream_kernel (pass 1): logits D[key][row] = K Q^T with keys as the MFMA M dimension, so
//     a lane holds one window row and 16 keys of each tile.  Every lane keeps, for its rows, a
//     running offset m, the sum z of 2^(t - m) and the largest term e = 2^(t_max - m)
//     (t = logit * scale * log2 e).  A tile is summed against the running offset directly; only
//     when that sum is not below 2^32 (the first tile, a larger logit, an overflow) is the tile's
//     maximum logit taken and the lane rebased on it, so the common tile needs no maximum of the
//     logits, only one of its exponentials.  At the end every lane converts to the row maximum
//     m + log2 e and the sum z / e relative to it; the lanes, then the waves, are merged and the
//     segment's (max, sum) per row goes to the workspace.
//   mu_sigma_stream_kernel (pass 2): merges the segment partials of its unit into the normalisers
//     b = M + log2 Z (segment 0 also writes row_max / row_sum), or takes them from given
//     row_max / row_sum; then logits again with keys as N (a lane holds one key),
//     a = 2^(t - b) summed over the group's heads, the mean and the two-pass sample variance over
//     the 32 window rows, stored as mu / sigma.  With `sigma_all` the variance runs over all G x 32
//     (head, row) values instead: every head's mean and squared deviations over its 32 rows, merged
//     across heads with the pairwise update of Chan, Golub and LeVeque.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kTileKeys = 32;
constexpr int kSlots = 3;  // register slots of key tiles per wave (kSlots - 1 tiles in flight)
static_assert(kSlots == 3 || kSlots == 4, "the tile loop is unrolled for three or four slots");

struct StreamArgs {
  const uint16_t* q_win;
  const uint16_t* k;
  const int32_t* lens;
  const int64_t* tok_off;
  int h_q, h_kv;
  float c;  // softmax scale * log2(e)
  int seg_keys, max_segs;
  float2* part;           // [n_units][max_segs][R] segment partials (m, z), base 2
  const float* row_max;   // pass 2 from given statistics (part == nullptr)
  const float* row_sum;
  float* row_max_out;     // pass 2 from partials: written by segment 0
  float* row_sum_out;
  float* mu;
  float* sigma;
  int sigma_all;          // pass 2: dispersion over all G x 32 (head, row) values
};

template <int D, int NB> struct SGeo {
  static constexpr int R = NB * 32;       // window rows of a unit (G heads x 32)
  static constexpr int NS = D / 16;       // MFMA K steps
  static constexpr int CH = D * 2 / 16;   // 16-byte chunks of a query row
  // chunk `ch` of query row `row` sits at chunk ch ^ (row % CH) of the row in LDS, so that a
  // fragment read of 16 consecutive rows touches 16 different chunks (all banks)
  __device__ static int qslot(int row, int ch) { return row * CH + (ch ^ (row % CH)); }
};

__device__ __forceinline__ float sum_halves(float x) {  // x + x of lane ^ 32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// The unit's window rows (heads g G .. g G + G - 1 of problem p, contiguous in q_win) into LDS.
template <int D, int NB>
__device__ __forceinline__ void stage_unit_queries(const uint16_t* __restrict__ qg, uint16_t* qs) {
  using Gm = SGeo<D, NB>;
  for (int e = threadIdx.x; e < Gm::R * Gm::CH; e += kThreads) {
    const int row = e / Gm::CH, ch = e % Gm::CH;
    *reinterpret_cast<bf16x8_t*>(qs + Gm::qslot(row, ch) * 8) =
        *reinterpret_cast<const bf16x8_t*>(qg + 8 * e);
  }
}

// query fragments of head b (window rows b*32 + l32), all K steps
template <int D, int NB>
__device__ __forceinline__ void read_qfrags(bf16x8_t (&qf)[D / 16], const uint16_t* qs, int b,
                                            int l32, int half) {
  using Gm = SGeo<D, NB>;
  const int row = b * 32 + l32;
#pragma unroll
  for (int s = 0; s < Gm::NS; ++s)
    qf[s] = *reinterpret_cast<const bf16x8_t*>(qs + Gm::qslot(row, 2 * s + half) * 8);
}

// keys of this wave's tile starting at key t0 of the unit; a lane's key is clamped to the last key
// of the segment (kend - 1), so that the prefetches past the segment's last tile re-read one row
// instead of the next segment
template <int D>
__device__ __forceinline__ void load_tile(bf16x8_t (&t)[D / 16], const uint16_t* kg, int t0,
                                          int kend, int l32, int half) {
  const uint16_t* row = kg + (size_t)min(t0 + l32, kend - 1) * D + 8 * half;
#pragma unroll
  for (int s = 0; s < D / 16; ++s) t[s] = *reinterpret_cast<const bf16x8_t*>(row + 16 * s);
}

// ------------------------------------------------------------------------------------------------
// Pass 1
// ------------------------------------------------------------------------------------------------
template <int D, int NB>
__global__ __launch_bounds__(kThreads, 1) void stats_stream_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS;
  __shared__ __align__(16) uint16_t qs[R * D];
  __shared__ float2 red[kWaves][R];

  const int seg = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int L = a.lens[p];
  const int k0 = seg * a.seg_keys;
  if (k0 >= L) return;
  const int k1 = min(k0 + a.seg_keys, L);
  const int G = a.h_q / a.h_kv;
  const int lane = threadIdx.x & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const float c = a.c;

  stage_unit_queries<D, NB>(a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, qs);
  const uint16_t* kg = a.k + ((size_t)a.tok_off[p] * a.h_kv + (size_t)g * L) * D;
  const int n_tiles = (k1 - k0 + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + kWaves - 1) / kWaves : 0;
  auto tile_key = [&](int j) { return k0 + (j * kWaves + wave) * kTileKeys; };

  float m_run[NB], z_run[NB], e_run[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    m_run[b] = -INFINITY;
    z_run[b] = 0.f;
    e_run[b] = 0.f;
  }
  bf16x8_t slot[kSlots][NS];
#pragma unroll
  for (int q = 0; q + 1 < kSlots; ++q) load_tile<D>(slot[q], kg, tile_key(q), k1, l32, half);
  __syncthreads();

  auto tile = [&](const bf16x8_t (&t)[NS], int t0) __attribute__((always_inline)) {
    // window row l32 of every head sees keys <= L - 32 + l32; keys >= k1 belong to the next
    // segment.  The key of register j is t0 + 4 half + 8 (j / 4) + (j % 4).
    const bool edge = t0 + 31 >= min(k1, L - 31);
    const int thr = min(k1 - 1, L - 32 + l32) - t0 - 4 * half;
    // heads one after another: the scheduling barrier at the end of each keeps the compiler from
    // hoisting the next head's fragment reads (registers stay at one head's worth)
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      bf16x8_t qf[NS];
      read_qfrags<D, NB>(qf, qs, b, l32, half);
      f32x16_t d = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) d = mfma_step(t[s], qf[s], d);
      if (edge) {
#pragma unroll
        for (int j = 0; j < 16; ++j)
          if (8 * (j >> 2) + (j & 3) > thr) d[j] = -INFINITY;
      }
      const float mo = m_run[b];
      float ex[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) ex[j] = __builtin_amdgcn_exp2f(fmaf(d[j], c, -mo));
      // the terms are not negative: their bit patterns order like their values
      float zs[4];
      unsigned es[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        zs[u] = (ex[4 * u] + ex[4 * u + 1]) + (ex[4 * u + 2] + ex[4 * u + 3]);
        es[u] = max(max(__float_as_uint(ex[4 * u]), __float_as_uint(ex[4 * u + 1])),
                    max(__float_as_uint(ex[4 * u + 2]), __float_as_uint(ex[4 * u + 3])));
      }
      const float zt = (zs[0] + zs[1]) + (zs[2] + zs[3]);
      if (zt <= 4294967296.f) {
        z_run[b] += zt;
        e_run[b] = __uint_as_float(max(__float_as_uint(e_run[b]), max(max(es[0], es[1]), max(es[2], es[3]))));
      } else {
        // first tile of the lane, a larger logit or an overflow (also NaN from -inf - -inf):
        // rebase on the larger of the offset and the tile's maximum logit
        float mx = d[0];
#pragma unroll
        for (int j = 1; j < 16; ++j) mx = fmaxf(mx, d[j]);
        const float tm = mx * c;
        const float mn = fmaxf(mo, tm);
        if (mn != -INFINITY) {
          const float keep = mo == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mo - mn);
          float z = z_run[b] * keep;
#pragma unroll
          for (int j = 0; j < 16; ++j) z += __builtin_amdgcn_exp2f(fmaf(d[j], c, -mn));
          m_run[b] = mn;
          z_run[b] = z;
          e_run[b] = fmaxf(e_run[b] * keep, tm == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(tm - mn));
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  auto step = [&](auto sc, int j) __attribute__((always_inline)) {
    constexpr int S = decltype(sc)::value;
    constexpr int SN = (S + kSlots - 1) % kSlots;
    // tile j + kSlots - 1 into the slot tile j - 1 released (unconditional: a fixed number of
    // loads per step keeps every wait on exactly the tile it needs)
    load_tile<D>(slot[SN], kg, tile_key(j + kSlots - 1), k1, l32, half);
    if (j < my_tiles) tile(slot[S], tile_key(j));
  };
  for (int j0 = 0; j0 < my_tiles; j0 += kSlots) {
    step(std::integral_constant<int, 0>{}, j0);
    step(std::integral_constant<int, 1>{}, j0 + 1);
    step(std::integral_constant<int, 2>{}, j0 + 2);
    if constexpr (kSlots > 3) step(std::integral_constant<int, 3 % kSlots>{}, j0 + 3);
  }

  // (max, sum relative to it) of this lane's keys; lanes l and l ^ 32 hold the same rows
  // (different keys); then the waves
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const bool any = e_run[b] > 0.f;
    float m = any ? m_run[b] + __builtin_log2f(e_run[b]) : -INFINITY;
    float z = any ? z_run[b] / e_run[b] : 0.f;
    merge_mz(m, z, swap_halves(m), swap_halves(z));
    if (half == 0) red[wave][b * 32 + l32] = make_float2(m, z);
  }
  __syncthreads();
  if (threadIdx.x < R) {
    float2 v = red[0][threadIdx.x];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) merge_mz(v.x, v.y, red[w][threadIdx.x].x, red[w][threadIdx.x].y);
    a.part[(((size_t)p * a.h_kv + g) * a.max_segs + seg) * R + threadIdx.x] = v;
  }
}

// ------------------------------------------------------------------------------------------------
// Pass 2
// ------------------------------------------------------------------------------------------------
template <int D, int NB, bool ALL>
__global__ __launch_bounds__(kThreads, 1) void mu_sigma_stream_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS;
  __shared__ __align__(16) uint16_t qs[R * D];
  __shared__ __align__(16) float bsh[R];

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

  stage_unit_queries<D, NB>(a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, qs);
  if (threadIdx.x < R) {
    const size_t ri = ((size_t)p * a.h_q + (size_t)g * G) * 32 + threadIdx.x;
    float bv;
    if (a.part) {
      const int n_seg = (L + a.seg_keys - 1) / a.seg_keys;
      const float2* src = a.part + ((size_t)p * a.h_kv + g) * a.max_segs * R + threadIdx.x;
      float M = -INFINITY, Z = 0.f;
      for (int q = 0; q < n_seg; ++q) merge_mz(M, Z, src[(size_t)q * R].x, src[(size_t)q * R].y);
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
  const uint16_t* kg = a.k + ((size_t)a.tok_off[p] * a.h_kv + (size_t)g * L) * D;
  const size_t stat_base = (size_t)a.tok_off[p] * a.h_kv + (size_t)g * L;
  const int n_tiles = (k1 - k0 + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + kWaves - 1) / kWaves : 0;
  auto tile_key = [&](int j) { return k0 + (j * kWaves + wave) * kTileKeys; };

  bf16x8_t slot[kSlots][NS];
#pragma unroll
  for (int q = 0; q + 1 < kSlots; ++q) load_tile<D>(slot[q], kg, tile_key(q), k1, l32, half);
  __syncthreads();

  auto tile = [&](const bf16x8_t (&t)[NS], int t0) __attribute__((always_inline)) {
    const int key = t0 + l32;
    // window row r = 4 half + 8 (j / 4) + (j % 4) of every head sees the key iff key <= L - 32 + r
    const bool edge = t0 + 31 > L - 32;
    const int thr = key - (L - 32) - 4 * half;
    float ab[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) ab[j] = 0.f;
    float h_mean = 0.f, h_m2 = 0.f;  // ALL: running mean and squared deviations of the heads so far
    auto accumulate = [&](auto masked) __attribute__((always_inline)) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        float eb[16];
        bf16x8_t qf[NS];
        read_qfrags<D, NB>(qf, qs, b, l32, half);
        f32x16_t d = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s) d = mfma_step(qf[s], t[s], d);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // window rows 8 q + 4 half + 0..3 of query head b
          const float4 bv = *reinterpret_cast<const float4*>(bsh + b * 32 + 8 * q + 4 * half);
          const float bb[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int j = 4 * q + u;
            float e = __builtin_amdgcn_exp2f(fmaf(d[j], c, -bb[u]));
            if (decltype(masked)::value && 8 * q + u < thr) e = 0.f;
            ab[j] += e;
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
        __builtin_amdgcn_sched_barrier(0);  // one head at a time, as in pass 1
      }
    };
    if (edge) accumulate(std::true_type{});
    else accumulate(std::false_type{});
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

  auto step = [&](auto sc, int j) __attribute__((always_inline)) {
    constexpr int S = decltype(sc)::value;
    constexpr int SN = (S + kSlots - 1) % kSlots;
    load_tile<D>(slot[SN], kg, tile_key(j + kSlots - 1), k1, l32, half);
    if (j < my_tiles) tile(slot[S], tile_key(j));
  };
  for (int j0 = 0; j0 < my_tiles; j0 += kSlots) {
    step(std::integral_constant<int, 0>{}, j0);
    step(std::integral_constant<int, 1>{}, j0 + 1);
    step(std::integral_constant<int, 2>{}, j0 + 2);
    if constexpr (kSlots > 3) step(std::integral_constant<int, 3 % kSlots>{}, j0 + 3);
  }
}

template <int D, int NB>
hipError_t stream_dispatch(const Shape& s, const StreamArgs& args, bool pass1, hipStream_t st) {
  const int max_segs = args.max_segs;
  const dim3 grid(max_segs, s.h_kv, s.n_prob);
  if (pass1) stats_stream_kernel<D, NB><<<grid, kThreads, 0, st>>>(args);
  else if (args.sigma_all) mu_sigma_stream_kernel<D, NB, true><<<grid, kThreads, 0, st>>>(args);
  else mu_sigma_stream_kernel<D, NB, false><<<grid, kThreads, 0, st>>>(args);
  return hipGetLastError();
}

hipError_t stream_launch(const Shape& s, const StreamArgs& args, bool pass1, hipStream_t st) {
  const int G = s.group();
  if (s.d == 128) {
    if (G == 4) return stream_dispatch<128, 4>(s, args, pass1, st);
    if (G == 2) return stream_dispatch<128, 2>(s, args, pass1, st);
    return stream_dispatch<128, 1>(s, args, pass1, st);
  }
  if (G == 4) return stream_dispatch<64, 4>(s, args, pass1, st);
  if (G == 2) return stream_dispatch<64, 2>(s, args, pass1, st);
  return stream_dispatch<64, 1>(s, args, pass1, st);
}

StreamArgs base_args(const Shape& s, const StreamPlan& plan, const void* q_win, const void* k,
                     float scale) {
  StreamArgs a{};
  a.q_win = static_cast<const uint16_t*>(q_win);
  a.k = static_cast<const uint16_t*>(k);
  a.lens = s.lens;
  a.tok_off = s.tok_off;
  a.h_q = s.h_q;
  a.h_kv = s.h_kv;
  a.c = scale * kLog2e;
  a.seg_keys = plan.seg_keys;
  a.max_segs = plan.max_segs;
  return a;
}

}  // namespace

bool stream_shape_ok(const Shape& s, float scale) {
  const int G = s.group();
  // pass 1 takes a tile's maximum logit as the scaled maximum of the raw dot products
  return s.dtype == kDtBf16 && s.w == 32 && (s.d == 64 || s.d == 128) &&
         (G == 1 || G == 2 || G == 4) && scale > 0.f;
}

StreamPlan stream_plan(const Shape& s, int64_t total_keys) {
  // about one segment per compute unit (256 on MI355X), whole 256-key steps of the eight waves
  constexpr int64_t kTarget = 256, kStep = kWaves * kTileKeys, kMinSeg = 1024;
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
                               const void* k, float scale, void* ws, hipStream_t stream) {
  StreamArgs a = base_args(s, plan, q_win, k, scale);
  a.part = static_cast<float2*>(ws);
  return stream_launch(s, a, true, stream);
}

hipError_t launch_stream_mu_sigma(const Shape& s, const StreamPlan& plan, const void* q_win,
                                  const void* k, float scale, const void* ws,
                                  const float* row_max_in, const float* row_sum_in,
                                  float* row_max_out, float* row_sum_out, float* mu, float* sigma,
                                  bool sigma_all, hipStream_t stream) {
  StreamArgs a = base_args(s, plan, q_win, k, scale);
  a.part = const_cast<float2*>(static_cast<const float2*>(ws));
  a.row_max = row_max_in;
  a.row_sum = row_sum_in;
  a.row_max_out = row_max_out;
  a.row_sum_out = row_sum_out;
  a.mu = mu;
  a.sigma = sigma;
  a.sigma_all = sigma_all ? 1 : 0;
  return stream_launch(s, a, false, stream);
}

}  // namespace kv
