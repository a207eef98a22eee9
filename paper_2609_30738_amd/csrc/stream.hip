// Streaming window statistics for bf16 caches with w = 32 (section 3.1, Eq. (1), Eq. (3)): two
// passes over the keys, each a plain stream from HBM with no communication between workgroups.
//
//   Work item: one segment of `seg_keys` consecutive keys of one (problem, kv head) unit, 512
//   threads = 8 waves.  Every lane holds the MFMA fragments of its window rows of all G heads of
//   the unit in registers for the whole segment.  Each wave streams 32-key tiles (tile j of the
//   segment goes to wave j % 8) from HBM into a private two-tile ring in LDS with direct-to-LDS,
//   non-temporal loads: every load instruction covers 1 KiB of consecutive key bytes (four 256-byte
//   rows at d = 128), and each lane picks the 16-byte chunk that lands at its LDS position, so the
//   tile is stored with its chunks XOR-swizzled by row (chunk c of row r at slot c ^ (r mod CH)).
//   The MFMA operand reads of 16 consecutive rows then touch 16 different chunk slots (all banks).
//   While a tile is computed, the next two are in flight.
//
//   stats_stream_kernel (pass 1): logits D[key][row] = K Q^T with keys as the MFMA M dimension, so
//     a lane holds one window row and 16 keys of each tile.  Every lane keeps, per head, the exact
//     running maximum m of t = logit * scale * log2 e and the sum z of 2^(t - m), rescaled when m
//     grows (online softmax).  At the end the lanes, then the waves, are merged and the segment's
//     (max, sum) per row goes to the workspace.
//   mu_sigma_stream_kernel (pass 2): merges the segment partials of its unit into the normalisers
//     b = M + log2 Z (segment 0 also writes row_max / row_sum), or takes them from given
//     row_max / row_sum; then logits again with keys as N (a lane holds one key),
//     a = 2^(t - b) summed over the group's heads, the mean and the two-pass sample variance over
//     the 32 window rows, stored as mu / sigma.  With `sigma_all` the variance runs over all G x 32
//     (head, row) values instead: every head's mean and squared deviations over its 32 rows, merged
//     across heads with the pairwise update of Chan, Golub and LeVeque.
//
//   Tiles with a masked key (the causal triangle of the window, keys past the segment end) take a
//   separate, guarded path; every other tile runs without masks or branches.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kTileKeys = 32;

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
  static constexpr int R = NB * 32;          // window rows of a unit (G heads x 32)
  static constexpr int NS = D / 16;          // MFMA K steps
  static constexpr int CH = D * 2 / 16;      // 16-byte chunks of a key row
  static constexpr int TE = kTileKeys * D;   // elements of a tile
  static constexpr int NDMA = TE * 2 / 1024; // 1 KiB load instructions per tile
  // LDS slot (in 16-byte chunks) of chunk `ch` of tile row `row`
  __device__ static int slot_of(int row, int ch) { return row * CH + (ch ^ (row % CH)); }
};

typedef const __attribute__((address_space(1))) void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

// s_waitcnt vmcnt(N): at most N vector memory operations of this wave still outstanding.  Vector
// memory operations complete in issue order, so this waits for everything issued before the last N.
template <int N> __device__ __forceinline__ void wait_vmem() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// maximum of three values (NaN-propagating, no canonicalisation of the operands)
__device__ __forceinline__ float fmax3(float a, float b, float c) {
  return __builtin_elementwise_maximum(__builtin_elementwise_maximum(a, b), c);
}

__device__ __forceinline__ float sum_halves(float x) {  // x + x of lane ^ 32
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Per-wave key stream of one segment: a two-tile ring in LDS filled by direct-to-LDS loads.
template <int D, int NB> struct KeyStream {
  using Gm = SGeo<D, NB>;
  uint16_t* ring;       // this wave's two tiles
  const uint16_t* kg;   // keys of the unit
  int k0, k1, wave, lane;

  __device__ int tile_key(int j) const { return k0 + (j * kWaves + wave) * kTileKeys; }

  // tile j into ring slot j & 1; rows past the segment end re-read its last key
  __device__ __forceinline__ void issue(int j) const {
    const int t0 = tile_key(j);
    uint16_t* dst = ring + (j & 1) * Gm::TE;
#pragma unroll
    for (int i = 0; i < Gm::NDMA; ++i) {
      const int pos = 64 * i + lane;  // LDS chunk slot written by this lane
      const int row = pos / Gm::CH;
      const int ch = (pos % Gm::CH) ^ (row % Gm::CH);
      const uint16_t* src = kg + (size_t)min(t0 + row, k1 - 1) * D + ch * 8;
      // aux 2: non-temporal (the keys are read once per pass)
      __builtin_amdgcn_global_load_lds((gptr_t)src, (lptr_t)(dst + i * 512), 16, 0, 2);
    }
  }

  // MFMA operand fragments of tile j (lane: row l32, K half `half`), once its loads have landed
  __device__ __forceinline__ void read(bf16x8_t (&a)[Gm::NS], int j, int l32, int half) const {
    const uint16_t* src = ring + (j & 1) * Gm::TE;
#pragma unroll
    for (int s = 0; s < Gm::NS; ++s)
      a[s] = *reinterpret_cast<const bf16x8_t*>(src + Gm::slot_of(l32, 2 * s + half) * 8);
  }

  // Wait for tile j (tile j + 1, if issued, may stay in flight), copy it into registers and hand
  // its slot to tile j + 2.  STORES: vector memory stores the caller issues per tile, after the
  // tile's computation; the tile's loads are then followed by the stores of tiles j - 2 and j - 1
  // and the loads of tile j + 1.
  template <int STORES>
  __device__ __forceinline__ void next(bf16x8_t (&a)[Gm::NS], int j, int my_tiles, int l32,
                                       int half) const {
    if (j + 1 < my_tiles) wait_vmem<Gm::NDMA + 2 * STORES>();
    else wait_vmem<0>();
    read(a, j, l32, half);
    wait_lds();
    if (j + 2 < my_tiles) issue(j + 2);
  }
};

// the unit's window-row fragments of every head (head b, rows b * 32 + l32), all K steps
template <int D, int NB>
__device__ __forceinline__ void load_queries(bf16x8_t (&q)[NB][D / 16], const uint16_t* qg, int l32,
                                             int half) {
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int s = 0; s < D / 16; ++s)
      q[b][s] = *reinterpret_cast<const bf16x8_t*>(qg + (size_t)(b * 32 + l32) * D + 16 * s + 8 * half);
}

// An empty use of every query register: the compiler waits for the query loads here, once,
// instead of at the first MFMA of the tile loop, where its wait would also cover the key tiles in
// flight.
template <int D, int NB>
__device__ __forceinline__ void hold_until_loaded(bf16x8_t (&q)[NB][D / 16]) {
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int s = 0; s < D / 16; ++s) asm volatile("" ::"v"(q[b][s]));
}

template <int NS>
__device__ __forceinline__ f32x16_t chain(const bf16x8_t (&x)[NS], const bf16x8_t (&y)[NS]) {
  f32x16_t d = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) d = mfma_step(x[s], y[s], d);
  return d;
}

// ------------------------------------------------------------------------------------------------
// Pass 1
// ------------------------------------------------------------------------------------------------
template <int D, int NB>
__global__ __launch_bounds__(kThreads, 1) void stats_stream_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS;
  __shared__ __align__(16) uint16_t ring[kWaves][2 * Gm::TE];
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

  KeyStream<D, NB> ks{ring[wave], a.k + ((size_t)a.tok_off[p] * a.h_kv + (size_t)g * L) * D, k0, k1,
                      wave, lane};
  const int n_tiles = (k1 - k0 + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + kWaves - 1) / kWaves : 0;
  // the query loads go first: vector memory operations complete in issue order, so the waits on
  // key tiles below also cover them
  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  if (my_tiles > 0) ks.issue(0);
  if (my_tiles > 1) ks.issue(1);
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
  __shared__ __align__(16) uint16_t ring[kWaves][2 * Gm::TE];
  __shared__ __align__(16) float bsh[R];
  __shared__ float2 mz_part[kThreads / R][R];

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

  KeyStream<D, NB> ks{ring[wave], a.k + ((size_t)a.tok_off[p] * a.h_kv + (size_t)g * L) * D, k0, k1,
                      wave, lane};
  const int n_tiles = (k1 - k0 + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + kWaves - 1) / kWaves : 0;
  // the query loads go first: vector memory operations complete in issue order, so the waits on
  // key tiles below also cover them
  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  if (my_tiles > 0) ks.issue(0);
  if (my_tiles > 1) ks.issue(1);
  hold_until_loaded<D, NB>(q);

  // Normalisers of the unit's rows.  From segment partials: thread (row, part) merges segments
  // part, part + P, ... of its row (four loads in flight), then one thread per row merges the P
  // results in a fixed order.
  constexpr int P = kThreads / R;
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
        // window rows 8 qq + 4 half + 0..3 of query head b
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
