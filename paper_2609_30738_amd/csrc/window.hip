// Observation-window attention statistics (section 3.1, Eq. (1), Eq. (3)) on gfx950.
//
// Work item: one (problem p, kv head g, chunk of CHUNK keys), 256 threads = 4 waves.  The G*w window
// rows of the group (row m = h_local * w + r, padded to NB * 32) are staged once in LDS; each wave
// streams 32-key tiles of K straight from HBM into MFMA operand registers (the next tile is loaded
// while the current one is consumed).
//
//   window_stats_kernel: logits with keys as the MFMA M dimension (lane = window row, 16 keys per
//     lane), so the running max / sum of exponentials over keys is an in-lane online softmax in
//     base 2; per-chunk partials (m, z) go to the workspace.
//   combine_stats_kernel: merges the chunk partials of every window row into row_max / row_sum.
//   mu_sigma_kernel: recomputes the logits with keys as the N dimension (lane = key, 16 rows per
//     lane and M block), A = 2^(t - b) with b = row_max*log2(e) + log2(row_sum); for w = 32 every
//     M block is one query head, so the group mean, the mean over the window and the two-pass sample
//     variance are in-lane sums plus one exchange with lane ^ 32.  Other windows reduce through LDS.
//     With `sigma_all` the variance runs over all G w (head, row) values of the group.
#include "common.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;

template <typename T, int D> struct Lds {
  static constexpr int PITCH = D + 16 / (int)sizeof(T);  // padded row (elements): no bank conflicts
};

// Stage the R = G*w window rows of kv group g (contiguous in q_win) into LDS, zero-padding to NB*32.
template <typename T, int D, int NB>
__device__ __forceinline__ void stage_queries(const T* __restrict__ qg, int R, T* q_lds) {
  constexpr int VEC = 16 / (int)sizeof(T);
  constexpr int PER_ROW = D / VEC;
  constexpr int PITCH = Lds<T, D>::PITCH;
  for (int e = threadIdx.x; e < NB * 32 * PER_ROW; e += kThreads) {
    const int m = e / PER_ROW;
    const int c = (e % PER_ROW) * VEC;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (m < R) v = *reinterpret_cast<const uint4*>(qg + (size_t)m * D + c);
    *reinterpret_cast<uint4*>(q_lds + m * PITCH + c) = v;
  }
}

}  // namespace

// ------------------------------------------------------------------------------------------------
// Pass 1: per-chunk row statistics
// ------------------------------------------------------------------------------------------------
template <int DT, int D, int NB>
__global__ __launch_bounds__(kThreads) void window_stats_kernel(
    const typename Elem<DT>::T* __restrict__ q_win, const typename Elem<DT>::T* __restrict__ k,
    const int32_t* __restrict__ lens, const int64_t* __restrict__ tok_off, int h_q, int h_kv, int w,
    float c, int chunk_keys, int max_chunks, float2* __restrict__ partial) {
  using T = typename Elem<DT>::T;
  constexpr int ROWS = NB * 32;
  constexpr int PITCH = Lds<T, D>::PITCH;
  __shared__ __align__(16) T q_lds[ROWS * PITCH];
  __shared__ float2 wave_part[kWaves][ROWS];

  const int chunk = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int L = lens[p];
  const int k0 = chunk * chunk_keys;
  if (k0 >= L) return;
  const int k1 = min(k0 + chunk_keys, L);
  const int G = h_q / h_kv, R = G * w;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;

  stage_queries<T, D, NB>(q_win + ((size_t)p * h_q + (size_t)g * G) * w * D, R, q_lds);
  const T* kg = k + ((size_t)tok_off[p] * h_kv + (size_t)g * L) * D;

  // This lane's window row in every N block and the last key that row may see (causal mask).
  int lim[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int m = b * 32 + l32;
    lim[b] = (m < R) ? (L - w + (m % w)) : -1;
  }
  float m_run[NB], z_run[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    m_run[b] = -INFINITY;
    z_run[b] = 0.f;
  }
  __syncthreads();

  int t0 = k0 + wave * 32;
  Frags<DT, D> kf, kn;
  if (t0 < k1) kf.load_global(kg + (size_t)min(t0 + l32, L - 1) * D, half);
  for (; t0 < k1; t0 += kWaves * 32) {
    const int tn = t0 + kWaves * 32;
    if (tn < k1) kn.load_global(kg + (size_t)min(tn + l32, L - 1) * D, half);
    // Re-read the query fragments and row shifts from LDS every tile instead of pinning them in
    // registers for the whole loop: keeps the wave small enough for several waves per SIMD.
    asm volatile("" ::: "memory");
    // keys t0..t0+31 all present and visible to every row?
    const bool full = (t0 + 32 <= k1) && (t0 + 31 <= L - w);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      Frags<DT, D> qf;
      qf.load_lds(q_lds + (b * 32 + l32) * PITCH, half);
      const f32x16_t acc = mfma_tile<DT, D>(kf, qf);  // D[key][row]
      float tv[16];
      float tmax = -INFINITY;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        float t = acc[j] * c;
        if (!full) {
          const int key = t0 + acc_row(j, lane);
          if (key >= k1 || key > lim[b]) t = -INFINITY;
        }
        tv[j] = t;
        tmax = fmaxf(tmax, t);
      }
      const float mn = fmaxf(m_run[b], tmax);
      if (mn != -INFINITY) {
        float z = (m_run[b] == -INFINITY) ? 0.f : z_run[b] * __builtin_amdgcn_exp2f(m_run[b] - mn);
#pragma unroll
        for (int j = 0; j < 16; ++j) z += __builtin_amdgcn_exp2f(tv[j] - mn);
        m_run[b] = mn;
        z_run[b] = z;
      }
    }
    kf = kn;
  }

  // Lanes l and l ^ 32 hold the same row (different keys); then merge the four waves.
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const float m2 = swap_halves(m_run[b]);
    const float z2 = swap_halves(z_run[b]);
    merge_mz(m_run[b], z_run[b], m2, z2);
    if (half == 0) wave_part[wave][b * 32 + l32] = make_float2(m_run[b], z_run[b]);
  }
  __syncthreads();
  if (threadIdx.x < ROWS) {
    float2 acc = wave_part[0][threadIdx.x];
#pragma unroll
    for (int v = 1; v < kWaves; ++v) {
      const float2 o = wave_part[v][threadIdx.x];
      merge_mz(acc.x, acc.y, o.x, o.y);
    }
    partial[(((size_t)p * h_kv + g) * max_chunks + chunk) * ROWS + threadIdx.x] = acc;
  }
}

// One thread per (problem, q head, window row): merge the chunk partials.
__global__ __launch_bounds__(kThreads) void combine_stats_kernel(
    const float2* __restrict__ partial, const int32_t* __restrict__ lens, int n_prob, int h_q,
    int h_kv, int w, int rows_pad, int chunk_keys, int max_chunks, float* __restrict__ row_max,
    float* __restrict__ row_sum) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)n_prob * h_q * w) return;
  const int p = (int)(idx / ((int64_t)h_q * w));
  const int rem = (int)(idx % ((int64_t)h_q * w));
  const int h = rem / w, r = rem % w;
  const int G = h_q / h_kv, g = h / G, m = (h % G) * w + r;
  const int n_chunks = (lens[p] + chunk_keys - 1) / chunk_keys;
  float M = -INFINITY, Z = 0.f;
  const float2* src = partial + ((size_t)p * h_kv + g) * max_chunks * rows_pad + m;
  for (int ch0 = 0; ch0 < n_chunks; ch0 += 4) {  // four loads in flight
    float2 o[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      o[u] = ch0 + u < n_chunks ? src[(size_t)(ch0 + u) * rows_pad] : make_float2(-INFINITY, 0.f);
#pragma unroll
    for (int u = 0; u < 4; ++u) merge_mz(M, Z, o[u].x, o[u].y);
  }
  row_max[idx] = M * kLn2;
  row_sum[idx] = Z;
}

// ------------------------------------------------------------------------------------------------
// Pass 2: attention, group mean, mean and sample dispersion over the window
// ------------------------------------------------------------------------------------------------
template <int DT, int D, int NB, bool W32, bool ALL>
__global__ __launch_bounds__(kThreads) void mu_sigma_kernel(
    const typename Elem<DT>::T* __restrict__ q_win, const typename Elem<DT>::T* __restrict__ k,
    const int32_t* __restrict__ lens, const int64_t* __restrict__ tok_off, int h_q, int h_kv, int w,
    float c, int chunk_keys, const float* __restrict__ row_max, const float* __restrict__ row_sum,
    float* __restrict__ mu, float* __restrict__ sigma, float* __restrict__ attn) {
  using T = typename Elem<DT>::T;
  constexpr int ROWS = NB * 32;
  constexpr int PITCH = Lds<T, D>::PITCH;
  constexpr int RED_ROWS = W32 ? 1 : ROWS;
  __shared__ __align__(16) T q_lds[ROWS * PITCH];
  __shared__ __align__(16) float bsh[ROWS];
  __shared__ float red[kWaves][RED_ROWS][33];

  const int chunk = blockIdx.x, g = blockIdx.y, p = blockIdx.z;
  const int L = lens[p];
  const int k0 = chunk * chunk_keys;
  if (k0 >= L) return;
  const int k1 = min(k0 + chunk_keys, L);
  const int G = h_q / h_kv, R = G * w;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, half = lane >> 5, l32 = lane & 31;

  stage_queries<T, D, NB>(q_win + ((size_t)p * h_q + (size_t)g * G) * w * D, R, q_lds);
  for (int m = threadIdx.x; m < ROWS; m += kThreads) {
    float b = INFINITY;  // padded rows contribute 2^(-inf) = 0
    if (m < R) {
      const size_t ri = ((size_t)p * h_q + (size_t)g * G + m / w) * w + (m % w);
      b = row_max[ri] * kLog2e + log2f(row_sum[ri]);
    }
    bsh[m] = b;
  }
  const T* kg = k + ((size_t)tok_off[p] * h_kv + (size_t)g * L) * D;
  const size_t stat_base = (size_t)tok_off[p] * h_kv + (size_t)g * L;
  float* attn_g = attn ? attn + (size_t)tok_off[p] * h_q * w + (size_t)g * G * w * L : nullptr;
  const float inv_g = 1.f / (float)G;
  const float inv_w = 1.f / (float)w;
  const float inv_w1 = 1.f / (float)(w - 1);
  __syncthreads();

  int t0 = k0 + wave * 32;
  Frags<DT, D> kf, kn;
  if (t0 < k1) kf.load_global(kg + (size_t)min(t0 + l32, L - 1) * D, half);
  for (; t0 < k1; t0 += kWaves * 32) {
    const int tn = t0 + kWaves * 32;
    if (tn < k1) kn.load_global(kg + (size_t)min(tn + l32, L - 1) * D, half);
    // Re-read the query fragments and row shifts from LDS every tile instead of pinning them in
    // registers for the whole loop: keeps the wave small enough for several waves per SIMD.
    asm volatile("" ::: "memory");
    const int key = t0 + l32;
    const bool key_ok = key < k1;
    const bool full = (t0 + 32 <= k1) && (t0 + 31 <= L - w);
    float abar[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) abar[j] = 0.f;
    float h_mean = 0.f, h_m2 = 0.f;  // W32 && ALL: running mean / squared deviations over heads
#pragma unroll 1
    for (int b = 0; b < NB; ++b) {
      Frags<DT, D> qf;
      qf.load_lds(q_lds + (b * 32 + l32) * PITCH, half);
      const f32x16_t acc = mfma_tile<DT, D>(qf, kf);  // D[row][key]
      float ah[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int m = b * 32 + acc_row(j, lane);
        float a = __builtin_amdgcn_exp2f(acc[j] * c - bsh[m]);
        if (!full) {
          const int r = m % w;
          if (!key_ok || key > L - w + r) a = 0.f;
        }
        if constexpr (W32)
          abar[j] += a;
        else
          red[wave][m][l32] = a;  // every (row, key) of the tile is held by exactly one lane
        ah[j] = a;
        if (attn_g && key_ok && m < R) attn_g[(size_t)m * L + key] = a;
      }
      if constexpr (W32 && ALL) {
        // head b (rows b*32 .. b*32+31, all real when b < G) merged into the running moments with
        // the pairwise update of Chan, Golub and LeVeque
        if (b < G) {
          float hs = 0.f;
#pragma unroll
          for (int j = 0; j < 16; ++j) hs += ah[j];
          const float mb = (hs + swap_halves(hs)) * (1.f / 32.f);
          float hv = 0.f;
#pragma unroll
          for (int j = 0; j < 16; ++j) hv = fmaf(ah[j] - mb, ah[j] - mb, hv);
          const float m2b = hv + swap_halves(hv);
          const float dl = mb - h_mean;
          const float fb = (float)b;
          h_mean = fmaf(dl, 1.f / (fb + 1.f), h_mean);
          h_m2 += fmaf(dl * dl, 32.f * fb / (fb + 1.f), m2b);
        }
      }
    }
    if constexpr (W32) {
      // rows acc_row(j, lane) are window rows r; the other 16 rows live in lane ^ 32
      float s = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        abar[j] *= inv_g;
        s += abar[j];
      }
      const float mean = (s + swap_halves(s)) * inv_w;
      float v = 0.f;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float dlt = abar[j] - mean;
        v += dlt * dlt;
      }
      v = (v + swap_halves(v)) * inv_w1;
      if constexpr (ALL) v = h_m2 / (float)(R - 1);
      if (half == 0 && key_ok) {
        mu[stat_base + key] = mean;
        sigma[stat_base + key] = sqrtf(v);
      }
    } else {
      // the tile's values were written by other lanes of this wave
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      if (ALL && half == 0 && key_ok) {
        float s = 0.f;
        for (int m = 0; m < R; ++m) s += red[wave][m][l32];
        const float mean = s / (float)R;
        float v = 0.f;
        for (int m = 0; m < R; ++m) {
          const float dlt = red[wave][m][l32] - mean;
          v += dlt * dlt;
        }
        mu[stat_base + key] = mean;
        sigma[stat_base + key] = sqrtf(v / (float)(R - 1));
      } else if (half == 0 && key_ok) {
        float s = 0.f;
        for (int r = 0; r < w; ++r) {
          float ab = 0.f;
          for (int hl = 0; hl < G; ++hl) ab += red[wave][hl * w + r][l32];
          s += ab * inv_g;
        }
        const float mean = s * inv_w;
        float v = 0.f;
        for (int r = 0; r < w; ++r) {
          float ab = 0.f;
          for (int hl = 0; hl < G; ++hl) ab += red[wave][hl * w + r][l32];
          const float dlt = ab * inv_g - mean;
          v += dlt * dlt;
        }
        mu[stat_base + key] = mean;
        sigma[stat_base + key] = sqrtf(v * inv_w1);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    kf = kn;
  }
}

// ------------------------------------------------------------------------------------------------
// Launchers
// ------------------------------------------------------------------------------------------------
size_t window_stats_ws_bytes(const Shape& s) {
  return (size_t)s.n_prob * s.h_kv * s.max_chunks() * (s.row_blocks() * 32) * sizeof(float2);
}

namespace {

template <int DT, int D, int NB>
hipError_t stats_dispatch(const Shape& s, const void* q, const void* k, float scale, void* ws,
                          float* row_max, float* row_sum, hipStream_t st) {
  using T = typename Elem<DT>::T;
  const dim3 grid(s.max_chunks(), s.h_kv, s.n_prob);
  window_stats_kernel<DT, D, NB><<<grid, kThreads, 0, st>>>(
      static_cast<const T*>(q), static_cast<const T*>(k), s.lens, s.tok_off, s.h_q, s.h_kv, s.w,
      scale * kLog2e, kWindowChunk, s.max_chunks(), static_cast<float2*>(ws));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t rows = (int64_t)s.n_prob * s.h_q * s.w;
  combine_stats_kernel<<<(unsigned)((rows + kThreads - 1) / kThreads), kThreads, 0, st>>>(
      static_cast<const float2*>(ws), s.lens, s.n_prob, s.h_q, s.h_kv, s.w, NB * 32,
      kWindowChunk, s.max_chunks(), row_max, row_sum);
  return hipGetLastError();
}

template <int DT, int D, int NB, bool W32>
hipError_t mu_sigma_dispatch(const Shape& s, const void* q, const void* k, float scale,
                             const float* row_max, const float* row_sum, float* mu,
                             float* sigma, float* attn, bool all, hipStream_t st) {
  using T = typename Elem<DT>::T;
  const dim3 grid(s.max_chunks(), s.h_kv, s.n_prob);
  auto kern = all ? mu_sigma_kernel<DT, D, NB, W32, true> : mu_sigma_kernel<DT, D, NB, W32, false>;
  kern<<<grid, kThreads, 0, st>>>(
      static_cast<const T*>(q), static_cast<const T*>(k), s.lens, s.tok_off, s.h_q, s.h_kv, s.w,
      scale * kLog2e, kWindowChunk, row_max, row_sum, mu, sigma, attn);
  return hipGetLastError();
}

template <int DT, int D>
hipError_t stats_nb(const Shape& s, const void* q, const void* k, float scale, void* ws,
                    float* rm, float* rs, hipStream_t st) {
  switch (s.row_blocks()) {
    case 1: return stats_dispatch<DT, D, 1>(s, q, k, scale, ws, rm, rs, st);
    case 2: return stats_dispatch<DT, D, 2>(s, q, k, scale, ws, rm, rs, st);
    default: return stats_dispatch<DT, D, 4>(s, q, k, scale, ws, rm, rs, st);
  }
}

template <int DT, int D>
hipError_t mu_sigma_nb(const Shape& s, const void* q, const void* k, float scale,
                       const float* rm, const float* rs, float* mu, float* sg, float* attn,
                       bool all, hipStream_t st) {
  const int nb = s.row_blocks();
  if (s.w == 32) {
    switch (nb) {
      case 1: return mu_sigma_dispatch<DT, D, 1, true>(s, q, k, scale, rm, rs, mu, sg, attn, all, st);
      case 2: return mu_sigma_dispatch<DT, D, 2, true>(s, q, k, scale, rm, rs, mu, sg, attn, all, st);
      default: return mu_sigma_dispatch<DT, D, 4, true>(s, q, k, scale, rm, rs, mu, sg, attn, all, st);
    }
  }
  if (nb == 1)
    return mu_sigma_dispatch<DT, D, 1, false>(s, q, k, scale, rm, rs, mu, sg, attn, all, st);
  return mu_sigma_dispatch<DT, D, 2, false>(s, q, k, scale, rm, rs, mu, sg, attn, all, st);
}

}  // namespace

hipError_t launch_combine_partials(const Shape& s, const void* part, int chunk_keys,
                                   int max_chunks, int rows_pad, float* row_max, float* row_sum,
                                   hipStream_t stream) {
  const int64_t rows = (int64_t)s.n_prob * s.h_q * s.w;
  combine_stats_kernel<<<(unsigned)((rows + kThreads - 1) / kThreads), kThreads, 0, stream>>>(
      static_cast<const float2*>(part), s.lens, s.n_prob, s.h_q, s.h_kv, s.w, rows_pad, chunk_keys,
      max_chunks, row_max, row_sum);
  return hipGetLastError();
}

hipError_t launch_window_stats(const Shape& s, const void* q_win, const void* k, float scale,
                               void* ws, float* row_max, float* row_sum, hipStream_t stream) {
  if (s.dtype == kDtBf16)
    return s.d == 64 ? stats_nb<kDtBf16, 64>(s, q_win, k, scale, ws, row_max, row_sum, stream)
                     : stats_nb<kDtBf16, 128>(s, q_win, k, scale, ws, row_max, row_sum, stream);
  return s.d == 64 ? stats_nb<kDtF32, 64>(s, q_win, k, scale, ws, row_max, row_sum, stream)
                   : stats_nb<kDtF32, 128>(s, q_win, k, scale, ws, row_max, row_sum, stream);
}

hipError_t launch_mu_sigma(const Shape& s, const void* q_win, const void* k, float scale,
                           const float* row_max, const float* row_sum, float* mu, float* sigma,
                           float* attn, bool sigma_all, hipStream_t stream) {
  const bool all = sigma_all;
  if (s.dtype == kDtBf16)
    return s.d == 64
               ? mu_sigma_nb<kDtBf16, 64>(s, q_win, k, scale, row_max, row_sum, mu, sigma, attn, all, stream)
               : mu_sigma_nb<kDtBf16, 128>(s, q_win, k, scale, row_max, row_sum, mu, sigma, attn, all, stream);
  return s.d == 64
             ? mu_sigma_nb<kDtF32, 64>(s, q_win, k, scale, row_max, row_sum, mu, sigma, attn, all, stream)
             : mu_sigma_nb<kDtF32, 128>(s, q_win, k, scale, row_max, row_sum, mu, sigma, attn, all, stream);
}

}  // namespace kv
