// Per-segment loops of the two streaming passes (section 3.1, Eq. (1); section 3.2, Eq. (3)),
// shared by the pass kernels (stream_stats.hip, stream_mu_sigma.hip) and by the kernel that runs
// both passes over a whole unit in one workgroup (stream_window.hip).  The tile geometry and the
// key stream are described in stream_common.h.
#pragma once

#include "stream_common.h"

namespace kv {
namespace stream {

// Per-tile hook of pass 1 that does nothing (the plain statistics).
struct NoTileHook {
  static constexpr int kStores = 0;  // vector memory stores the hook issues per tile
  template <int NB>
  __device__ __forceinline__ void interior(int, const float (&)[NB]) const {}
  __device__ __forceinline__ void guarded(int) const {}
};

// Pass 1 over the wave's tiles of a segment [k0, k1) of a unit with L keys: for every head, the
// running maximum m of t = logit * c and the sum z of 2^(t - m) over the keys the lane's window
// row sees (online softmax; base 2).  Interior tiles run without masks or branches; a tile with a
// masked key (the causal triangle of the window, keys past the segment end) takes a guarded path.
// After each tile the hook sees the tile's index in the segment and, for an interior tile, the
// lane's largest logit (unscaled) of every head over its 16 keys; it issues Hook::kStores vector
// memory stores per tile, which the stream's waits count.
template <int D, int NB, int NW, int S, class Hook = NoTileHook>
__device__ __forceinline__ void stats_tiles(const KeyStream<D, NB, NW, S>& ks,
                                            const bf16x8_t (&q)[NB][D / 16], int my_tiles, int k1,
                                            int L, float c, int l32, int half, float (&m_run)[NB],
                                            float (&z_run)[NB], const Hook& hook = Hook{}) {
  constexpr int NS = D / 16;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    m_run[b] = -INFINITY;
    z_run[b] = 0.f;
  }
  // a tile is interior when none of its keys is masked: t0 + 31 < min(k1, L - 31)
  const int kedge = min(k1, L - 31);
  for (int j = 0; j < my_tiles; ++j) {
    bf16x8_t kt[NS];
    ks.template next<Hook::kStores>(kt, j, my_tiles, l32, half);
    const int t0 = ks.tile_key(j);
    if (t0 + 31 < kedge) {
      float tmax[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const f32x16_t d = chain<NS>(kt, q[b]);
        float mx = fmax3(fmax3(fmax3(d[0], d[1], d[2]), d[3], d[4]), d[5], d[6]);
        mx = fmax3(fmax3(mx, d[7], d[8]), d[9], d[10]);
        mx = fmax3(fmax3(mx, d[11], d[12]), d[13], d[14]);
        tmax[b] = __builtin_elementwise_maximum(mx, d[15]);
        const float mn = __builtin_elementwise_maximum(m_run[b], tmax[b] * c);
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
      hook.template interior<NB>(ks.tile_index(j), tmax);
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
      hook.guarded(ks.tile_index(j));
    }
  }
}

// Lanes l and l ^ 32 hold the same rows (different keys): merge them and put the wave's (m, z) of
// unit row b * 32 + l32 into red[b * 32 + l32].  The caller merges the waves after a barrier.
template <int NB>
__device__ __forceinline__ void stats_to_lds(const float (&m_run)[NB], const float (&z_run)[NB],
                                             float2* red, int l32, int half) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    float m = m_run[b], z = z_run[b];
    merge_mz(m, z, swap_halves(m), swap_halves(z));
    if (half == 0) red[b * 32 + l32] = make_float2(m, z);
  }
}

// (m, z) of one row over the NW waves' entries red[w * R + row], merged in wave order
template <int NW, int R>
__device__ __forceinline__ float2 merge_waves(const float2* red, int row) {
  float2 v = red[row];
#pragma unroll
  for (int w = 1; w < NW; ++w) merge_mz(v.x, v.y, red[w * R + row].x, red[w * R + row].y);
  return v;
}

// One mu or sigma value to HBM with the device-scope store policy (sc1).  These 128-byte pieces
// trickle out between the key loads of a stream that keeps HBM busy; on MI355X the default policy
// costs about 0.03 ms more per 2 GiB pass (the values are the same).  The store is counted by the
// explicit vmcnt waits of the key stream like any other vector memory operation.
__device__ __forceinline__ void store_stat(float* dst, float v) {
  asm volatile("global_store_dword %0, %1, off sc1" ::"v"(dst), "v"(v) : "memory");
}

// Output of pass 2 in base-score mode: the unit's score row and the base-score parameters.
struct ScoreOut {
  float* score_u;
  float lam1, w_mu;
};

// What pass 2 writes per key: mu and sigma, the base score, or (candidate mode) the base score of
// the keys of the tiles it evaluates, which also enter the unit's histogram of scores below.
enum PassOut { kOutMuSigma = 0, kOutScore = 1, kOutCand = 2 };

// Shared state of the second pass of candidate mode (stream_prune.hip), which revisits the unit's
// tiles in decreasing order of their score bound and stops at the first tile whose bound is below
// the unit's cut: the order key of the C-th best base score among the keys evaluated so far,
// rounded down to its bin of an LDS histogram of those keys (a lower bound of the final cut, so
// no key left out can be among the C best).  Every evaluated key's base score is stored at
// score_u[key] (section 3.2, the top-4B restriction: the candidate set is cut from them after the
// pass).
constexpr int kPruneShift = 21;                     // histogram bin = order key >> kPruneShift
constexpr int kPruneBins = 1 << (32 - kPruneShift);
struct Prune {
  const float* ubs;      // [n_tiles] LDS: score bound of the i-th tile of the order
  uint32_t* hist;        // [kPruneBins] LDS: evaluated candidate keys per bin
  uint32_t* cut;         // LDS: the unit's current cut (an order key; 0: none yet)
  float* score_u;        // the unit's score row (the evaluated keys only)
  int top_bin;           // where the cut's scan starts: the bin of the largest finite tile bound
  int n_cand, C;
  float smax;            // the lane's largest score over candidate positions (NaN ignored)
  int evaluated;         // tiles this wave evaluated

  // The wave's next tile is worth evaluating (its bound is not below the cut).
  __device__ __forceinline__ bool wanted(int idx) const {
    const uint32_t c = __builtin_amdgcn_readfirstlane(*cut);
    const uint32_t u = __builtin_amdgcn_readfirstlane(order_key(ubs[idx]));
    return u >= c;
  }

  // The evaluated candidate keys of a tile (one per lane of half 0) into the histogram and the
  // running maximum (the store of the score is the caller's).
  __device__ __forceinline__ void add(float sv, bool valid) {
    if (valid) smax = fmaxf(smax, sv);
    wave_hist_add(hist, order_key(sv) >> kPruneShift, valid);
  }

  // Raise the cut to the lower edge of the bin that holds the C-th best evaluated key among the
  // bins from top_bin down (the histogram as this wave sees it: counts only grow, so a stale view,
  // like keys above top_bin left out, gives a lower cut).
  __device__ __forceinline__ void update_cut(int lane) {
    uint32_t cum = 0;
    for (int b0 = top_bin; b0 >= 0; b0 -= 64) {
      const int b = b0 - lane;
      const uint32_t pre = wave_inclusive_sum(b >= 0 ? hist[b] : 0u);
      const uint64_t hit = __ballot(cum + pre >= (uint32_t)C);
      if (hit) {
        const int bin = b0 - (__ffsll((unsigned long long)hit) - 1);
        if (lane == 0) atomicMax(cut, (uint32_t)bin << kPruneShift);
        return;
      }
      cum += (uint32_t)__builtin_amdgcn_readlane((int)pre, 63);
    }
  }
};

// Pass 2 over the wave's tiles of a segment: logits again with keys as the MFMA N dimension (a
// lane holds one key), a = 2^(t - b) with the row normalisers b = M + log2 Z read from bsh, summed
// over the group's heads, then the mean and the two-pass sample variance over the 32 window rows,
// stored as mu / sigma (mu_u, sigma_u: the unit's rows).  With ALL the variance runs over all
// G x 32 (head, row) values: every head's mean and squared deviations over its 32 rows, merged
// across heads with the pairwise update of Chan, Golub and LeVeque.  With OUT = kOutScore the
// key's base score s = fma(lam1, sigma, w_mu mu) (section 3.2, Eq. (5)) is stored instead, with the
// same rounding as a score formed later from the stored mu and sigma; with OUT = kOutCand the
// score is also stored (at pr->score_u) and counted by the candidate state `pr` (keys below
// n_cand), and the wave stops at its first tile that pr no longer wants.
template <int D, int NB, bool ALL, int NW, int S, int OUT = kOutMuSigma>
__device__ __forceinline__ void mu_sigma_tiles(const KeyStream<D, NB, NW, S>& ks,
                                               const bf16x8_t (&q)[NB][D / 16], const float* bsh,
                                               int my_tiles, int k1, int L, float c, float inv_g,
                                               float* mu_u, float* sigma_u, int l32, int half,
                                               ScoreOut so = {}, Prune* pr = nullptr) {
  constexpr int kStores = 1;  // global stores per tile (the waits count them)
  const int lane = threadIdx.x & 63;
  constexpr int NS = D / 16;
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
    if constexpr (OUT == kOutScore) {
      // both halves hold the key's mean and variance; half 0 stores (every tile has a key < k1,
      // so the store the waits count is issued)
      const float sv = fmaf(so.lam1, __builtin_amdgcn_sqrtf(var), so.w_mu * mean);
      if (half == 0 && key < k1) store_stat(so.score_u + key, sv);
    } else if constexpr (OUT == kOutCand) {
      const float sv = fmaf(so.lam1, __builtin_amdgcn_sqrtf(var), so.w_mu * mean);
      pr->add(sv, half == 0 && key < pr->n_cand);
      if (half == 0 && key < k1) store_stat(pr->score_u + key, sv);
    } else {
      if (key < k1) store_stat((half == 0 ? mu_u : sigma_u) + key, half == 0 ? mean : __builtin_amdgcn_sqrtf(var));
    }
  };

  int j = 0;
  for (; j < my_tiles; ++j) {
    if constexpr (OUT == kOutCand) {
      if (!pr->wanted(j * NW + ks.wave)) break;
    }
    bf16x8_t kt[NS];
    ks.template next<kStores>(kt, j, my_tiles, l32, half);  // stores per tile in flight
    const int t0 = ks.tile_key(j);
    if (t0 + 31 > L - 32) tile(kt, t0, std::true_type{});
    else tile(kt, t0, std::false_type{});
    if constexpr (OUT == kOutCand) pr->update_cut(lane);
  }
  if constexpr (OUT == kOutCand) pr->evaluated = j;
}

}  // namespace stream
}  // namespace kv
