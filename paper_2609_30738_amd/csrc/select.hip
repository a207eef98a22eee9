// Greedy diversity-aware admission (section 3.2, Eq. (2), (4), (5)) on gfx950.
//
// One workgroup per (problem, kv head): 1024 threads for bf16 keys (one candidate per thread), 256
// for fp32 keys (up to four per thread, whose key rows need more registers):
//   1. base scores s_i = fma(lambda1, sigma_i, w_mu mu_i) over the candidates [0, n_cand) (optionally
//      max-pooled over an odd window of positions, the outside of [0, n_cand) ignored), their maximum
//      (the normaliser, clamped at 1e-12), and the C-th largest score by a most-significant-digit
//      radix select over order-preserving 32-bit keys (4 passes of 8 bits, wave-private LDS
//      histograms filled with LDS atomics); the keys are staged in LDS once with
//      coalesced loads when they fit (up to 34816 candidates), otherwise recomputed per pass;
//   2. the candidate set P: every score above the threshold plus the lowest positions among those
//      equal to it, compacted in ascending position order (ballot ranks inside a wave, LDS prefix
//      across waves);
//   3. B greedy steps.  Thread t owns candidates t, t + NT, ...: it keeps their keys in registers,
//      their normalised score s~, running max-cosine and admitted flag.  Each step updates the
//      running maxima against the last admitted key (read from an LDS copy of the candidate keys),
//      forms s~ + lambda2 * corr, and finds the (score, lowest slot) maximum: a DPP / permlane
//      maximum and a ballot inside each wave, then one barrier; the per-wave winners are
//      double-buffered so that one barrier per step suffices.
#include <float.h>

#include <algorithm>

#include "common.h"
#include "compact_rows.h"
#include "kernels.h"

namespace kv {

namespace {

constexpr int kMaxCandBytes = 131072;        // LDS copy of the candidate keys
constexpr int kMaxStagedKeyBytes = 139264;  // LDS copy of every candidate's score key (34816)
constexpr size_t kLdsBytes = 163840;        // LDS of one CU

__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Add one to hist[digit] for every active lane.  The digit of the first active lane is counted
// with one ballot and a single LDS add (the common case: most scores share their leading digits);
// lanes with other digits use LDS atomics, which handle scattered digits without conflicts.
__device__ __forceinline__ void wave_hist_add(uint32_t* hist, uint32_t digit, bool active) {
  const uint64_t act = __ballot(active);
  if (act == 0) return;
  const int leader = __ffsll((unsigned long long)act) - 1;
  const uint32_t dl = __builtin_amdgcn_readlane(digit, leader);
  const uint64_t same = __ballot(active && digit == dl);
  if ((int)(threadIdx.x & 63) == leader) atomicAdd(&hist[dl], (uint32_t)__popcll(same));
  if (active && digit != dl) atomicAdd(&hist[digit], 1u);
}

// (score, slot) packed so that a larger value means a larger score, then a lower slot.
__device__ __forceinline__ uint64_t pack_best(float score, int slot) {
  return ((uint64_t)order_key(score) << 32) | (uint32_t)(0x7FFFFFFF - slot);
}
__device__ __forceinline__ int unpack_slot(uint64_t v) { return 0x7FFFFFFF - (int)(uint32_t)v; }
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}
// Maximum over the 64 lanes, in every lane: quad and row steps with DPP, then permlane swaps
// between rows and between the wave's halves.
__device__ __forceinline__ float wave_max_f(float v) {
#define KV_DPPF(x, CTRL) __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), CTRL, 0xF, 0xF, false))
#define KV_MAX(a, b) __builtin_elementwise_maximum(a, b)  // no operand canonicalisation
  v = KV_MAX(v, KV_DPPF(v, 0xB1));   // quad_perm [1,0,3,2]
  v = KV_MAX(v, KV_DPPF(v, 0x4E));   // quad_perm [2,3,0,1]
  v = KV_MAX(v, KV_DPPF(v, 0x124));  // row_ror:4
  v = KV_MAX(v, KV_DPPF(v, 0x128));  // row_ror:8
  auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = KV_MAX(__uint_as_float(r16[0]), __uint_as_float(r16[1]));
  auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return KV_MAX(__uint_as_float(r32[0]), __uint_as_float(r32[1]));
#undef KV_MAX
#undef KV_DPPF
}

// (score, slot) of the best candidate of the wave, ties to the lowest slot.  With one candidate
// per lane (slots ascending with the lane) the lowest tied lane holds the lowest slot.
template <bool ONE_PER_LANE>
__device__ __forceinline__ uint64_t wave_best(float score, int slot) {
  const float wm = wave_max_f(score);
  const uint64_t tied = __ballot(score == wm);
  int best = __builtin_amdgcn_readlane(slot, __ffsll((unsigned long long)tied) - 1);
  if (!ONE_PER_LANE && wm > -INFINITY && __popcll(tied) > 1) {
    // exact tie between lanes: lowest slot among them (a wave with no live slot left ties at -inf)
    uint64_t rest = tied;
    while (rest) {
      const int l = __ffsll((unsigned long long)rest) - 1;
      best = min(best, __builtin_amdgcn_readlane(slot, l));
      rest &= rest - 1;
    }
  }
  return pack_best(wm, best);
}

// Key row of one candidate held in registers, and its dot product with a row in LDS.
template <int DT, int D> struct KeyRow;

template <int D> struct KeyRow<kDtBf16, D> {
  typedef __bf16 __attribute__((ext_vector_type(2))) bf2;
  bf2 v[D / 2];
  __device__ __forceinline__ void load(const uint16_t* row) {
    const uint4* src = reinterpret_cast<const uint4*>(row);
#pragma unroll
    for (int q = 0; q < D / 8; ++q) {
      const uint4 x = src[q];
      v[4 * q + 0] = __builtin_bit_cast(bf2, x.x);
      v[4 * q + 1] = __builtin_bit_cast(bf2, x.y);
      v[4 * q + 2] = __builtin_bit_cast(bf2, x.z);
      v[4 * q + 3] = __builtin_bit_cast(bf2, x.w);
    }
  }
  __device__ __forceinline__ void store(uint16_t* row) const {
    uint4* dst = reinterpret_cast<uint4*>(row);
#pragma unroll
    for (int q = 0; q < D / 8; ++q)
      dst[q] = make_uint4(__builtin_bit_cast(uint32_t, v[4 * q + 0]), __builtin_bit_cast(uint32_t, v[4 * q + 1]),
                          __builtin_bit_cast(uint32_t, v[4 * q + 2]), __builtin_bit_cast(uint32_t, v[4 * q + 3]));
  }
  __device__ __forceinline__ float dot_lds(const uint16_t* row) const {
    const uint4* src = reinterpret_cast<const uint4*>(row);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < D / 8; ++q) {
      const uint4 x = src[q];
      acc[0] = __builtin_amdgcn_fdot2_f32_bf16(v[4 * q + 0], __builtin_bit_cast(bf2, x.x), acc[0], false);
      acc[1] = __builtin_amdgcn_fdot2_f32_bf16(v[4 * q + 1], __builtin_bit_cast(bf2, x.y), acc[1], false);
      acc[2] = __builtin_amdgcn_fdot2_f32_bf16(v[4 * q + 2], __builtin_bit_cast(bf2, x.z), acc[2], false);
      acc[3] = __builtin_amdgcn_fdot2_f32_bf16(v[4 * q + 3], __builtin_bit_cast(bf2, x.w), acc[3], false);
    }
    return (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  __device__ __forceinline__ float sq_norm() const {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < D / 2; ++i)
      acc[i & 3] = __builtin_amdgcn_fdot2_f32_bf16(v[i], v[i], acc[i & 3], false);
    return (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
};

template <int D> struct KeyRow<kDtF32, D> {
  float v[D];
  __device__ __forceinline__ void load(const float* row) {
    const float4* src = reinterpret_cast<const float4*>(row);
#pragma unroll
    for (int q = 0; q < D / 4; ++q) {
      const float4 x = src[q];
      v[4 * q + 0] = x.x;
      v[4 * q + 1] = x.y;
      v[4 * q + 2] = x.z;
      v[4 * q + 3] = x.w;
    }
  }
  __device__ __forceinline__ void store(float* row) const {
    float4* dst = reinterpret_cast<float4*>(row);
#pragma unroll
    for (int q = 0; q < D / 4; ++q) dst[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  }
  __device__ __forceinline__ float dot_lds(const float* row) const {
    const float4* src = reinterpret_cast<const float4*>(row);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int q = 0; q < D / 4; ++q) {
      const float4 x = src[q];
      acc[0] = fmaf(v[4 * q + 0], x.x, acc[0]);
      acc[1] = fmaf(v[4 * q + 1], x.y, acc[1]);
      acc[2] = fmaf(v[4 * q + 2], x.z, acc[2]);
      acc[3] = fmaf(v[4 * q + 3], x.w, acc[3]);
    }
    return (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
  __device__ __forceinline__ float sq_norm() const {
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < D; ++i) acc[i & 3] = fmaf(v[i], v[i], acc[i & 3]);
    return (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
};

template <int NW> struct SelectShared {
  uint32_t hist[NW][256];
  uint32_t scan[256];
  uint32_t wave_cnt[2][NW];
  float wave_max[NW];
  uint4 best[2][NW];  // per wave and step parity: the packed (score, slot) pair, 1 / |k|
  uint32_t halo[2][32];  // raw keys left of a pooling chunk (pool_h <= 31)
  uint32_t sel_threshold;
  int sel_need;
};

// Compaction after the selection (k_out == nullptr: none); K, V, outputs as 16-byte vectors.
struct CompactOut {
  const uint4* k;
  const uint4* v;
  uint4* k_out;
  uint4* v_out;
  int out_rows;
};

}  // namespace

template <int DT, int D, int NT, int CPT, bool STAGED>
__global__ __launch_bounds__(NT) void mmr_select_kernel(
    const float* __restrict__ mu, const float* __restrict__ sigma,
    const typename Elem<DT>::T* __restrict__ k, const int32_t* __restrict__ lens,
    const int64_t* __restrict__ tok_off, const float* __restrict__ lambda1,
    const float* __restrict__ lambda2, int pool_h, float w_mu, int h_kv, int budget,
    const int32_t* __restrict__ budgets, int cand_mult, int keep_tail,
    int cand_stride, int max_cand, int32_t* __restrict__ sel_idx, float* __restrict__ sel_score,
    int32_t* __restrict__ cand_idx, float* __restrict__ cand_corr, CompactOut co) {
  using T = typename Elem<DT>::T;
  constexpr int kThreads = NT, kWaves = NT / 64;
  static_assert(NT >= 256, "one thread per histogram bin");
  __shared__ SelectShared<kWaves> sh;
  // dynamic LDS: [max_cand] positions, [max_cand] 1/|k|, then a region that first holds the
  // order-preserving keys of every candidate score (STAGED) and then the candidates' key rows
  extern __shared__ __align__(16) unsigned char dyn[];
  const int g = blockIdx.x % h_kv, p = blockIdx.x / h_kv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int L = lens[p];
  const int n_cand = L - keep_tail;
  const int bp = budgets ? budgets[p] : budget;  // this problem's budget; `budget` is the row stride
  const int C = cand_mult > 0 ? min(cand_mult * bp, n_cand) : n_cand;
  const size_t base = (size_t)tok_off[p] * h_kv + (size_t)g * L;
  const float* mu_g = mu + base;
  const float* sg_g = sigma + base;
  const T* kg = k + base * D;
  const float lam1 = lambda1[p], lam2 = lambda2[p];
  int32_t* cpos = reinterpret_cast<int32_t*>(dyn);
  float* cinv = reinterpret_cast<float*>(dyn + (size_t)max_cand * 4);
  unsigned char* region = dyn + (((size_t)max_cand * 8 + 15) & ~(size_t)15);
  uint32_t* skeys = reinterpret_cast<uint32_t*>(region);
  T* ckeys = reinterpret_cast<T*>(region);
  const bool take_all = (C >= n_cand);

  // ---- 0. base scores s_i = mu_i + lambda1 sigma_i (one rounding) and their maximum -----------
  float local_max = -INFINITY;
  if constexpr (STAGED) {
    // mu / sigma rows start at a multiple of 4 floats only if base is; stage element-wise until
    // the first aligned index, then 4 per lane with several loads in flight
    const int head = (int)((4 - (base & 3)) & 3) < n_cand ? (int)((4 - (base & 3)) & 3) : n_cand;
    if (tid < head) {
      const float sv = fmaf(lam1, sg_g[tid], w_mu * mu_g[tid]);
      local_max = fmaxf(local_max, sv);
      skeys[tid] = order_key(sv);
    }
    const int n4 = (n_cand - head) / 4;
    const float4* mu4 = reinterpret_cast<const float4*>(mu_g + head);
    const float4* sg4 = reinterpret_cast<const float4*>(sg_g + head);
#pragma unroll 4
    for (int v = tid; v < n4; v += kThreads) {
      const float4 m = mu4[v], sgv = sg4[v];
      const float s0 = fmaf(lam1, sgv.x, w_mu * m.x), s1 = fmaf(lam1, sgv.y, w_mu * m.y);
      const float s2 = fmaf(lam1, sgv.z, w_mu * m.z), s3 = fmaf(lam1, sgv.w, w_mu * m.w);
      local_max = fmaxf(fmaxf(local_max, fmaxf(s0, s1)), fmaxf(s2, s3));
      const int i = head + 4 * v;
      skeys[i] = order_key(s0);
      skeys[i + 1] = order_key(s1);
      skeys[i + 2] = order_key(s2);
      skeys[i + 3] = order_key(s3);
    }
    for (int i = head + 4 * n4 + tid; i < n_cand; i += kThreads) {
      const float sv = fmaf(lam1, sg_g[i], w_mu * mu_g[i]);
      local_max = fmaxf(local_max, sv);
      skeys[i] = order_key(sv);
    }
    __syncthreads();
  } else {
    for (int i = tid; i < n_cand; i += kThreads)
      local_max = fmaxf(local_max, fmaf(lam1, sg_g[i], w_mu * mu_g[i]));
  }
  // Max-pooling keeps the largest score of the window, whose key is also the largest key.
  if constexpr (STAGED) {
    if (pool_h > 0) {
      // In place, a chunk of kPer * kThreads positions at a time: pooled keys of the chunk go to
      // registers, the raw keys of its last pool_h positions to a halo that the next chunk reads
      // instead of the (by then overwritten) chunk, then the chunk is overwritten.
      constexpr int kPer = 8, kChunk = kPer * kThreads;
      for (int c0 = 0, c = 0; c0 < n_cand; c0 += kChunk, ++c) {
        const int c1 = min(n_cand, c0 + kChunk);
        const uint32_t* halo_in = sh.halo[c & 1];  // positions c0 - pool_h .. c0 - 1
        uint32_t pk[kPer];
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
          const int i = c0 + q * kThreads + tid;
          uint32_t m = 0u;
          if (i < c1) {
            const int j1 = min(n_cand - 1, i + pool_h);
            for (int j = max(0, i - pool_h); j <= j1; ++j)
              m = max(m, j < c0 ? halo_in[j - (c0 - pool_h)] : skeys[j]);
          }
          pk[q] = m;
        }
        if (tid < pool_h && c1 < n_cand) sh.halo[(c + 1) & 1][tid] = skeys[c1 - pool_h + tid];
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
          const int i = c0 + q * kThreads + tid;
          if (i < c1) skeys[i] = pk[q];
        }
      }
      __syncthreads();
    }
  }
  // key of the (pooled) score at position i
  auto key_at = [&](int i) -> uint32_t {
    if constexpr (STAGED) {
      return skeys[i];
    } else {
      uint32_t kmax = order_key(fmaf(lam1, sg_g[i], w_mu * mu_g[i]));
      if (pool_h > 0) {
        const int j1 = min(n_cand - 1, i + pool_h);
        for (int j = max(0, i - pool_h); j <= j1; ++j)
          kmax = max(kmax, order_key(fmaf(lam1, sg_g[j], w_mu * mu_g[j])));
      }
      return kmax;
    }
  };
  {
    const float wm = wave_max_f(local_max);
    if (lane == 0) sh.wave_max[wave] = wm;
  }

  // ---- 1. the C-th largest key: most-significant-digit radix select ---------------------------
  uint32_t prefix = 0, pmask = 0;
  int need = C;
  for (int pass = 0; pass < (take_all ? 0 : 4); ++pass) {
    const int shift = 24 - 8 * pass;
    for (int i = tid; i < kWaves * 256; i += kThreads) (&sh.hist[0][0])[i] = 0u;
    __syncthreads();
    const int n_iter = (n_cand + 4 * kThreads - 1) / (4 * kThreads);
    for (int it = 0; it < n_iter; ++it) {
      uint32_t kk[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {  // four independent reads in flight
        const int i = (4 * it + q) * kThreads + tid;
        kk[q] = i < n_cand ? key_at(i) : 0u;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = (4 * it + q) * kThreads + tid;
        wave_hist_add(sh.hist[wave], (kk[q] >> shift) & 255u, i < n_cand && (kk[q] & pmask) == prefix);
      }
    }
    __syncthreads();
    // suffix sums over bins (bin 255 = largest digit); thread tid < 256 (waves 0..3) holds bin
    // tid: a suffix scan inside each wave, then the totals of the waves above it
    const bool bin = tid < 256;
    uint32_t cnt = 0, suf = 0;
    if (bin) {
#pragma unroll
      for (int v = 0; v < kWaves; ++v) cnt += sh.hist[v][tid];
      suf = cnt;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t o = __shfl_down(suf, off, 64);
        if (lane + off < 64) suf += o;
      }
      if (lane == 0) sh.scan[wave] = suf;
    }
    __syncthreads();
    if (bin) {
      uint32_t above = 0;
      for (int v = wave + 1; v < 4; ++v) above += sh.scan[v];
      const uint32_t ge = suf + above;  // count with digit >= tid
      const uint32_t gt = ge - cnt;     // count with digit > tid
      if (ge >= (uint32_t)need && gt < (uint32_t)need) {
        sh.sel_threshold = prefix | ((uint32_t)tid << shift);
        sh.sel_need = need - (int)gt;
      }
    }
    __syncthreads();
    prefix = sh.sel_threshold;
    need = sh.sel_need;
    pmask |= 255u << shift;
    __syncthreads();
  }
  __syncthreads();
  float den = sh.wave_max[0];
#pragma unroll
  for (int v = 1; v < kWaves; ++v) den = fmaxf(den, sh.wave_max[v]);
  den = fmaxf(den, 1e-12f);

  // ---- 2. candidate positions in ascending order ----------------------------------------------
  // key > threshold: taken; key == threshold: the `need` lowest positions are taken.
  {
    const uint32_t thr = prefix;
    const int per_wave = (n_cand + kWaves - 1) / kWaves;
    const int w0 = wave * per_wave, w1 = min(n_cand, w0 + per_wave);
    uint32_t n_gt = 0, n_eq = 0;
    for (int i0 = w0; i0 < w1; i0 += 256) {
      uint32_t kk[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + 64 * q + lane;
        kk[q] = (i < w1 && !take_all) ? key_at(i) : 0u;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bool in = i0 + 64 * q + lane < w1;
        n_gt += __popcll(__ballot(in && (take_all || kk[q] > thr)));
        n_eq += __popcll(__ballot(in && !take_all && kk[q] == thr));
      }
    }
    if (lane == 0) {
      sh.wave_cnt[0][wave] = n_gt;
      sh.wave_cnt[1][wave] = n_eq;
    }
    __syncthreads();
    uint32_t out = 0, eq_before = 0;
    for (int v = 0; v < wave; ++v) {
      const uint32_t eq_v = sh.wave_cnt[1][v];
      const uint32_t eq_taken = eq_before >= (uint32_t)need ? 0u : min(eq_v, (uint32_t)need - eq_before);
      out += sh.wave_cnt[0][v] + eq_taken;
      eq_before += eq_v;
    }
    const uint64_t lanes_below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int i0 = w0; i0 < w1; i0 += 256) {
      uint32_t kk[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + 64 * q + lane;
        kk[q] = (i < w1 && !take_all) ? key_at(i) : 0u;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {  // blocks of 64 in ascending position order
        const int i = i0 + 64 * q + lane;
        const bool in = i < w1;
        const bool is_gt = in && (take_all || kk[q] > thr);
        const bool is_eq = in && !take_all && kk[q] == thr;
        const uint64_t eqm = __ballot(is_eq);
        const uint32_t eq_rank = eq_before + (uint32_t)__popcll(eqm & lanes_below);
        const bool taken = is_gt || (is_eq && eq_rank < (uint32_t)need);
        const uint64_t tm = __ballot(taken);
        const uint32_t slot = out + (uint32_t)__popcll(tm & lanes_below);
        if (taken && slot < (uint32_t)C) cpos[slot] = i;
        out += (uint32_t)__popcll(tm);
        eq_before += (uint32_t)__popcll(eqm);
      }
    }
  }
  __syncthreads();  // the staged score keys are dead from here on: the region takes key rows

  // ---- 3. greedy admission -------------------------------------------------------------------
  KeyRow<DT, D> key[CPT];
  float st[CPT], corr[CPT], inv[CPT];
  bool admitted[CPT];
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int c = tid + q * kThreads;
    admitted[q] = c >= C;  // slots beyond C never compete
    corr[q] = 0.f;
    st[q] = 0.f;
    inv[q] = 0.f;
    if (c < C) {
      const int pos = cpos[c];
      key[q].load(kg + (size_t)pos * D);
      key[q].store(ckeys + (size_t)c * D);
      const float n2 = key[q].sq_norm();
      inv[q] = n2 > 0.f ? 1.f / sqrtf(n2) : 0.f;  // a zero key has cosine 0 to everything
      cinv[c] = inv[q];
      float sv = fmaf(lam1, sg_g[pos], w_mu * mu_g[pos]);
      for (int j = max(0, pos - pool_h); j <= min(n_cand - 1, pos + pool_h); ++j)
        sv = fmaxf(sv, fmaf(lam1, sg_g[j], w_mu * mu_g[j]));
      st[q] = sv / den;
    }
  }
  __syncthreads();

  int last = -1;
  float last_inv = 0.f;
  // the greedy trace (admitted slot and score key per step) reuses the radix histograms: at most
  // C <= 2 NT steps (2 NT = 128 NW words each)
  uint32_t* trace_slot = &sh.hist[0][0];
  uint32_t* trace_key = &sh.hist[0][0] + kWaves * 128;
  // only the waves that own candidate slots take part; the others just keep step with the
  // barrier (sleeping there instead of taking issue slots from the live waves)
  const int live_waves = min(kWaves, (C + 63) / 64);
  const bool live = wave < live_waves;
  for (int t = 0; t < bp; ++t) {
    if (live) {
      float my_score = -INFINITY;  // admitted slots rank below every live score
      int my_slot = 0x7FFFFFFF;
#pragma unroll
      for (int q = 0; q < CPT; ++q) {
        if (!admitted[q]) {
          if (last >= 0) {
            const float cs = key[q].dot_lds(ckeys + (size_t)last * D) * inv[q] * last_inv;
            corr[q] = fmaxf(corr[q], cs);
          }
          float sc = fmaf(lam2, corr[q], st[q]);
          if (!(sc > -INFINITY)) sc = -FLT_MAX;  // NaN or -inf still ranks above admitted slots
          if (sc > my_score) {  // q ascending: ties keep the lower slot
            my_score = sc;
            my_slot = tid + q * kThreads;
          }
        }
      }
      const uint64_t wbest = wave_best<CPT == 1>(my_score, my_slot);
      // the wave's best slot is owned by one of its lanes (slot = tid + q NT): its 1 / |k| rides
      // along, so that no lookup follows the barrier
      const int bslot = unpack_slot(wbest);
      float binv = 0.f;
#pragma unroll
      for (int q = 0; q < CPT; ++q) {
        const uint32_t v = __builtin_amdgcn_readlane(__float_as_uint(inv[q]), bslot & 63);
        if ((bslot - q * kThreads) >> 6 == wave) binv = __uint_as_float(v);
      }
      if (lane == 0)
        sh.best[t & 1][wave] = make_uint4((uint32_t)wbest, (uint32_t)(wbest >> 32), __float_as_uint(binv), 0u);
    }
    __syncthreads();
    if (live) {
      // the live waves' records (score key, slot, 1 / |k|), four reads in flight at a time
      uint64_t b = 0;
      float bi = 0.f;
      for (int v0 = 0; v0 < live_waves; v0 += 4) {
        // records past the live waves are read (v0 + 3 < NW) but never win
        uint4 r[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) r[u] = sh.best[t & 1][v0 + u];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint64_t o = v0 + u < live_waves ? ((uint64_t)r[u].y << 32) | r[u].x : 0ull;
          if (o > b) {
            b = o;
            bi = __uint_as_float(r[u].z);
          }
        }
      }
      last = min(max(unpack_slot(b), 0), C - 1);  // always a live slot: bp <= C
#pragma unroll
      for (int q = 0; q < CPT; ++q)
        if (tid + q * kThreads == last) admitted[q] = true;
      last_inv = bi;
      if (tid == 0) {  // the step's record; written out after the last step
        trace_slot[t] = (uint32_t)last;
        trace_key[t] = (uint32_t)(b >> 32);
      }
    }
  }
  __syncthreads();
  for (int t = tid; t < bp; t += kThreads) {
    const size_t o = ((size_t)p * h_kv + g) * budget + t;
    sel_idx[o] = cpos[trace_slot[t]];
    if (sel_score) {
      const uint32_t kk = trace_key[t];
      const uint32_t u = (kk & 0x80000000u) ? (kk & 0x7FFFFFFFu) : ~kk;
      sel_score[o] = __uint_as_float(u);
    }
  }

  // steps beyond this problem's budget: padding
  for (int t = bp + tid; t < budget; t += kThreads) {
    const size_t o = ((size_t)p * h_kv + g) * budget + t;
    sel_idx[o] = -1;
    if (sel_score) sel_score[o] = 0.f;
  }

  if (cand_idx || cand_corr) {
    // corr after the last step includes the last admitted key
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
      if (!admitted[q]) {
        const float cs = key[q].dot_lds(ckeys + (size_t)last * D) * inv[q] * last_inv;
        corr[q] = fmaxf(corr[q], cs);
      }
    }
    const size_t o = ((size_t)p * h_kv + g) * cand_stride;
#pragma unroll
    for (int q = 0; q < CPT; ++q) {
      const int c = tid + q * kThreads;
      if (c < cand_stride) {
        if (cand_idx) cand_idx[o + c] = c < C ? cpos[c] : -1;
        if (cand_corr) cand_corr[o + c] = c < C ? corr[q] : 0.f;
      }
    }
    for (int c = tid + CPT * kThreads; c < cand_stride; c += kThreads) {
      if (cand_idx) cand_idx[o + c] = -1;
      if (cand_corr) cand_corr[o + c] = 0.f;
    }
  }

  if (co.k_out) {
    // the unit's compacted rows: the admitted positions sorted in the key-row region (dead once
    // the last candidate has read it), then the rows copied as in compact.hip
    int32_t* srt = reinterpret_cast<int32_t*>(region);
    int n2 = 1;
    while (n2 < bp) n2 <<= 1;
    __syncthreads();
    for (int i = tid; i < n2; i += kThreads) srt[i] = i < bp ? cpos[trace_slot[i]] : INT_MAX;
    __syncthreads();
    sort_positions(srt, n2, tid, kThreads);
    constexpr int kRowVecs = D * (int)sizeof(T) / 16;
    copy_kept_rows(co.k, co.v, srt, bp, keep_tail, L, kRowVecs, base * kRowVecs,
                   ((size_t)p * h_kv + g) * co.out_rows * kRowVecs, co.k_out, co.v_out, tid,
                   kThreads);
  }
}

// ------------------------------------------------------------------------------------------------
int select_max_candidates(int d, int elem_bytes) {
  const int by_lds = kMaxCandBytes / (d * elem_bytes);
  const int by_regs = elem_bytes == 2 ? 1024 : 4 * 256;  // candidate slots of the workgroup
  return by_lds < by_regs ? by_lds : by_regs;
}

namespace {
template <int DT, int D, int NT, int CPT, bool STAGED>
hipError_t select_launch(const Shape& s, const SelectArgs& a, hipStream_t st) {
  using T = typename Elem<DT>::T;
  const size_t region = std::max((size_t)a.max_cand * D * sizeof(T),
                                 STAGED ? (size_t)a.max_cand_all * 4 : (size_t)0);
  const size_t dyn = (((size_t)a.max_cand * 8 + 15) & ~(size_t)15) + region;
  auto kern = mmr_select_kernel<DT, D, NT, CPT, STAGED>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  kern<<<dim3((unsigned)(s.n_prob * s.h_kv)), NT, dyn, st>>>(
      a.mu, a.sigma, static_cast<const T*>(a.k), s.lens, s.tok_off, a.lambda1, a.lambda2,
      a.pool / 2, a.w_mu, s.h_kv,
      a.budget, a.budgets, a.cand_mult, a.keep_tail, a.cand_stride, a.max_cand, a.sel_idx, a.sel_score,
      a.cand_idx, a.cand_corr,
      CompactOut{static_cast<const uint4*>(a.k), static_cast<const uint4*>(a.v),
                 static_cast<uint4*>(a.k_out), static_cast<uint4*>(a.v_out), a.out_rows});
  return hipGetLastError();
}

// Score keys are staged in LDS when every problem's candidates fit next to the key rows (and the
// whole workgroup's LDS stays within the 160 KiB of a CU).
template <int DT, int D, int NT, int CPT>
hipError_t select_dispatch(const Shape& s, const SelectArgs& a, hipStream_t st) {
  using T = typename Elem<DT>::T;
  const size_t rows = (size_t)a.max_cand * D * sizeof(T);
  const size_t staged = (((size_t)a.max_cand * 8 + 15) & ~(size_t)15) +
                        std::max(rows, (size_t)a.max_cand_all * 4) + sizeof(SelectShared<NT / 64>);
  if ((size_t)a.max_cand_all * 4 <= (size_t)kMaxStagedKeyBytes && staged <= kLdsBytes)
    return select_launch<DT, D, NT, CPT, true>(s, a, st);
  return select_launch<DT, D, NT, CPT, false>(s, a, st);
}

template <int DT, int D>
hipError_t select_cpt(const Shape& s, const SelectArgs& a, hipStream_t st) {
  constexpr int kMaxCand = kMaxCandBytes / (D * (int)sizeof(typename Elem<DT>::T));
  if constexpr (DT == kDtBf16) {
    // bf16 key rows fit the registers of 16 waves: one candidate per thread of 1024
    static_assert(kMaxCand <= 1024, "one candidate per thread");
    return select_dispatch<DT, D, 1024, 1>(s, a, st);
  } else {
    // only the candidates-per-thread counts that the LDS key copy allows are instantiated
    constexpr int kNT = 256;
    const int cpt = (a.max_cand + kNT - 1) / kNT;
    if (cpt <= 1) return select_dispatch<DT, D, kNT, 1>(s, a, st);
    if constexpr (kMaxCand > kNT) {
      if (cpt <= 2) return select_dispatch<DT, D, kNT, 2>(s, a, st);
    }
    if constexpr (kMaxCand > 2 * kNT) return select_dispatch<DT, D, kNT, 4>(s, a, st);
    return hipErrorInvalidValue;
  }
}
}  // namespace

hipError_t launch_mmr_select(const Shape& s, const SelectArgs& a, hipStream_t stream) {
  if (s.dtype == kDtBf16)
    return s.d == 64 ? select_cpt<kDtBf16, 64>(s, a, stream) : select_cpt<kDtBf16, 128>(s, a, stream);
  return s.d == 64 ? select_cpt<kDtF32, 64>(s, a, stream) : select_cpt<kDtF32, 128>(s, a, stream);
}

}  // namespace kv
