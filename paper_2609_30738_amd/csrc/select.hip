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
//   3. B greedy steps, in one of two ways:
//      - Gram (bf16, C <= 256; select_gram.h): the candidates' key rows are staged in LDS, the
//        cosines of every candidate pair formed once with MFMA tiles into a strict upper triangle
//        in LDS; then ONE wave runs every step, each lane holding up to four candidates' s~ and
//        running max-cosine: a step reads one triangle entry per candidate against the last
//        admitted slot and takes a DPP / permlane maximum, with no barrier;
//      - rows (larger C): thread t owns candidates t, t + NT, ... and keeps their keys in
//        registers; each step updates the running maxima against the last admitted key (read from
//        an LDS copy of the candidate keys), forms s~ + lambda2 * corr, and finds the (score,
//        lowest slot) maximum: a DPP / permlane maximum and a ballot inside each wave, then one
//        barrier; the per-wave winners are double-buffered so that one barrier per step suffices.
#include <float.h>

#include <algorithm>

#include "common.h"
#include "compact_rows.h"
#include "kernels.h"
#include "select_gram.h"

namespace kv {

namespace {

constexpr int kMaxCandBytes = 131072;        // LDS copy of the candidate keys
constexpr int kMaxStagedKeyBytes = 139264;  // LDS copy of every candidate's score key (34816)
constexpr size_t kLdsBytes = 163840;        // LDS of one CU
constexpr int kMaxSlotWords = 64;           // bitmap words over the candidate slots (C <= 2048)

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

// Append the positions of the lanes where `pred` holds to out[] at slots taken from *counter
// (one LDS atomic per wave); the order of the appended entries is unspecified.
template <typename F>
__device__ __forceinline__ void wave_append(bool pred, uint32_t* counter, int lane, F&& write) {
  const uint64_t m = __ballot(pred);
  if (m == 0) return;
  const int leader = __ffsll((unsigned long long)m) - 1;
  uint32_t base = 0;
  if (lane == leader) base = atomicAdd(counter, (uint32_t)__popcll(m));
  base = __builtin_amdgcn_readlane(base, leader);
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  if (pred) write(base + (uint32_t)__popcll(m & below));
}

// Add one to hist[digit] (LDS) for every active lane, with few colliding atomics where most keys
// share one bin (the bulk of the scores, which holds about three in four keys of the workloads
// here): the wave's `hot` digit (the largest bin of its earlier calls) is counted with one ballot
// and one atomic, then the digit of the first lane left likewise, and only the lanes left after
// that add one each.  Every lane of the wave must call it; `hot` is wave-uniform.
__device__ __forceinline__ void wave_hist_add_hot(uint32_t* hist, uint32_t digit, bool active,
                                                  uint32_t& hot, int lane) {
  uint64_t rem = __ballot(active);
  if (rem == 0) return;
  const uint64_t s1 = __ballot(active && digit == hot);
  if (s1 != 0 && lane == __ffsll((unsigned long long)s1) - 1) atomicAdd(&hist[hot], (uint32_t)__popcll(s1));
  rem &= ~s1;
  if (rem == 0) return;
  const int leader = __ffsll((unsigned long long)rem) - 1;
  const uint32_t dl = __builtin_amdgcn_readlane(digit, leader);
  const uint64_t s2 = __ballot(digit == dl) & rem;
  if (lane == leader) atomicAdd(&hist[dl], (uint32_t)__popcll(s2));
  rem &= ~s2;
  if (__popcll(s2) > __popcll(s1)) hot = dl;
  if ((rem >> lane) & 1ull) atomicAdd(&hist[digit], 1u);
}

constexpr int kFastBins = 2048;  // 11-bit digit
constexpr int kFastShift = 21;
constexpr int kListCap = 1024;   // members of the cut's bin ranked exactly

// The candidate positions (C of the n_cand staged keys, the largest keys, ties to the lower
// position) in ascending order into cpos, when the bin of the C-th largest key under an 11-bit
// digit holds at most kListCap keys; returns false (having written nothing the general path
// reads) otherwise.  Uses the radix histograms' space; starts and ends synchronised.
template <int NW>
__device__ bool fast_candidates(SelectShared<NW>& sh, const uint32_t* skeys, int32_t* cpos,
                                int n_cand, int C, int tid, int lane, int wave) {
  constexpr int NT = NW * 64;
  static_assert(NT * 2 == kFastBins, "two bins per thread");
  static_assert(sizeof(sh.hist) >= kFastBins * 4 + kListCap * 8, "histogram and list space");
  uint32_t* h = &sh.hist[0][0];
  uint64_t* list = reinterpret_cast<uint64_t*>(h + kFastBins);
  for (int i = tid; i < kFastBins; i += NT) h[i] = 0u;
  if (tid < 2) sh.wave_cnt[0][tid] = 0u;  // append counters: candidates above the bin, list
  __syncthreads();
  uint32_t hot = ~0u;  // no digit yet
  for (int i0 = 0; i0 < n_cand; i0 += 4 * NT) {
    uint32_t kk[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + q * NT + tid;
      kk[q] = i < n_cand ? skeys[i] : 0u;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q)
      wave_hist_add_hot(h, kk[q] >> kFastShift, i0 + q * NT + tid < n_cand, hot, lane);
  }
  __syncthreads();
  // suffix sums over the bins (larger bins = larger keys): thread t owns bins 2t, 2t + 1
  const uint32_t c0 = h[2 * tid], c1 = h[2 * tid + 1];
  uint32_t suf = c0 + c1;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_down(suf, off, 64);
    if (lane + off < 64) suf += o;
  }
  if (lane == 0) sh.scan[wave] = suf;
  __syncthreads();
  uint32_t above = 0;
  for (int v = wave + 1; v < NW; ++v) above += sh.scan[v];
  const uint32_t gt_hi = suf - (c0 + c1) + above;  // keys in bins above 2t + 1
  const uint32_t gt_lo = gt_hi + c1;               // keys in bins above 2t
  if (gt_hi < (uint32_t)C && gt_hi + c1 >= (uint32_t)C) {
    sh.sel_threshold = 2 * tid + 1;
    sh.sel_need = C - (int)gt_hi;
    sh.wave_cnt[1][0] = c1;
  }
  if (gt_lo < (uint32_t)C && gt_lo + c0 >= (uint32_t)C) {
    sh.sel_threshold = 2 * tid;
    sh.sel_need = C - (int)gt_lo;
    sh.wave_cnt[1][0] = c0;
  }
  __syncthreads();
  const uint32_t bin = sh.sel_threshold;
  const int need = sh.sel_need;
  const int members = (int)sh.wave_cnt[1][0];
  if (members > kListCap) return false;
  // every key above the bin is a candidate (C - need of them, any order); the bin's members go
  // to the list as (~key, position): ascending order is the key descending, then the position
  for (int i0 = 0; i0 < n_cand; i0 += 4 * NT) {
    uint32_t kk[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + q * NT + tid;
      kk[q] = i < n_cand ? skeys[i] : 0u;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int i = i0 + q * NT + tid;
      const bool in = i < n_cand;
      wave_append(in && (kk[q] >> kFastShift) > bin, &sh.wave_cnt[0][0], lane,
                  [&](uint32_t slot) { cpos[slot] = i; });
      wave_append(in && (kk[q] >> kFastShift) == bin, &sh.wave_cnt[0][1], lane,
                  [&](uint32_t slot) { list[slot] = ((uint64_t)(~kk[q]) << 32) | (uint32_t)i; });
    }
  }
  int n2 = 1;
  while (n2 < members) n2 <<= 1;
  for (int i = members + tid; i < n2; i += NT) list[i] = ~0ull;
  __syncthreads();
  bitonic_sort(list, n2, tid, NT);
  // the candidates in ascending position order: a bitmap over the positions (the histogram's
  // space, free again: n_cand <= kMaxStagedKeyBytes / 4 positions), then each thread writes the
  // set positions of its words at its offset
  uint32_t* bits = h;
  constexpr int kWords = kMaxStagedKeyBytes / 4 / 32;
  static_assert(kWords * 4 <= kFastBins * 4, "bitmap space");
  const int words = (n_cand + 31) / 32;
  for (int w = tid; w < words; w += NT) bits[w] = 0u;
  __syncthreads();
  for (int t = tid; t < C; t += NT) {
    const int pos = t < C - need ? cpos[t] : (int32_t)(uint32_t)list[t - (C - need)];
    atomicOr(&bits[pos >> 5], 1u << (pos & 31));
  }
  __syncthreads();
  // words [per * tid, per * tid + per) belong to thread tid
  const int per = (words + NT - 1) / NT;
  uint32_t cnt = 0;
  for (int w = per * tid; w < min(words, per * tid + per); ++w) cnt += __popc(bits[w]);
  uint32_t incl = cnt;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) sh.scan[wave] = incl;
  __syncthreads();
  uint32_t out = incl - cnt;
  for (int v = 0; v < wave; ++v) out += sh.scan[v];
  for (int w = per * tid; w < min(words, per * tid + per); ++w) {
    uint32_t m = bits[w];
    while (m) {
      const int b = __ffs(m) - 1;
      cpos[out++] = 32 * w + b;
      m &= m - 1;
    }
  }
  __syncthreads();
  return true;
}

// Compaction after the selection (k_out == nullptr: none); K, V, outputs as 16-byte vectors.
struct CompactOut {
  const uint4* k;
  const uint4* v;
  uint4* k_out;
  uint4* v_out;
  int out_rows;
};

}  // namespace

template <int DT, int D, int NT, int CPT, bool STAGED, bool GRAM>
__global__ __launch_bounds__(NT) void mmr_select_kernel(
    const float* __restrict__ mu, const float* __restrict__ sigma,
    const float* __restrict__ score, const uint64_t* __restrict__ cand_in,
    const float* __restrict__ cand_in_max, uint64_t* __restrict__ cut_out,
    float* __restrict__ cut_max, int list_stride,
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
  // dynamic LDS: [max_cand] positions, [max_cand] 1/|k|, [max_cand] s~ (Gram greedy), then a region
  // that first holds the order-preserving keys of every candidate score (STAGED) and then the
  // candidates' key rows or (GRAM) the triangle of their dot products
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
  // no lambda1 with scores given, no lambda2 for the candidate cut alone
  const float lam1 = lambda1 ? lambda1[p] : 0.f, lam2 = lambda2 ? lambda2[p] : 0.f;
  const float* sc_g = score ? score + base : nullptr;  // base scores given: mu / sigma unused
  // base score of candidate position i
  auto base_score = [&](int i) -> float {
    return sc_g ? sc_g[i] : fmaf(lam1, sg_g[i], w_mu * mu_g[i]);
  };
  const T* kg = k + base * D;
  int32_t* cpos = reinterpret_cast<int32_t*>(dyn);
  float* cinv = reinterpret_cast<float*>(dyn + (size_t)max_cand * 4);
  float* cst = reinterpret_cast<float*>(dyn + (size_t)max_cand * 8);
  unsigned char* region = dyn + (((size_t)max_cand * 12 + 15) & ~(size_t)15);
  uint32_t* skeys = reinterpret_cast<uint32_t*>(region);
  T* ckeys = reinterpret_cast<T*>(region);
  const bool take_all = (C >= n_cand);
  float den = 0.f;
  if (cand_in) {
    // ---- 0-2 from a candidate list: the unit's C candidates (order key of the score, position)
    //      in ascending position order
    const uint64_t* src = cand_in + (size_t)blockIdx.x * list_stride;
    for (int i = tid; i < C; i += kThreads) {
      const uint64_t e = src[i];
      cpos[i] = (int32_t)cand_entry_pos(e);
      cst[i] = key_float((uint32_t)(e >> 32));
    }
    den = cand_in_max[blockIdx.x];
    __syncthreads();
  } else {

  // ---- 0. base scores s_i = mu_i + lambda1 sigma_i (one rounding, or given) and their maximum -
  float local_max = -INFINITY;
  if constexpr (STAGED) {
    // the rows start at a multiple of 4 floats only if base is; stage element-wise until the
    // first aligned index, then 4 per lane with several loads in flight
    const int head = (int)((4 - (base & 3)) & 3) < n_cand ? (int)((4 - (base & 3)) & 3) : n_cand;
    if (tid < head) {
      const float sv = base_score(tid);
      local_max = fmaxf(local_max, sv);
      skeys[tid] = order_key(sv);
    }
    const int n4 = (n_cand - head) / 4;
    auto stage4 = [&](int v, float s0, float s1, float s2, float s3) {
      local_max = fmaxf(fmaxf(local_max, fmaxf(s0, s1)), fmaxf(s2, s3));
      const int i = head + 4 * v;
      skeys[i] = order_key(s0);
      skeys[i + 1] = order_key(s1);
      skeys[i + 2] = order_key(s2);
      skeys[i + 3] = order_key(s3);
    };
    if (sc_g) {
      const float4* sc4 = reinterpret_cast<const float4*>(sc_g + head);
#pragma unroll 4
      for (int v = tid; v < n4; v += kThreads) {
        const float4 sv = sc4[v];
        stage4(v, sv.x, sv.y, sv.z, sv.w);
      }
    } else {
      const float4* mu4 = reinterpret_cast<const float4*>(mu_g + head);
      const float4* sg4 = reinterpret_cast<const float4*>(sg_g + head);
#pragma unroll 4
      for (int v = tid; v < n4; v += kThreads) {
        const float4 m = mu4[v], sgv = sg4[v];
        stage4(v, fmaf(lam1, sgv.x, w_mu * m.x), fmaf(lam1, sgv.y, w_mu * m.y),
               fmaf(lam1, sgv.z, w_mu * m.z), fmaf(lam1, sgv.w, w_mu * m.w));
      }
    }
    for (int i = head + 4 * n4 + tid; i < n_cand; i += kThreads) {
      const float sv = base_score(i);
      local_max = fmaxf(local_max, sv);
      skeys[i] = order_key(sv);
    }
    __syncthreads();
  } else {
    for (int i = tid; i < n_cand; i += kThreads) local_max = fmaxf(local_max, base_score(i));
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
      uint32_t kmax = order_key(base_score(i));
      if (pool_h > 0) {
        const int j1 = min(n_cand - 1, i + pool_h);
        for (int j = max(0, i - pool_h); j <= j1; ++j) kmax = max(kmax, order_key(base_score(j)));
      }
      return kmax;
    }
  };
  {
    const float wm = wave_max_f(local_max);
    if (lane == 0) sh.wave_max[wave] = wm;
  }

  // ---- 1a. fast front end (staged keys, 1024 threads): one 11-bit histogram of the keys finds
  //      the bin of the C-th largest; every key above that bin is a candidate, and the bin's own
  //      members (a few hundred where salient tokens set the cut) are sorted exactly, by key and then
  //      position, in LDS.  The candidates are then sorted by position.  A bin too full for the
  //      list (a cut through the flat bulk of the scores) takes the general path below.
  bool fast_done = false;
  if constexpr (STAGED && NT == 1024) {
    if (!take_all) fast_done = fast_candidates<kWaves>(sh, skeys, cpos, n_cand, C, tid, lane, wave);
  }

  // ---- 1. the C-th largest key: most-significant-digit radix select ---------------------------
  uint32_t prefix = 0, pmask = 0;
  int need = C;
  for (int pass = 0; pass < (take_all || fast_done ? 0 : 4); ++pass) {
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
  den = sh.wave_max[0];
#pragma unroll
  for (int v = 1; v < kWaves; ++v) den = fmaxf(den, sh.wave_max[v]);
  den = fmaxf(den, 1e-12f);

  // ---- 2. candidate positions in ascending order ----------------------------------------------
  // key > threshold: taken; key == threshold: the `need` lowest positions are taken.
  if (!fast_done) {
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
  __syncthreads();
  if (cut_out) {
    // the candidate list of a unit for the selection from a list: the C candidates in position
    // order, then nothing
    uint64_t* dst = cut_out + (size_t)blockIdx.x * list_stride;
    for (int i = tid; i < list_stride; i += kThreads)
      dst[i] = i < C ? cand_entry(order_key(base_score(cpos[i])), (uint32_t)cpos[i]) : 0ull;
    if (tid == 0) cut_max[blockIdx.x] = den;
    return;
  }
  }  // phases 0-2
  __syncthreads();  // the staged score keys are dead from here on: the region takes key rows

  // ---- 3. greedy admission -------------------------------------------------------------------
  // the greedy trace (admitted slot and score key per step) reuses the radix histograms: at most
  // C <= 2 NT steps (2 NT = 128 NW words each)
  uint32_t* trace_slot = &sh.hist[0][0];
  uint32_t* trace_key = &sh.hist[0][0] + kWaves * 128;
  int last = -1;
  if constexpr (GRAM) {
    static_assert(DT == kDtBf16, "the Gram greedy takes bf16 keys");
    // s~ of every candidate (its base score, pooled as in phase 0, over the normaliser)
    for (int c = tid; c < C; c += kThreads) {
      const int pos = cpos[c];
      float sv;
      if (cand_in) {
        sv = cst[c];  // the entry's score (no pooling with candidate lists)
      } else {
        sv = base_score(pos);
        for (int j = max(0, pos - pool_h); j <= min(n_cand - 1, pos + pool_h); ++j)
          sv = fmaxf(sv, base_score(j));
      }
      cst[c] = sv / den;
    }
    gram::cosines<D, kWaves>(kg, cpos, C, cinv, region, tid);
    const float* tri = reinterpret_cast<const float*>(region) + 1;
    if (wave == 0) {
      gram::Greedy gr;
      gr.init(cst, C, lane);
      if (sel_score) gr.run_for<true>(tri, C, bp, lam2, lane, trace_slot, trace_key);
      else gr.run_for<false>(tri, C, bp, lam2, lane, trace_slot, trace_key);
      last = gr.last;
      if (cand_idx || cand_corr) {
        // an admitted slot reports its corr at admission: the largest of 0 and its cosines to the
        // slots admitted before it (the same maximum the steps formed); the slot of s~ keeps it
        float* corr_adm = cst;
        for (int t = lane; t < bp; t += 64) {
          const int si = (int)trace_slot[t];
          float m = 0.f;
          for (int u = 0; u < t; ++u) {
            const int su = (int)trace_slot[u];
            m = __builtin_elementwise_maximum(m, tri[gram::row_off(min(si, su), C) + max(si, su)]);
          }
          corr_adm[si] = m;
        }
        // corr after the last step includes the last admitted key
        const size_t o = ((size_t)p * h_kv + g) * cand_stride;
        float gl[gram::kSlots];
        gr.cos_to(tri, last, C, gl);
#pragma unroll
        for (int q = 0; q < gram::kSlots; ++q) {
          const int c = lane + 64 * q;
          float cr = 0.f;
          if (c < C) {
            const bool adm = gr.st[q] == -INFINITY;
            cr = adm ? corr_adm[c] : __builtin_elementwise_maximum(gr.corr[q], gl[q]);
          }
          if (c < cand_stride) {
            if (cand_idx) cand_idx[o + c] = c < C ? cpos[c] : -1;
            if (cand_corr) cand_corr[o + c] = cr;
          }
        }
      }
    }
    if (cand_idx || cand_corr) {
      const size_t o = ((size_t)p * h_kv + g) * cand_stride;
      for (int c = gram::kSlots * 64 + tid; c < cand_stride; c += kThreads) {
        if (cand_idx) cand_idx[o + c] = -1;
        if (cand_corr) cand_corr[o + c] = 0.f;
      }
    }
    __syncthreads();
  } else {
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
        float sv;
        if (cand_in) {
          sv = cst[c];  // the entry's score (no pooling with candidate lists)
        } else {
          sv = base_score(pos);
          for (int j = max(0, pos - pool_h); j <= min(n_cand - 1, pos + pool_h); ++j)
            sv = fmaxf(sv, base_score(j));
        }
        st[q] = sv / den;
      }
    }
    __syncthreads();

    float last_inv = 0.f;
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

  if (co.k_out) {
    // the unit's compacted rows: the admitted positions in ascending order, then the rows copied
    // as in compact.hip.  The candidates are in position order, so the admitted slots in ascending
    // order give the positions in ascending order: a bitmap over the slots and the prefix counts of
    // its words rank them (in the key-row region, dead once the last candidate has read it).
    static_assert(kMaxSlotWords <= 64, "one bitmap word per lane of a wave");
    uint32_t* bits = reinterpret_cast<uint32_t*>(region);
    uint32_t* pre = bits + kMaxSlotWords;
    int32_t* srt = reinterpret_cast<int32_t*>(pre + kMaxSlotWords);
    const int words = (C + 31) >> 5;
    __syncthreads();
    for (int w = tid; w < words; w += kThreads) bits[w] = 0u;
    __syncthreads();
    for (int t = tid; t < bp; t += kThreads)
      atomicOr(&bits[trace_slot[t] >> 5], 1u << (trace_slot[t] & 31));
    __syncthreads();
    if (wave == 0) {
      const uint32_t v = lane < words ? (uint32_t)__popc(bits[lane]) : 0u;
      uint32_t incl = v;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t o = (uint32_t)__shfl_up((int)incl, off, 64);
        if (lane >= off) incl += o;
      }
      if (lane < words) pre[lane] = incl - v;
    }
    __syncthreads();
    for (int t = tid; t < bp; t += kThreads) {
      const uint32_t sl = trace_slot[t];
      srt[pre[sl >> 5] + (uint32_t)__popc(bits[sl >> 5] & ((1u << (sl & 31)) - 1u))] = cpos[sl];
    }
    __syncthreads();
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
// Bytes of dynamic LDS before the region: positions, 1 / |k| and s~ of max_cand candidates.
size_t lds_head(int max_cand) { return ((size_t)max_cand * 12 + 15) & ~(size_t)15; }

template <int DT, int D, int NT, int CPT, bool STAGED, bool GRAM>
hipError_t select_launch(const Shape& s, const SelectArgs& a, size_t body, hipStream_t st) {
  using T = typename Elem<DT>::T;
  // the region also holds the compaction's slot bitmap, its word prefixes and the positions
  const size_t region =
      std::max(std::max(body, STAGED ? (size_t)a.max_cand_all * 4 : (size_t)0),
               (size_t)(2 * kMaxSlotWords + a.max_cand) * 4);
  const size_t dyn = lds_head(a.max_cand) + region;
  auto kern = mmr_select_kernel<DT, D, NT, CPT, STAGED, GRAM>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)dyn);
  if (e != hipSuccess) return e;
  kern<<<dim3((unsigned)(s.n_prob * s.h_kv)), NT, dyn, st>>>(
      a.mu, a.sigma, a.score, a.cand_in, a.cand_in_max, a.cut_out, a.cut_max, a.list_stride,
      static_cast<const T*>(a.k), s.lens, s.tok_off,
      a.lambda1, a.lambda2,
      a.pool / 2, a.w_mu, s.h_kv,
      a.budget, a.budgets, a.cand_mult, a.keep_tail, a.cand_stride, a.max_cand, a.sel_idx, a.sel_score,
      a.cand_idx, a.cand_corr,
      CompactOut{static_cast<const uint4*>(a.k), static_cast<const uint4*>(a.v),
                 static_cast<uint4*>(a.k_out), static_cast<uint4*>(a.v_out), a.out_rows});
  return hipGetLastError();
}

// Score keys are staged in LDS when every problem's candidates fit next to the key rows or the
// Gram triangle (and the whole workgroup's LDS stays within the 160 KiB of a CU).
template <int DT, int D, int NT, int CPT, bool GRAM>
hipError_t select_dispatch(const Shape& s, const SelectArgs& a, hipStream_t st) {
  using T = typename Elem<DT>::T;
  const size_t body = GRAM ? gram::region_bytes<D>(a.max_cand) : (size_t)a.max_cand * D * sizeof(T);
  const size_t staged = lds_head(a.max_cand) + std::max(body, (size_t)a.max_cand_all * 4) +
                        sizeof(SelectShared<NT / 64>);
  if ((size_t)a.max_cand_all * 4 <= (size_t)kMaxStagedKeyBytes && staged <= kLdsBytes)
    return select_launch<DT, D, NT, CPT, true, GRAM>(s, a, body, st);
  return select_launch<DT, D, NT, CPT, false, GRAM>(s, a, body, st);
}

template <int DT, int D>
hipError_t select_cpt(const Shape& s, const SelectArgs& a, hipStream_t st) {
  constexpr int kMaxCand = kMaxCandBytes / (D * (int)sizeof(typename Elem<DT>::T));
  if constexpr (DT == kDtBf16) {
    // bf16 key rows fit the registers of 16 waves: one candidate per thread of 1024
    static_assert(kMaxCand <= 1024, "one candidate per thread");
    if (a.max_cand <= gram::kMaxCand) return select_dispatch<DT, D, 1024, 1, true>(s, a, st);
    return select_dispatch<DT, D, 1024, 1, false>(s, a, st);
  } else {
    // only the candidates-per-thread counts that the LDS key copy allows are instantiated
    constexpr int kNT = 256;
    const int cpt = (a.max_cand + kNT - 1) / kNT;
    if (cpt <= 1) return select_dispatch<DT, D, kNT, 1, false>(s, a, st);
    if constexpr (kMaxCand > kNT) {
      if (cpt <= 2) return select_dispatch<DT, D, kNT, 2, false>(s, a, st);
    }
    if constexpr (kMaxCand > 2 * kNT) return select_dispatch<DT, D, kNT, 4, false>(s, a, st);
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
