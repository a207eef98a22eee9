// Window statistics and the candidate set of the selection in one workgroup per unit, reading the
// keys once in full (section 3.1, Eq. (1), Eq. (3); section 3.2, Eq. (5) and the top-4B
// restriction).
//
// Pass 1 streams every key tile, as in stream_window.hip, and also bounds the base score of every
// key of each tile from above with the running softmax normalisers known at that point (Bound,
// stream_passes.h).  After the row normalisers b are complete, the tiles are sorted by their
// bounds and pass 2 evaluates the exact base scores tile by tile in that order, wave w taking
// positions w, w + 8, ... of the order.  The evaluated keys of the candidate range go into an LDS
// histogram and the waves' candidate lists (Prune, CandList); the histogram gives a lower bound of
// the unit's cut (the C-th best score), and a wave stops at its first tile whose bound lies below
// it: every key of the tiles left out scores below the cut.  Scores are formed by the same code as
// in the other window kernels, so each evaluated key's score is the one kv_window_base_scores
// writes, bit for bit; the candidate lists therefore hold exactly the unit's C best entries.
//
// On the 32-layer Mistral-shaped pass at L = 32768 (C = 256) pass 2 revisits about one tile in
// six; pass 1 is a plain stream of the keys.
#include "stream_passes.h"

namespace kv {
namespace stream {
namespace {

constexpr int kPruneMaxTiles = kCandMaxLen / kTileKeys;

template <int D, int NB, bool ALL, int NW, int S>
__global__ __launch_bounds__(NW * 64, 1) void window_prune_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS, NT = NW * 64;
  constexpr int kRedWords = NW * R * 2;
  static_assert(NW == kCandLists, "one candidate list per wave");
  static_assert((size_t)NW * S * Gm::TE * 2 >= (size_t)kPruneMaxTiles * 8, "the sort fits the ring");
  __shared__ __align__(16) uint16_t ring[NW][S * Gm::TE];
  // the waves' statistics in pass 1, the histogram of evaluated scores in pass 2
  __shared__ __align__(16) uint32_t red_hist[kRedWords > kPruneBins ? kRedWords : kPruneBins];
  __shared__ __align__(16) float bsh[R];
  __shared__ float tot_l[R];
  __shared__ float ub[kPruneMaxTiles];
  __shared__ uint16_t order[kPruneMaxTiles];
  __shared__ uint32_t c_okey[NW * kCandCap];
  __shared__ uint16_t c_pos[NW * kCandCap];
  __shared__ float c_max[NW];
  __shared__ uint32_t cut, top_bin;

  const int g = blockIdx.y, p = blockIdx.z;
  const int L = a.lens[p];
  const int G = a.h_q / a.h_kv;
  const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5, l32 = lane & 31;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const float c = a.c;
  const float inv_g = 1.f / (float)G;
  const float lam1 = a.lambda1[p];
  const size_t stat_base = (size_t)a.tok_off[p] * a.h_kv + (size_t)g * L;
  float2* red = reinterpret_cast<float2*>(red_hist);

  const uint16_t* kg = a.k + stat_base * D;
  KeyStream<D, NB, NW, S> ks{ring[wave], kg, 0, L, wave, lane};
  const int n_tiles = (L + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + NW - 1) / NW : 0;
  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  ks.prologue(my_tiles);
  hold_until_loaded<D, NB>(q);

  // ---- pass 1: statistics and tile bounds
  float m_run[NB], z_run[NB];
  const Bound bd{ub, red, tot_l, fmaxf(a.w_mu, 0.f), fmaxf(lam1, 0.f), inv_g,
                 ALL ? 1.f / (float)(NB * 32 - 1) : 1.f / 31.f};
  stats_bound_tiles<D, NB, ALL, NW, S>(ks, q, my_tiles, n_tiles / NW, L, c, l32, half, m_run,
                                       z_run, bd);
  stats_to_lds<NB>(m_run, z_run, red + wave * R, l32, half);
  __syncthreads();
  if (tid < R) {
    const float2 v = merge_waves<NW, R>(red, tid);
    bsh[tid] = v.x + __builtin_log2f(v.y);  // b = M + log2 Z, base 2
    const size_t ri = ((size_t)p * a.h_q + (size_t)g * G) * 32 + tid;
    a.row_max_out[ri] = v.x * kLn2;
    a.row_sum_out[ri] = v.y;
  }
  // ---- the tiles in decreasing order of their bounds, sorted in the ring (every load of pass 1
  //      has landed and been read: its last wait is vmcnt(0))
  int n2 = 1;
  while (n2 < n_tiles) n2 <<= 1;
  uint64_t* se = reinterpret_cast<uint64_t*>(&ring[0][0]);
  __syncthreads();  // the statistics are read from red; the ring is idle
  for (int i = tid; i < n2; i += NT)
    se[i] = i < n_tiles ? ((uint64_t)order_key(ub[i]) << 32) | (uint32_t)(0xFFFF - i) : 0ull;
  for (int i = tid; i < kPruneBins; i += NT) red_hist[i] = 0u;
  if (tid == 0) {
    cut = 0u;
    top_bin = 0u;
  }
  __syncthreads();
  bitonic_sort(se, n2, tid, NT);  // ascending
  for (int i = tid; i < n_tiles; i += NT) {
    const uint64_t e = se[n2 - 1 - i];
    order[i] = (uint16_t)(0xFFFF - (uint32_t)e);
    ub[i] = key_float((uint32_t)(e >> 32));
  }
  __syncthreads();  // the order is complete and the ring is free again

  // ---- pass 2: exact scores of the wanted tiles
  const int n_cand = L - a.keep_tail;
  const int bp = a.budgets ? a.budgets[p] : a.budget;
  const int C = min(a.cand_mult * bp, n_cand);
  KeyStream<D, NB, NW, S> ks2{ring[wave], kg, 0, L, wave, lane, order};
  ks2.prologue(my_tiles);
  Prune pr{CandList{c_okey + wave * kCandCap, c_pos + wave * kCandCap, C, 0, 0ull, false, -INFINITY},
           ub, red_hist, &cut, &top_bin, n_cand};
  const ScoreOut so{nullptr, lam1, a.w_mu};
  mu_sigma_tiles<D, NB, ALL, NW, S, kOutCand>(ks2, q, bsh, my_tiles, L, L, c, inv_g, nullptr,
                                              nullptr, l32, half, so, &pr);
  wait_vmem<0>();  // no load into the ring may outlive the workgroup (a stopped wave has some)
  CandList& cl = pr.cl;
  // the wave's best C (all of its entries when it holds no more), then zeros
  if (cl.n > C) cl.compact(lane);
  uint64_t* dst = a.cand_out + (((size_t)p * a.h_kv + g) * kCandLists + wave) * a.cand_stride;
  for (int i = lane; i < a.cand_stride; i += 64)
    dst[i] = i < cl.n ? cand_entry(cl.okey[i], cl.pos[i]) : 0ull;
  float m = cl.smax;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  if (lane == 0) c_max[wave] = m;
  __syncthreads();
  if (tid == 0) {
    float d = c_max[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) d = fmaxf(d, c_max[w]);
    a.cand_max[(size_t)p * a.h_kv + g] = fmaxf(d, 1e-12f);
  }
}

template <int D, int NB> struct PruneLaunch {
  static hipError_t run(const Shape& s, const StreamArgs& args, hipStream_t st) {
    const dim3 grid(1, s.h_kv, s.n_prob);
    if (args.sigma_all) window_prune_kernel<D, NB, true, kWaves, 2><<<grid, kThreads, 0, st>>>(args);
    else window_prune_kernel<D, NB, false, kWaves, 2><<<grid, kThreads, 0, st>>>(args);
    return hipGetLastError();
  }
};

}  // namespace
}  // namespace stream

hipError_t launch_stream_window_cands(const Shape& s, const StreamPlan& plan, const void* q_win,
                                      const void* k, float scale, const float* lambda1, float w_mu,
                                      int budget, const int32_t* budgets, int cand_mult,
                                      int keep_tail, float* row_max, float* row_sum,
                                      uint64_t* cand_out, float* cand_max, int cand_stride,
                                      bool sigma_all, hipStream_t stream) {
  if (plan.max_segs != 1 || !cand_out || !cand_max || s.max_len > kCandMaxLen)
    return hipErrorInvalidValue;
  stream::StreamArgs a = stream::base_args(s, plan, q_win, k, scale);
  a.row_max_out = row_max;
  a.row_sum_out = row_sum;
  a.sigma_all = sigma_all ? 1 : 0;
  a.lambda1 = lambda1;
  a.w_mu = w_mu;
  a.cand_out = cand_out;
  a.cand_max = cand_max;
  a.cand_stride = cand_stride;
  a.budget = budget;
  a.budgets = budgets;
  a.cand_mult = cand_mult;
  a.keep_tail = keep_tail;
  return stream::launch_for_shape<stream::PruneLaunch>(s, a, stream);
}

}  // namespace kv
