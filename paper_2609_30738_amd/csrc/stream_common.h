// Building blocks of the streaming window kernels (pass 1 in stream_stats.hip, pass 2 in
// stream_mu_sigma.hip, both passes of a unit in one workgroup in stream_window.hip; the passes'
// per-segment loops in stream_passes.h): the argument block, the tile geometry, the per-wave key
// stream into LDS and small wave-level helpers.
//
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
#pragma once

#include <algorithm>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace kv {
namespace stream {

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
  float2* part;           // [n_units][max_segs][R] segment partials (m, z), base 2; pass 1 with
                          // part == nullptr (one segment per unit) writes row_max_out / row_sum_out
  const float* row_max;   // pass 2 from given statistics (part == nullptr)
  const float* row_sum;
  float* row_max_out;     // pass 2 from partials: written by segment 0
  float* row_sum_out;
  float* mu;
  float* sigma;
  int sigma_all;          // pass 2: dispersion over all G x 32 (head, row) values
  // base-score mode of pass 2: s = fma(lambda1[p], sigma, w_mu mu) per key into `score` instead
  // of mu / sigma
  float* score;
  const float* lambda1;
  float w_mu;
  // candidate mode of pass 2 (every unit one segment): per unit the candidate list,
  // [n_units][cand_stride] entries (the C_p candidates in position order, then 0), and the maximum
  // base score over the candidate positions clamped at 1e-12 (the selection's normaliser);
  // C_p = min(cand_mult B_p, L_p - keep_tail), B_p = budgets[p] or budget
  uint64_t* cand_out;
  float* cand_max;
  int cand_stride;
  int budget, cand_mult, keep_tail;
  const int32_t* budgets;
  // candidate mode, pass 1: per unit code_stride words of tile codes (32 words per tile)
  uint32_t* codes;
  int code_stride;
  // candidate mode with the selection in the same launch (sel_idx != nullptr, every C_p <= 256):
  // the greedy's outputs as from the selection kernel, [n_prob][h_kv][budget], and with k_out the
  // compacted rows of K and V, [n_prob][h_kv][out_rows][D]
  const float* lambda2;
  int32_t* sel_idx;
  float* sel_score;
  const uint16_t* v;
  uint16_t* k_out;
  uint16_t* v_out;
  int out_rows;
};

constexpr int kCandLists = kWaves;  // candidate lists per unit: one per wave of the fused kernel

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

__device__ __forceinline__ float max_halves(float x) {  // max(x, x of lane ^ 32)
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// inclusive prefix sum over the 64 lanes in lane order: steps of 1, 2, 4 and 8 lanes within each
// row of 16 (DPP row shifts, lanes shifted in from outside the row read 0), then the last lane of
// each row added to the rows after it (DPP row broadcasts)
__device__ __forceinline__ uint32_t wave_inclusive_sum(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xF, 0xF, true);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xF, 0xF, true);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xF, 0xF, true);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xF, 0xF, true);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0u, x, 0x142, 0xA, 0xF, false);  // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0u, x, 0x143, 0xC, 0xF, false);  // row_bcast:31 into rows 2, 3
  return x;
}

// s_waitcnt vmcnt(later NDMA + (stores ? TS : 0)) for a run-time later in [0, 3]
template <int NDMA, int TS>
__device__ __forceinline__ void wait_vmem_tiles(int later, bool stores) {
  if (stores) {
    switch (later) {
      case 0: wait_vmem<TS>(); break;
      case 1: wait_vmem<NDMA + TS>(); break;
      case 2: wait_vmem<2 * NDMA + TS>(); break;
      default: wait_vmem<3 * NDMA + TS>(); break;
    }
  } else {
    switch (later) {
      case 0: wait_vmem<0>(); break;
      case 1: wait_vmem<NDMA>(); break;
      case 2: wait_vmem<2 * NDMA>(); break;
      default: wait_vmem<3 * NDMA>(); break;
    }
  }
}

// Per-wave key stream of one segment: a ring of S tiles in LDS filled by direct-to-LDS loads.
// Tile j of the wave (keys k0 + (j NW + wave) 32 ..) goes to slot j mod S.
template <int D, int NB, int NW, int S> struct KeyStream {
  using Gm = SGeo<D, NB>;
  static_assert(S == 2 || S == 4, "ring of 2 or 4 tiles");
  uint16_t* ring;       // this wave's S tiles
  const uint16_t* kg;   // keys of the unit
  int k0, k1, wave, lane;
  // nullptr: tile j of the wave is the segment's tile j NW + wave; otherwise order[j NW + wave]
  // (LDS) names it
  const uint16_t* order = nullptr;
  // loads that stay in the caches (a second visit of a few tiles whose keys are read again soon);
  // otherwise non-temporal (aux 2: each key read once per pass)
  bool keep = false;

  // the segment's tile index of the wave's tile j
  __device__ int tile_index(int j) const {
    return order ? (int)order[j * NW + wave] : j * NW + wave;
  }
  __device__ int tile_key(int j) const { return k0 + tile_index(j) * kTileKeys; }

  // Byte offset, within a tile, of the 16-byte chunk that load instruction i of this lane fetches
  // (the chunk that lands at the lane's LDS slot 64 i + lane).  Four consecutive rows per
  // instruction at d = 128, so the swizzle repeats every four instructions and the offset of
  // instruction i is that of i mod 4 plus 4 KiB per four; at d = 64 it is that of 0 plus 1 KiB
  // per instruction.
  __device__ static int chunk_off(int i, int lane) {
    const int pos = 64 * i + lane;  // LDS chunk slot written by this lane
    const int row = pos / Gm::CH;
    const int ch = (pos % Gm::CH) ^ (row % Gm::CH);
    return (row * D + ch * 8) * (int)sizeof(uint16_t);
  }
  static constexpr int kOffRegs = Gm::NDMA < 4 ? Gm::NDMA : 4;

  // tile j into its slot; rows past the segment end re-read its last key
  __device__ __forceinline__ void issue(int j) const {
    const int t0 = tile_key(j);
    uint16_t* dst = ring + (j & (S - 1)) * Gm::TE;
    if (t0 + kTileKeys <= k1) {
      // a whole tile: a wave-uniform base and per-lane offsets that do not change from tile to
      // tile
      const char* base = reinterpret_cast<const char*>(kg + (size_t)t0 * D);
      int off[kOffRegs];
#pragma unroll
      for (int i = 0; i < kOffRegs; ++i) off[i] = chunk_off(i, lane);
#pragma unroll
      for (int i = 0; i < Gm::NDMA; ++i) {
        const gptr_t src = (gptr_t)(base + (i / 4) * 4096 + off[i % 4]);
        if (keep) __builtin_amdgcn_global_load_lds(src, (lptr_t)(dst + i * 512), 16, 0, 0);
        else __builtin_amdgcn_global_load_lds(src, (lptr_t)(dst + i * 512), 16, 0, 2);
      }
    } else {
#pragma unroll
      for (int i = 0; i < Gm::NDMA; ++i) {
        const int pos = 64 * i + lane;
        const int row = pos / Gm::CH;
        const int ch = (pos % Gm::CH) ^ (row % Gm::CH);
        const gptr_t src = (gptr_t)(kg + (size_t)min(t0 + row, k1 - 1) * D + ch * 8);
        if (keep) __builtin_amdgcn_global_load_lds(src, (lptr_t)(dst + i * 512), 16, 0, 0);
        else __builtin_amdgcn_global_load_lds(src, (lptr_t)(dst + i * 512), 16, 0, 2);
      }
    }
  }

  // the first min(S, my_tiles) tiles
  __device__ __forceinline__ void prologue(int my_tiles) const {
#pragma unroll
    for (int j = 0; j < S; ++j)
      if (j < my_tiles) issue(j);
  }

  // MFMA operand fragments of tile j (lane: row l32, K half `half`), once its loads have landed
  __device__ __forceinline__ void read(bf16x8_t (&a)[Gm::NS], int j, int l32, int half) const {
    const uint16_t* src = ring + (j & (S - 1)) * Gm::TE;
#pragma unroll
    for (int s = 0; s < Gm::NS; ++s)
      a[s] = *reinterpret_cast<const bf16x8_t*>(src + Gm::slot_of(l32, 2 * s + half) * 8);
  }

  // Wait for tile j, copy it into registers and hand its slot to tile j + S.  After tile j's loads
  // the wave has issued the loads of the (up to S - 1) tiles after it and, from tile S on, the
  // STORES vector memory stores per tile of the S tiles before it (the caller's, issued after each
  // tile's computation); those may stay in flight.
  template <int STORES>
  __device__ __forceinline__ void next(bf16x8_t (&a)[Gm::NS], int j, int my_tiles, int l32,
                                       int half) const {
    wait_vmem_tiles<Gm::NDMA, STORES * S>(min(S - 1, my_tiles - 1 - j), STORES > 0 && j >= S);
    read(a, j, l32, half);
    wait_lds();
    if (j + S < my_tiles) issue(j + S);
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


inline StreamArgs base_args(const Shape& s, const StreamPlan& plan, const void* q_win, const void* k,
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

// Launch of either pass for the unit shape of `s` (d in {64, 128}, G in {1, 2, 4}).
template <template <int, int> class Launch>
hipError_t launch_for_shape(const Shape& s, const StreamArgs& args, hipStream_t st) {
  const int G = s.group();
  if (s.d == 128) {
    if (G == 4) return Launch<128, 4>::run(s, args, st);
    if (G == 2) return Launch<128, 2>::run(s, args, st);
    return Launch<128, 1>::run(s, args, st);
  }
  if (G == 4) return Launch<64, 4>::run(s, args, st);
  if (G == 2) return Launch<64, 2>::run(s, args, st);
  return Launch<64, 1>::run(s, args, st);
}

}  // namespace stream
}  // namespace kv
