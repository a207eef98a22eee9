// Window statistics and the candidate set of the selection in one workgroup per unit, reading the
// keys once in full (section 3.1, Eq. (1), Eq. (3); section 3.2, Eq. (5) and the top-4B
// restriction).
//
// Pass 1 streams every key tile, as in stream_window.hip, and also records, per tile and per
// (head, window row), the tile's largest logit as a one-byte code below the tile's largest logit
// (TileCodes; 128 bytes per tile in the workspace).  Once the row normalisers b are complete, these
// codes bound the base score of every key of each tile from above (tile_bound).  The tiles are
// then ordered by their bounds (a counting sort into bins of 1/16 of an octave below the largest
// bound, each tile standing for its bin's upper edge) and pass 2 evaluates the exact base scores
// tile by tile in that order, wave w taking positions w, w + 8, ... of the order.  The evaluated
// keys of the candidate range go into an LDS histogram (Prune), which gives a lower bound of the
// unit's cut (the C-th best score), and a wave stops at its first tile whose bound lies below it:
// every key of the tiles left out scores below the cut.  The evaluated scores are stored over the
// tiles' codes; after the pass the C-th largest (score, position) entry among them is found digit
// by digit, and the C candidates are written in position order.  Scores are formed by the same
// code as in the other window kernels, so each evaluated key's score is the one
// kv_window_base_scores writes, bit for bit, and the candidates are exactly the unit's C best.
//
// On the 32-layer Mistral-shaped pass at L = 32768 (C = 256) the bounds leave about one tile in
// twenty to pass 2.
#include "select_gram.h"
#include "stream_passes.h"

namespace kv {
namespace stream {
namespace {

constexpr int kPruneMaxTiles = kCandMaxLen / kTileKeys;
// Order of the tiles for pass 2: bin 0 holds the tiles with a masked key (bound +inf), bin k >= 1
// the tiles whose bound lies within ((k - 1) / 16, k / 16] octaves below the largest finite bound
// (the last bin: everything further below).
constexpr int kOrderBins = 1024;
constexpr float kBinsPerOctave = 16.f;
// Bounds are widened by kBoundSlack for the rounding of both passes (logits formed in another
// MFMA operand order, approximate exp2 / log2) and kept above kBoundFloor.
constexpr float kBoundSlack = 1.00390625f;  // 1 + 2^-8
constexpr float kBoundFloor = 0x1p-100f;
constexpr float kCodeStep = 0.125f;          // code units: 1/8 of a factor of two

// Pass-1 hook of candidate mode: per tile, the largest t = logit * c of every (head, window row) as
// the number of 1/8-steps it lies below the tile's largest t (rounded down, one less where the
// exact number is an odd integer; at most 255), one byte per head of the row's word in the unit's
// code rows, and the tile's largest t into ref[tile] (LDS); a tile with a masked key gets
// ref = +inf and a tile with a NaN logit ref = NaN (both always revisited).  The row maxima of two
// heads are merged across the wave's halves in one exchange, leaving head k in lanes 0-31 and head
// k + NB / 2 in lanes 32-63, so each lane stores the bytes of its row's word that belong to its
// heads (one store per tile).
template <int NBH> struct TileCodes {
  static constexpr int kStores = 1;
  static_assert(NBH == 1 || NBH == 2 || NBH == 4, "one, two or four query heads per key head");
  uint32_t* codes;  // tile i at codes + 32 i: word r = window row r, byte b < NB = head b
  float* ref;       // [n_tiles] LDS
  float c;          // softmax scale * log2(e)
  int l32, lane;

  template <int NB>
  __device__ __forceinline__ void interior(int tile, const float (&tmax)[NB]) const {
    static_assert(NB == NBH, "head count");
    constexpr int NP = NB == 4 ? 2 : 1;  // heads per lane after the exchange
    float tm[NP];  // row maxima of t over the tile's 32 keys
    if constexpr (NB == 1) {
      tm[0] = max_halves(tmax[0]) * c;
    } else {
#pragma unroll
      for (int k = 0; k < NP; ++k) {
        const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(tmax[k]),
                                                        __float_as_uint(tmax[k + NB / 2]), false, false);
        tm[k] = __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1])) * c;
      }
    }
    const float m = NP == 2 ? __builtin_elementwise_maximum(tm[0], tm[NP - 1]) : tm[0];
    float r = wave_max_uniform(m);  // the tile's largest t
    if (__ballot(m != m)) r = __builtin_nanf("");
    // code: the steps (r - t) * 8 less half a step, rounded to nearest (even) and saturated to
    // [0, 255] by v_cvt_pk_u8_f32: never above the exact number of steps (NaN gives 0)
    uint32_t w = 0u;
#pragma unroll
    for (int k = 0; k < NP; ++k)
      w = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(r - tm[k], 1.f / kCodeStep, -0.5f), (uint32_t)k, w);
    char* dst = reinterpret_cast<char*>(codes + 32 * tile + l32);
    if constexpr (NB == 4) store_u16(dst + 2 * (lane >> 5), w);
    else if constexpr (NB == 2) store_u8(dst + (lane >> 5), w);
    else store_u8(dst, w);
    if (lane == 0) ref[tile] = r;
  }
  __device__ __forceinline__ void guarded(int tile) const {
    store_word(codes + 32 * tile + l32, 0xFFFFFFFFu);
    if (lane == 0) ref[tile] = INFINITY;
  }
  __device__ __forceinline__ static void store_word(uint32_t* dst, uint32_t v) {
    asm volatile("global_store_dword %0, %1, off sc1" ::"v"(dst), "v"(v) : "memory");
  }
  __device__ __forceinline__ static void store_u16(char* dst, uint32_t v) {
    asm volatile("global_store_short %0, %1, off sc1" ::"v"(dst), "v"(v) : "memory");
  }
  __device__ __forceinline__ static void store_u8(char* dst, uint32_t v) {
    asm volatile("global_store_byte %0, %1, off sc1" ::"v"(dst), "v"(v) : "memory");
  }
};

// Upper bound of the base score s = w_mu mu + lambda1 sigma (section 3.2, Eq. (5)) of every key of
// a tile from its codes (row r of head h: t <= ref - code / 8) and the final row normalisers b:
// a[h][r] = 2^(t - b[h][r]) <= a'[h][r], hence mu <= (1 / 32) sum_r abar'[r] (abar': mean over the
// G heads) and, since a variance is at most the mean square, sigma <= sqrt(sum_r abar'[r]^2 / 31)
// (sum_{h,r} a'^2 / (32 G - 1) for the dispersion over all rows).  The positive parts of w_mu and
// lambda1 enter.
template <int NB, bool ALL>
__device__ __forceinline__ float tile_bound(const uint32_t* codes_t, float ref, const float* bsh,
                                            float wmu_p, float lam1_p, float inv_g) {
  const uint4* src = reinterpret_cast<const uint4*>(codes_t);
  float p1 = 0.f, p2 = 0.f;
#pragma unroll 2
  for (int v = 0; v < 8; ++v) {
    const uint4 w4 = src[v];
    const uint32_t ws[4] = {w4.x, w4.y, w4.z, w4.w};
    float arow[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const float4 bv = *reinterpret_cast<const float4*>(bsh + b * 32 + 4 * v);
      const float bb[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float code = (float)((ws[e] >> (8 * b)) & 0xFFu);
        const float a = __builtin_amdgcn_exp2f(fmaf(code, -kCodeStep, ref) - bb[e]);
        arow[e] += a;
        if constexpr (ALL) p2 = fmaf(a, a, p2);
      }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      p1 += arow[e];
      if constexpr (!ALL) {
        const float ab = arow[e] * inv_g;
        p2 = fmaf(ab, ab, p2);
      }
    }
  }
  constexpr float inv_n1 = ALL ? 1.f / (float)(NB * 32 - 1) : 1.f / 31.f;
  const float mu_b = p1 * inv_g * (1.f / 32.f);
  return fmaf(fmaf(lam1_p, __builtin_sqrtf(p2 * inv_n1), wmu_p * mu_b), kBoundSlack, kBoundFloor);
}

// Bitmap words over the candidate positions of a unit (one bit per position).
constexpr int kBitmapWords = kCandMaxLen / 32;
// Entries that share every digit found so far and are ranked directly (by counting).
constexpr int kRankDirect = 512;

// The bin (order key >> kPruneShift) of the C-th largest entry counted in hist, scanning down from
// top (a bin at or above every nonempty one), into *cut_bin, and the number of entries in the bins
// above it into *above.  One wave; hist holds at least C entries.
__device__ __forceinline__ void find_cut_bin(const uint32_t* hist, uint32_t top, int C, int lane,
                                             uint32_t* cut_bin, uint32_t* above) {
  uint32_t cum = 0;
  for (int b0 = (int)top; b0 >= 0; b0 -= 64) {
    const int b = b0 - lane;
    const uint32_t own = b >= 0 ? hist[b] : 0u;
    const uint32_t pre = wave_inclusive_sum(own);
    const uint64_t hit = __ballot(cum + pre >= (uint32_t)C);
    if (hit) {
      const int hl = __ffsll((unsigned long long)hit) - 1;
      if (lane == hl) {
        *cut_bin = (uint32_t)b;
        *above = cum + pre - own;
      }
      return;
    }
    cum += (uint32_t)__builtin_amdgcn_readlane((int)pre, 63);
  }
}

template <int D, int NB, bool ALL, int NW, int S, bool SEL>
__global__ __launch_bounds__(NW * 64, 1) void window_prune_kernel(StreamArgs a) {
  using Gm = SGeo<D, NB>;
  constexpr int R = Gm::R, NS = Gm::NS, NT = NW * 64;
  constexpr int kRedWords = NW * R * 2;
  constexpr int kTilesPerThread = kPruneMaxTiles / NT;
  static_assert(kPruneMaxTiles % NT == 0, "whole tiles per thread");
  static_assert(NT % kTileKeys == 0, "whole tiles per visit");
  static_assert(kTileKeys == 32, "a half-wave visits the keys of one tile");
  static_assert(2 * kOrderBins >= kBitmapWords + 2 * kRankDirect,
                "the bitmap and the ranked group fit the order's bins");
  static_assert(kPruneBins >= kBitmapWords, "the word prefixes fit the histogram");
  // the waves' key rings; after the second pass, the order keys of the evaluated scores
  constexpr int kRingElems = NW * S * Gm::TE > 2 * kCandMaxLen ? NW * S * Gm::TE : 2 * kCandMaxLen;
  __shared__ __align__(16) uint16_t ring[kRingElems];
  static_assert(!SEL || gram::region_bytes<D>(gram::kMaxCand) <= sizeof(ring),
                "the staged key rows and the cosine triangle fit the ring");
  static_assert(!SEL || 4 * gram::kMaxCand <= kPruneMaxTiles, "the slot arrays fit the bounds");
  // the waves' statistics after pass 1, the histogram of evaluated scores in pass 2
  __shared__ __align__(16) uint32_t red_hist[kRedWords > kPruneBins ? kRedWords : kPruneBins];
  __shared__ __align__(16) float bsh[R];
  // pass 1: the tile's largest t; from the order on: the bound of the i-th tile of the order
  __shared__ float ub[kPruneMaxTiles];
  __shared__ uint16_t order[kPruneMaxTiles];
  // the bin counts and offsets of the order
  __shared__ uint32_t bins[2 * kOrderBins];
  __shared__ float c_max[NW];
  __shared__ uint32_t ev[NW];
  __shared__ uint32_t cut, bmax_bits, n_eval;
  __shared__ uint64_t cut_entry;

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
  uint32_t* codes_u = a.codes + ((size_t)p * a.h_kv + g) * a.code_stride;

  const uint16_t* kg = a.k + stat_base * D;
  KeyStream<D, NB, NW, S> ks{ring + wave * S * Gm::TE, kg, 0, L, wave, lane};
  const int n_tiles = (L + kTileKeys - 1) / kTileKeys;
  const int my_tiles = n_tiles > wave ? (n_tiles - wave + NW - 1) / NW : 0;
  bf16x8_t q[NB][NS];
  load_queries<D, NB>(q, a.q_win + ((size_t)p * a.h_q + (size_t)g * G) * 32 * D, l32, half);
  ks.prologue(my_tiles);
  hold_until_loaded<D, NB>(q);

  // ---- pass 1: statistics and tile codes
  float m_run[NB], z_run[NB];
  stats_tiles<D, NB, NW, S>(ks, q, my_tiles, L, L, c, l32, half, m_run, z_run,
                            TileCodes<NB>{codes_u, ub, c, l32, lane});
  wait_vmem<0>();  // this wave's code stores have landed (other waves read them below)
  stats_to_lds<NB>(m_run, z_run, red + wave * R, l32, half);
  if (tid == 0) {
    cut = 0u;
    bmax_bits = 0u;
  }
  __syncthreads();
  if (tid < R) {
    const float2 v = merge_waves<NW, R>(red, tid);
    bsh[tid] = v.x + __builtin_log2f(v.y);  // b = M + log2 Z, base 2
    const size_t ri = ((size_t)p * a.h_q + (size_t)g * G) * 32 + tid;
    a.row_max_out[ri] = v.x * kLn2;
    a.row_sum_out[ri] = v.y;
  }
  __syncthreads();  // the normalisers are complete; red is free

  // ---- bounds of the thread's tiles tid + u NT (-inf: no candidate key, never revisited)
  uint32_t* cnt = bins;                  // [kOrderBins] tiles per bin
  uint32_t* off = bins + kOrderBins;     // [kOrderBins] first position of each bin, then a cursor
  for (int i = tid; i < kPruneBins; i += NT) red_hist[i] = 0u;
  for (int i = tid; i < kOrderBins; i += NT) cnt[i] = 0u;
  const int n_cand = L - a.keep_tail;
  const float wmu_p = fmaxf(a.w_mu, 0.f), lam1_p = fmaxf(lam1, 0.f);
  float bnd[kTilesPerThread];
  float lmax = 0.f;  // largest finite bound (bounds are positive)
#pragma unroll
  for (int u = 0; u < kTilesPerThread; ++u) {
    const int i = tid + u * NT;
    bnd[u] = -INFINITY;
    if (i < n_tiles && i * kTileKeys < n_cand) {
      const float r = ub[i];
      float bd = INFINITY;
      if (r < INFINITY) bd = tile_bound<NB, ALL>(codes_u + 32 * i, r, bsh, wmu_p, lam1_p, inv_g);
      if (!(bd == bd)) bd = INFINITY;  // NaN inputs: revisit
      bnd[u] = bd;
      if (bd < INFINITY) lmax = fmaxf(lmax, bd);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) lmax = fmaxf(lmax, __shfl_xor(lmax, o, 64));
  if (lane == 0) atomicMax(&bmax_bits, __float_as_uint(lmax));  // positive floats order as integers
  __syncthreads();
  const float bmax = __uint_as_float(bmax_bits);
  const float lg_max = __builtin_amdgcn_logf(bmax);  // log2; only used when a finite bound exists
  int bin[kTilesPerThread];
#pragma unroll
  for (int u = 0; u < kTilesPerThread; ++u) {
    bin[u] = -1;
    if (bnd[u] == INFINITY) {
      bin[u] = 0;
    } else if (bnd[u] > 0.f) {
      // bins counted down from the largest bound, rounded towards the larger bound (the bin's
      // upper edge stays above every bound in it despite the rounding of log2)
      const float x = (lg_max - __builtin_amdgcn_logf(bnd[u])) * kBinsPerOctave - (1.f / 64.f);
      bin[u] = 1 + (int)fminf(fmaxf(x, 0.f), (float)(kOrderBins - 2));
    }
    if (bin[u] >= 0) atomicAdd(&cnt[bin[u]], 1u);
  }
  __syncthreads();
  if (wave == 0) {
    // exclusive scan of the counts: lane l holds bins 16 l .. 16 l + 15
    constexpr int PB = kOrderBins / 64;
    uint32_t v[PB];
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < PB; ++k) {
      v[k] = cnt[lane * PB + k];
      s += v[k];
    }
    uint32_t incl = s;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t t = (uint32_t)__shfl_up((int)incl, o, 64);
      if (lane >= o) incl += t;
    }
    uint32_t run = incl - s;
#pragma unroll
    for (int k = 0; k < PB; ++k) {
      off[lane * PB + k] = run;
      run += v[k];
    }
    if (lane == 63) n_eval = incl;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kTilesPerThread; ++u) {
    if (bin[u] >= 0) {
      const uint32_t pos = atomicAdd(&off[bin[u]], 1u);
      order[pos] = (uint16_t)(tid + u * NT);
      ub[pos] = bin[u] == 0 ? INFINITY
                            : bmax * __builtin_amdgcn_exp2f(-(float)(bin[u] - 1) * (1.f / kBinsPerOctave));
    }
  }
  __syncthreads();  // the order is complete; the ring is free

  // ---- pass 2: exact scores of the wanted tiles, stored over their codes
  const int n_ord = (int)n_eval;
  const int bp = a.budgets ? a.budgets[p] : a.budget;
  const int C = min(a.cand_mult * bp, n_cand);
  const int my_tiles2 = n_ord > wave ? (n_ord - wave + NW - 1) / NW : 0;
  // the second visit keeps its tiles in the caches: the selection reads the candidates' rows next
  KeyStream<D, NB, NW, S> ks2{ring + wave * S * Gm::TE, kg, 0, L, wave, lane, order, true};
  ks2.prologue(my_tiles2);
  float* score_u = reinterpret_cast<float*>(codes_u);  // a tile's codes are dead once bounded
  // the cut's scan starts at the bin of the largest finite bound: scores above it (in tiles with a
  // masked key) are left out of the scan, which only lowers the cut
  const int scan_top = bmax > 0.f ? (int)(order_key(bmax) >> kPruneShift) : kPruneBins - 1;
  Prune pr{ub, red_hist, &cut, score_u, scan_top, n_cand, C, -INFINITY, 0};
  const ScoreOut so{nullptr, lam1, a.w_mu};
  mu_sigma_tiles<D, NB, ALL, NW, S, kOutCand>(ks2, q, bsh, my_tiles2, L, L, c, inv_g, nullptr,
                                              nullptr, l32, half, so, &pr);
  wait_vmem<0>();  // the score stores have landed; no load into the ring outlives the workgroup
  float m = pr.smax;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if (lane == 0) {
    c_max[wave] = m;
    ev[wave] = (uint32_t)pr.evaluated;
  }

  // ---- the unit's candidates: the C largest entries (order key of the score, position) among
  //      the evaluated keys, written in ascending position order.  The C-th largest entry is
  //      found digit by digit (11 bits at a time, most significant first): the histogram of the
  //      pass gives the first digit; each further digit counts the evaluated entries that share
  //      the digits found so far, until few enough remain to rank them directly.
  __syncthreads();  // the scores, the histogram and every wave's tile count are final
  int max_ev = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) max_ev = max(max_ev, (int)ev[w]);
  const int n_pos = min(n_ord, max_ev * NW);  // order positions at or after this one: not evaluated
  // the order keys of the evaluated scores, copied once into the ring (free after the pass) at
  // [order position][key in tile] by waves 1.. while wave 0 finds the first digit of the cut; the
  // passes below visit them there
  uint32_t* okc = reinterpret_cast<uint32_t*>(ring);
  if (wave == 0) {
    find_cut_bin(red_hist, kPruneBins - 1, C, lane, &cut, &bmax_bits);
  } else {
    constexpr int kVisit = (NT - 64) / kTileKeys;  // tiles per visit
    for (int p0 = 0; p0 < n_pos; p0 += kVisit) {
      const int pos = p0 + (tid - 64) / kTileKeys;
      if (pos < n_pos && (pos / NW) < (int)ev[pos % NW]) {
        const int key = (int)order[pos] * kTileKeys + (tid % kTileKeys);
        // device-coherent load: the line may still sit in this CU's vector cache with the tile's
        // codes, read before the score was stored over them
        if (key < n_cand)
          okc[pos * kTileKeys + tid % kTileKeys] = order_key(__uint_as_float(__hip_atomic_load(
              reinterpret_cast<uint32_t*>(score_u + key), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)));
      }
    }
  }
  __syncthreads();
  // visit every evaluated key of the candidate range once: fn(entry, key)
  auto for_each_entry = [&](auto fn) __attribute__((always_inline)) {
    for (int p0 = 0; p0 < n_pos; p0 += NT / kTileKeys) {
      const int pos = p0 + tid / kTileKeys;
      if (pos < n_pos && (pos / NW) < (int)ev[pos % NW]) {
        const int key = (int)order[pos] * kTileKeys + (tid % kTileKeys);
        if (key < n_cand) fn(cand_entry(okc[pos * kTileKeys + tid % kTileKeys], (uint32_t)key), key);
      }
    }
  };
  uint64_t prefix = (uint64_t)cut << (64 - (32 - kPruneShift));  // the digits found so far
  int pbits = 32 - kPruneShift;                                   // their count
  int need = C - (int)bmax_bits;  // how many entries of the group the candidates still take
  uint32_t group = red_hist[cut];
  while (group > (uint32_t)kRankDirect && pbits < 64) {
    const int dbits = min(32 - kPruneShift, 64 - pbits);
    const int shift = 64 - pbits - dbits;
    __syncthreads();  // the last digit's readers are done with the histogram
    for (int i = tid; i < kPruneBins; i += NT) red_hist[i] = 0u;
    __syncthreads();
    for_each_entry([&](uint64_t e, int) {
      if ((e >> (64 - pbits)) == (prefix >> (64 - pbits)))
        atomicAdd(&red_hist[(uint32_t)(e >> shift) & ((1u << dbits) - 1u)], 1u);
    });
    __syncthreads();
    if (wave == 0) find_cut_bin(red_hist, (1 << dbits) - 1, need, lane, &cut, &bmax_bits);
    __syncthreads();
    prefix |= (uint64_t)cut << shift;
    pbits += dbits;
    need -= (int)bmax_bits;
    group = red_hist[cut];
  }
  // the group: at most kRankDirect entries (or one, once every digit is found); its need-th
  // largest entry is the C-th largest overall, found by counting the larger ones.  A half-wave
  // visits the 32 keys of one evaluated tile: the group is appended by ballot, the candidates'
  // bits of a tile are a ballot too.
  uint64_t* gb = reinterpret_cast<uint64_t*>(bins + kBitmapWords);
  uint32_t* bm = bins;          // the candidates in a bitmap over the positions (word = tile)
  uint32_t* gcnt = red_hist;    // [kRankDirect] entries of the group larger than each member
  const int n_words = (n_cand + 31) >> 5;
  if (tid == 0) {
    n_eval = 0u;
    cut_entry = ~0ull;
  }
  __syncthreads();  // every thread has read the group's size from the histogram
  for (int i = tid; i < kRankDirect; i += NT) gcnt[i] = 0u;
  for (int i = tid; i < n_words; i += NT) bm[i] = 0u;
  // entry of this thread's key in visit p0 (0: none)
  auto entry_at = [&](int p0, int* tile) __attribute__((always_inline)) -> uint64_t {
    const int pos = p0 + tid / kTileKeys;
    *tile = -1;
    if (pos < n_pos && (pos / NW) < (int)ev[pos % NW]) {
      *tile = (int)order[pos];
      const int key = *tile * kTileKeys + (tid % kTileKeys);
      if (key < n_cand) return cand_entry(okc[pos * kTileKeys + tid % kTileKeys], (uint32_t)key);
    }
    return 0ull;
  };
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int p0 = 0; p0 < n_pos; p0 += NT / kTileKeys) {
    int tile;
    const uint64_t e = entry_at(p0, &tile);
    const bool in = e != 0ull && (e >> (64 - pbits)) == (prefix >> (64 - pbits));
    const uint64_t m = __ballot(in);
    if (m) {
      const int leader = __ffsll((unsigned long long)m) - 1;
      uint32_t base = 0;
      if (lane == leader) base = atomicAdd(&n_eval, (uint32_t)__popcll(m));
      base = __builtin_amdgcn_readlane(base, leader);
      const uint32_t at_ = base + (uint32_t)__popcll(m & below);
      if (in && at_ < (uint32_t)kRankDirect) gb[at_] = e;
    }
  }
  __syncthreads();
  const int n_grp = min((int)n_eval, kRankDirect);
  {
    // member i against a share of the group: thread t takes member t % n_grp and share t / n_grp
    const int parts = n_grp > 0 ? max(1, NT / n_grp) : 1;
    if (tid < parts * n_grp) {
      const int i = tid % n_grp, part = tid / n_grp;
      const int j0 = part * n_grp / parts, j1 = (part + 1) * n_grp / parts;
      const uint64_t e = gb[i];
      uint32_t larger = 0;
      for (int j = j0; j < j1; ++j) larger += gb[j] > e ? 1u : 0u;
      if (larger) atomicAdd(&gcnt[i], larger);
    }
  }
  __syncthreads();
  for (int i = tid; i < n_grp; i += NT)
    if (gcnt[i] == (uint32_t)(need - 1)) cut_entry = gb[i];
  __syncthreads();
  const uint64_t t_entry = cut_entry;
  for (int p0 = 0; p0 < n_pos; p0 += NT / kTileKeys) {
    int tile;
    const uint64_t e = entry_at(p0, &tile);
    const uint64_t m = __ballot(e != 0ull && e >= t_entry);
    if ((tid & (kTileKeys - 1)) == 0 && tile >= 0) bm[tile] = (uint32_t)(m >> (lane & 32));
  }
  __syncthreads();
  uint32_t* wpre = red_hist;  // candidates in the bitmap words before each word
  if (wave == 0) {
    constexpr int PW = kBitmapWords / 64;
    uint32_t v[PW];
    uint32_t sum = 0;
#pragma unroll
    for (int k = 0; k < PW; ++k) {
      const int w = lane * PW + k;
      v[k] = w < n_words ? (uint32_t)__popc(bm[w]) : 0u;
      sum += v[k];
    }
    uint32_t run = wave_inclusive_sum(sum) - sum;
#pragma unroll
    for (int k = 0; k < PW; ++k) {
      wpre[lane * PW + k] = run;
      run += v[k];
    }
  }
  __syncthreads();
  uint64_t* dst = a.cand_out + ((size_t)p * a.h_kv + g) * a.cand_stride;
  // with the selection: the candidates' positions and scores by slot, their 1 / |k|, the greedy's
  // trace (the bounds are dead after pass 2; the ranked group's space after the cut)
  int32_t* cpos_l = reinterpret_cast<int32_t*>(ub);
  float* cst_l = ub + gram::kMaxCand;
  float* cinv_l = ub + 2 * gram::kMaxCand;
  uint32_t* trace_slot = reinterpret_cast<uint32_t*>(ub + 3 * gram::kMaxCand);
  uint32_t* trace_key = bins + kBitmapWords;
  for_each_entry([&](uint64_t e, int key) {
    if (e >= t_entry) {
      const uint32_t below = bm[key >> 5] & ((1u << (key & 31)) - 1u);
      const uint32_t rank = wpre[key >> 5] + (uint32_t)__popc(below);
      if (rank < (uint32_t)C) {  // exactly C entries are >= t_entry
        dst[rank] = e;
        if constexpr (SEL) {
          cpos_l[rank] = key;
          cst_l[rank] = key_float((uint32_t)(e >> 32));
        }
      }
    }
  });
  for (int i = C + tid; i < a.cand_stride; i += NT) dst[i] = 0ull;
  float den = c_max[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) den = fmaxf(den, c_max[w]);
  den = fmaxf(den, 1e-12f);
  if (tid == 0) a.cand_max[(size_t)p * a.h_kv + g] = den;
  if constexpr (SEL) {
    // ---- the selection of the unit (section 3.2, Eq. (2), (4)) from its C candidates, as the
    //      selection kernel runs it on the list just written: s~ = score / normaliser, the cosine
    //      triangle in the ring, the greedy on wave 0, then the outputs and the compaction
    __syncthreads();  // the slot arrays are complete; the ring's score keys are dead
    for (int c2 = tid; c2 < C; c2 += NT) cst_l[c2] = cst_l[c2] / den;
    gram::cosines<D, NW>(kg, cpos_l, C, cinv_l, reinterpret_cast<unsigned char*>(ring), tid);
    const float* tri = reinterpret_cast<const float*>(ring) + 1;
    constexpr int kRowVecs = D * 2 / 16;  // 16-byte vectors of a key row
    const uint4* k4 = reinterpret_cast<const uint4*>(a.k);
    const uint4* v4 = reinterpret_cast<const uint4*>(a.v);
    const size_t src0 = stat_base * kRowVecs;
    const size_t dst0 = ((size_t)p * a.h_kv + g) * a.out_rows * kRowVecs;
    if (wave == 0) {
      gram::Greedy gr;
      gr.init(cst_l, C, lane);
      if (a.sel_score) gr.run_for<true>(tri, C, bp, a.lambda2[p], lane, trace_slot, trace_key);
      else gr.run_for<false>(tri, C, bp, a.lambda2[p], lane, trace_slot, trace_key);
    } else if (a.k_out) {
      // meanwhile the other waves copy the kept tail (rows bp .. bp + keep_tail - 1 of the block)
      // and fetch the candidates' value rows into the caches for the compaction below
      const int t1 = tid - 64, nt1 = NT - 64;
      for (int e = t1; e < a.keep_tail * kRowVecs; e += nt1) {
        const int r = e / kRowVecs, cv = e % kRowVecs;
        const size_t sidx = src0 + (size_t)(L - a.keep_tail + r) * kRowVecs + cv;
        const size_t didx = dst0 + (size_t)(bp + r) * kRowVecs + cv;
        reinterpret_cast<uint4*>(a.k_out)[didx] = k4[sidx];
        reinterpret_cast<uint4*>(a.v_out)[didx] = v4[sidx];
      }
      // one dword per 128-byte line of each row, loaded straight into LDS words that nothing
      // reads (the histogram, cleared before its next use below)
      uint32_t* sink = red_hist + 64 * (wave & 7);
      for (int c2 = t1; c2 < C; c2 += nt1) {
        const uint4* row = v4 + src0 + (size_t)cpos_l[c2] * kRowVecs;
#pragma unroll
        for (int l = 0; l < kRowVecs; l += 8)
          __builtin_amdgcn_global_load_lds((gptr_t)(row + l), (lptr_t)sink, 4, 0, 0);
      }
      wait_vmem<0>();
    }
    __syncthreads();
    const size_t so0 = ((size_t)p * a.h_kv + g) * a.budget;
    for (int t = tid; t < a.budget; t += NT) {
      a.sel_idx[so0 + t] = t < bp ? cpos_l[trace_slot[t]] : -1;
      if (a.sel_score) a.sel_score[so0 + t] = t < bp ? key_float(trace_key[t]) : 0.f;
    }
    if (a.k_out) {
      // the admitted rows (the tail is copied)
      int32_t* srt = reinterpret_cast<int32_t*>(ring);  // the triangle is dead
      gram::admitted_in_order(trace_slot, cpos_l, bp, red_hist, srt, tid, NT);
      copy_kept_rows(k4, v4, srt, bp, 0, L, kRowVecs, src0, dst0,
                     reinterpret_cast<uint4*>(a.k_out), reinterpret_cast<uint4*>(a.v_out), tid, NT);
    }
  }
}

template <int D, int NB> struct PruneLaunch {
  static hipError_t run(const Shape& s, const StreamArgs& args, hipStream_t st) {
    const dim3 grid(1, s.h_kv, s.n_prob);
    if (args.sel_idx) {
      if (args.sigma_all) window_prune_kernel<D, NB, true, kWaves, 2, true><<<grid, kThreads, 0, st>>>(args);
      else window_prune_kernel<D, NB, false, kWaves, 2, true><<<grid, kThreads, 0, st>>>(args);
    } else {
      if (args.sigma_all) window_prune_kernel<D, NB, true, kWaves, 2, false><<<grid, kThreads, 0, st>>>(args);
      else window_prune_kernel<D, NB, false, kWaves, 2, false><<<grid, kThreads, 0, st>>>(args);
    }
    return hipGetLastError();
  }
};

}  // namespace
}  // namespace stream

int cand_code_stride(const Shape& s) {
  return (s.max_len + stream::kTileKeys - 1) / stream::kTileKeys * 32;
}

hipError_t launch_stream_window_cands(const Shape& s, const StreamPlan& plan, const void* q_win,
                                      const void* k, float scale, const float* lambda1, float w_mu,
                                      int budget, const int32_t* budgets, int cand_mult,
                                      int keep_tail, float* row_max, float* row_sum,
                                      uint64_t* cand_out, float* cand_max, int cand_stride,
                                      uint32_t* codes, bool sigma_all, const CandSelect* sel,
                                      hipStream_t stream) {
  if (plan.max_segs != 1 || !cand_out || !cand_max || !codes || s.max_len > kCandMaxLen)
    return hipErrorInvalidValue;
  if (sel && (!sel->lambda2 || !sel->sel_idx || (sel->k_out && (!sel->v || !sel->v_out))))
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
  a.codes = codes;
  a.code_stride = cand_code_stride(s);
  if (sel) {
    a.lambda2 = sel->lambda2;
    a.sel_idx = sel->sel_idx;
    a.sel_score = sel->sel_score;
    a.v = static_cast<const uint16_t*>(sel->v);
    a.k_out = static_cast<uint16_t*>(sel->k_out);
    a.v_out = static_cast<uint16_t*>(sel->v_out);
    a.out_rows = sel->out_rows;
  }
  return stream::launch_for_shape<stream::PruneLaunch>(s, a, stream);
}

}  // namespace kv
