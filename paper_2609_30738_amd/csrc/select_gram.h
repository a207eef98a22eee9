// The Gram-matrix form of the greedy selection (section 3.2, Eq. (2), (4)) for at most 256 bf16
// candidates of one unit, shared by the selection kernel (select.hip) and the window kernel that
// cuts the candidates and selects in the same launch (stream_prune.hip), so that both give the same
// bits:
//   cosines  - the candidates' key rows staged in LDS, their dot products with MFMA (32 x 32 blocks
//              of the upper triangle), scaled by the inverse norms into a strict upper triangle of
//              cosines in LDS (over the staged rows);
//   Greedy   - one wave runs every step: lane l holds slots l, l + 64, l + 128, l + 192 with their
//              s~ and running largest cosine to the admitted slots;
//   ranks    - the admitted slots in ascending order (the slots are in position order) for the
//              compaction of the kept rows.
#pragma once

#include <float.h>

#include "common.h"
#include "compact_rows.h"

namespace kv {
namespace gram {

constexpr int kMaxCand = kCandSelectMax;   // candidates of the Gram greedy (4 per lane of a wave)
constexpr int kSlots = kMaxCand / 64;
constexpr int kMaxBlocks = (kMaxCand / 32) * (kMaxCand / 32 + 1) / 2;  // 32 x 32 blocks, I <= J
constexpr int kSlotWords = kMaxCand / 32;  // bitmap words over the slots

// LDS of the staged key rows and of the triangle (one guard entry first, then the c (c - 1) / 2
// cosines, then one word per lane that the stores of lanes without an entry go to); the triangle
// is written over the rows.
template <int D> __host__ __device__ constexpr size_t stage_bytes(int c) {
  return (size_t)c * D * 2;
}
__host__ __device__ constexpr size_t tri_bytes(int c) {
  return ((size_t)c * (c > 0 ? c - 1 : 0) / 2 + 1 + 64) * 4;
}
template <int D> __host__ __device__ constexpr size_t region_bytes(int c) {
  return stage_bytes<D>(c) > tri_bytes(c) ? stage_bytes<D>(c) : tri_bytes(c);
}

// Cosine of slots (i, j), i < j, at tri[row_off(i, c) + j] (the strict upper triangle row by row;
// i (2c - i - 1) is even).  With i == j the index is that of another entry or of the guard (-1).
__device__ __forceinline__ int row_off(int i, int c) { return (i * (2 * c - i - 1)) / 2 - i - 1; }

// The triangle of the C candidates (slots in cpos[0, C), positions of rows of kg, D bf16 each):
// tri[row_off(i, C) + j] = (k_i . k_j / |k_i|) / |k_j| for i < j (a zero key has 1 / |k| = 0,
// hence cosine 0 to everything; a non-finite product counts as 0), and cinv[i] = 1 / |k_i|.
// region: region_bytes<D>(C) bytes of LDS (16-byte aligned); the triangle starts one float after it
// (the guard).  Every thread of the workgroup (NW >= 8 waves) calls it after cpos is visible; it
// ends synchronised.
typedef const __attribute__((address_space(1))) void* gptr;
typedef __attribute__((address_space(3))) void* lptr;

template <int D, int NW>
__device__ __forceinline__ void cosines(const uint16_t* __restrict__ kg, const int32_t* cpos, int C,
                                        float* cinv, unsigned char* region, int tid) {
  constexpr int NT = NW * 64, CH = D / 8, kSlices = D / 16;
  constexpr int kPer = kMaxCand * CH / NT;  // 16-byte chunks per thread
  constexpr int kBlk = (kMaxBlocks + NW - 1) / NW;
  static_assert(kMaxCand * CH % NT == 0, "whole chunks per thread");
  static_assert(NW >= 8, "one thread per (row, half) for the norms");
  const int lane = tid & 63, l32 = lane & 31, half = lane >> 5, wave = tid >> 6;
  uint16_t* rows = reinterpret_cast<uint16_t*>(region);
  // 16-byte chunk ch of staged row r sits in slot r CH + (ch ^ (r % CH)) (a rotation per row that
  // spreads the MFMA operand reads of consecutive rows over the banks).  Load i of a wave fills
  // slots 64 (wave kPer + i) .. + 63 straight from global memory, every load in flight at once.
  auto at = [&](int r, int ch) { return rows + 8 * (r * CH + (ch ^ (r % CH))); };
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int s0 = 64 * (wave * kPer + i), r = (s0 + lane) / CH;
    const int ch = ((s0 + lane) % CH) ^ (r % CH);
    if (r < C)
      __builtin_amdgcn_global_load_lds((gptr)(kg + (size_t)cpos[r] * D + 8 * ch),
                                       (lptr)(rows + 8 * s0), 16, 0, 0);
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // |k|^2 of row tid / 2: this thread's 8-element halves of every 16-element slice, then the
  // other halves from the neighbouring lane
  if (tid < 2 * C) {
    typedef __bf16 __attribute__((ext_vector_type(2))) bf2;
    const int r = tid >> 1, h = tid & 1;
    float n2 = 0.f;
#pragma unroll
    for (int sl = 0; sl < kSlices; ++sl) {
      const uint4 w = *reinterpret_cast<const uint4*>(at(r, 2 * sl + h));
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int u = 0; u < 4; ++u)
        n2 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf2, ws[u]), __builtin_bit_cast(bf2, ws[u]), n2, false);
    }
    n2 += __shfl_xor(n2, 1, 64);
    if (h == 0) cinv[r] = n2 > 0.f ? 1.f / sqrtf(n2) : 0.f;
  }
  // the dot products of blocks (I, J), I <= J: each wave takes a run of consecutive blocks of the
  // row-major enumeration (mostly one block row, so that the A operand is read once per slice)
  const int nb = (C + 31) / 32, n_blk = nb * (nb + 1) / 2;
  const int per = n_blk / NW, extra = n_blk % NW;
  const int first = wave * per + min(wave, extra), count = per + (wave < extra ? 1 : 0);
  int blk_i[kBlk], blk_j[kBlk];
  {
    int I = 0, rem = first;
    while (I < nb && rem >= nb - I) {
      rem -= nb - I;
      ++I;
    }
#pragma unroll
    for (int u = 0; u < kBlk; ++u) {
      blk_i[u] = u < count ? I : nb;  // nb: no block
      blk_j[u] = I + rem;
      if (++rem >= nb - I) {
        ++I;
        rem = 0;
      }
    }
  }
  f32x16_t acc[kBlk];
#pragma unroll
  for (int u = 0; u < kBlk; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[u][r] = 0.f;
#pragma unroll
  for (int sl = 0; sl < kSlices; ++sl) {
    bf16x8_t a = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
    int a_row = -1;  // the block row whose fragment `a` holds (wave-uniform)
#pragma unroll
    for (int u = 0; u < kBlk; ++u) {
      if (blk_i[u] < nb) {
        if (blk_i[u] != a_row) {
          a = *reinterpret_cast<const bf16x8_t*>(at(min(32 * blk_i[u] + l32, C - 1), 2 * sl + half));
          a_row = blk_i[u];
        }
        const bf16x8_t b =
            blk_j[u] == blk_i[u]
                ? a
                : *reinterpret_cast<const bf16x8_t*>(at(min(32 * blk_j[u] + l32, C - 1), 2 * sl + half));
        acc[u] = mfma_step(a, b, acc[u]);
      }
    }
  }
  __syncthreads();  // every row is read and every norm written: the triangle goes over the rows
  float* tri = reinterpret_cast<float*>(region) + 1;
  if (tid == 0) tri[-1] = 0.f;  // the guard
#pragma unroll
  for (int u = 0; u < kBlk; ++u) {
    if (blk_i[u] < nb) {
      // register jj holds row i = i0 + 8 (jj / 4) + jj % 4 of column j; row_off(i + 1) =
      // row_off(i) + C - 2 - i.  cinv is read up to 32 nb - 1 (past C: values not used).
      const int j = 32 * blk_j[u] + l32;
      const int i0 = 32 * blk_i[u] + 4 * half;
      const float inv_j = cinv[j];
      float inv_i[16];
#pragma unroll
      for (int jj = 0; jj < 16; ++jj) inv_i[jj] = cinv[i0 + 8 * (jj >> 2) + (jj & 3)];
      if (blk_i[u] < blk_j[u] && 32 * blk_j[u] + 32 <= C) {
        // a whole block above the diagonal: every register is an entry
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ir = i0 + 8 * r;
          int idx = row_off(ir, C) + j;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float cs = acc[u][4 * r + e] * inv_i[4 * r + e] * inv_j;
            tri[idx] = __builtin_isfinite(cs) ? cs : 0.f;
            idx += C - 2 - (ir + e);
          }
        }
      } else {
        // a lane without an entry (i >= j, j >= C) stores to its own word past the triangle
        const int spare = C * (C - 1) / 2 + lane;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ir = i0 + 8 * r;
          int idx = row_off(ir, C) + j;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float cs = acc[u][4 * r + e] * inv_i[4 * r + e] * inv_j;
            tri[j < C && ir + e < j ? idx : spare] = __builtin_isfinite(cs) ? cs : 0.f;
            idx += C - 2 - (ir + e);
          }
        }
      }
    }
  }
  __syncthreads();
}

// The greedy of one wave over the triangle: bp steps (bp <= C), each admitting the slot of largest
// fmaf(lam2, corr, s~) (ties to the lower slot), corr being a slot's largest cosine to the slots
// admitted before (0 before the first).
struct Greedy {
  float st[kSlots], corr[kSlots];  // s~ (-inf once admitted or past C), running corr
  int cq[kSlots], offq[kSlots];    // slot (clamped to C - 1), its row offset
  int cq4[kSlots], off4[kSlots];   // the same in bytes
  int last = -1;                   // the last admitted slot

  // cst[c]: s~ of slot c (finite after the clamp: a NaN or -inf score still ranks above the
  // admitted slots, as the lowest finite one)
  __device__ __forceinline__ void init(const float* cst, int C, int lane) {
#pragma unroll
    for (int q = 0; q < kSlots; ++q) {
      const int c = lane + 64 * q;
      cq[q] = min(c, C - 1);
      offq[q] = row_off(cq[q], C);
      cq4[q] = 4 * cq[q];
      off4[q] = 4 * offq[q];
      st[q] = c < C ? fmaxf(cst[c], -FLT_MAX) : -INFINITY;
      corr[q] = 0.f;
    }
  }
  // The cosine of every slot to slot `s` (read for all slots at once; slot s itself and the slots
  // past C read some entry of the triangle or the guard, never used).
  __device__ __forceinline__ void cos_to(const float* tri, int s, int C, float (&gv)[kSlots]) const {
    const int off_s = row_off(s, C);
#pragma unroll
    for (int q = 0; q < kSlots; ++q) gv[q] = tri[cq[q] <= s ? offq[q] + s : off_s + cq[q]];
  }
  // Steps t = 0 .. bp - 1: trace_slot[t] = the admitted slot, and with KEYS trace_key[t] = the
  // order key of its score (the wave's largest score; -inf's key when no live slot is left, in
  // which case slot C - 1 is recorded).  A step: the largest score of the wave, then the lowest
  // slot that holds it (one ballot per slot group q, whose lanes hold slots 64 q + lane), then
  // its s~ cleared and the cosines to it read for the next step (group q below the admitted
  // slot's group: every lane's slot lies before it, so the entry is in its column; groups above:
  // in its row; its own group: by lane).  Without CHECK (|lam2| <= 1e30: a live score
  // fmaf(lam2, corr <= 1, s~ >= -FLT_MAX) stays finite) the test for a live slot is left out.
  template <bool KEYS, bool CHECK>
  __device__ __forceinline__ void run(const float* tri, int C, int bp, float lam2, int lane,
                                      uint32_t* trace_slot, uint32_t* trace_key) {
    float gv[kSlots];
    for (int t = 0; t < bp; ++t) {
      if (t > 0) {
#pragma unroll
        for (int q = 0; q < kSlots; ++q) corr[q] = __builtin_elementwise_maximum(corr[q], gv[q]);
      }
      float sc[kSlots];
#pragma unroll
      for (int q = 0; q < kSlots; ++q) sc[q] = fmaf(lam2, corr[q], st[q]);
      static_assert(kSlots == 4, "four slot groups");
      const float lm = __builtin_elementwise_maximum(__builtin_elementwise_maximum(sc[0], sc[1]),
                                                     __builtin_elementwise_maximum(sc[2], sc[3]));
      const float wm = wave_max_uniform(lm);
      int slot = C - 1;  // no live slot left (every score -inf or NaN)
      if (!CHECK || wm > -INFINITY) {
        uint64_t m = __ballot(sc[0] == wm);
        int q = 0;
#pragma unroll
        for (int u = 1; u < kSlots; ++u) {
          if (m == 0) {
            m = __ballot(sc[u] == wm);
            q = u;
          }
        }
        slot = 64 * q + (__ffsll((unsigned long long)m) - 1);
      }
      last = __builtin_amdgcn_readfirstlane(slot);
      // the step's record (every lane stores the same value)
      trace_slot[t] = (uint32_t)last;
      if constexpr (KEYS) trace_key[t] = wm_key(wm, sc);
      // slot `last` leaves the race; the cosines of every slot to it for the next step
      const int ql = last >> 6, ll = last & 63;
#pragma unroll
      for (int q = 0; q < kSlots; ++q) st[q] = q == ql && lane == ll ? -INFINITY : st[q];
      if (t + 1 < bp) {
        // byte addresses: its column (slot < last) at + 4 row_off(slot), its row at + 4 slot
        const char* col = reinterpret_cast<const char*>(tri + last);
        const char* row = reinterpret_cast<const char*>(tri + row_off(last, C));
#pragma unroll
        for (int q = 0; q < kSlots; ++q) {
          const bool in_col = q < ql || (q == ql && lane <= ll);
          gv[q] = *reinterpret_cast<const float*>(in_col ? col + off4[q] : row + cq4[q]);
        }
      }
    }
  }
  // run<KEYS, CHECK> with CHECK decided by lam2
  template <bool KEYS>
  __device__ __forceinline__ void run_for(const float* tri, int C, int bp, float lam2, int lane,
                                          uint32_t* trace_slot, uint32_t* trace_key) {
    if (__builtin_fabsf(lam2) <= 1e30f) run<KEYS, false>(tri, C, bp, lam2, lane, trace_slot, trace_key);
    else run<KEYS, true>(tri, C, bp, lam2, lane, trace_slot, trace_key);
  }

  // The order key of the step's score: the largest score of the wave; a largest score of zero is
  // +0 if some lane's first zero (in slot order) is +0, else -0; -inf's key when no score is live.
  __device__ __forceinline__ static uint32_t wm_key(float wm, const float (&sc)[kSlots]) {
    if (!(wm > -INFINITY)) return order_key(-INFINITY);
    if (wm == 0.f) {
      bool found = false, pos = false;
#pragma unroll
      for (int q = 0; q < kSlots; ++q) {
        if (!found && sc[q] == 0.f) pos = !__builtin_signbit(sc[q]);
        found = found || sc[q] == 0.f;
      }
      return order_key(__ballot(pos) ? 0.f : -0.f);
    }
    return order_key(wm);
  }

};

// The positions of the admitted slots (trace_slot[0, bp), slots < C <= kMaxCand) in ascending
// order into srt[0, bp): a bitmap over the slots and the prefix counts of its words rank them
// (the candidates are in position order).  bits: kSlotWords words of LDS.  Every thread of the
// workgroup calls it; it starts and ends synchronised.
__device__ __forceinline__ void admitted_in_order(const uint32_t* trace_slot, const int32_t* cpos,
                                                  int bp, uint32_t* bits, int32_t* srt, int tid,
                                                  int nt) {
  for (int w = tid; w < kSlotWords; w += nt) bits[w] = 0u;
  __syncthreads();
  for (int t = tid; t < bp; t += nt) atomicOr(&bits[trace_slot[t] >> 5], 1u << (trace_slot[t] & 31));
  __syncthreads();
  for (int t = tid; t < bp; t += nt) {
    const uint32_t sl = trace_slot[t];
    uint32_t rank = (uint32_t)__popc(bits[sl >> 5] & ((1u << (sl & 31)) - 1u));
    for (uint32_t w = 0; w < (sl >> 5); ++w) rank += (uint32_t)__popc(bits[w]);
    srt[rank] = cpos[sl];
  }
  __syncthreads();
}

}  // namespace gram
}  // namespace kv
