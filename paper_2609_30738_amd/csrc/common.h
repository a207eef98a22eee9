// Device-side building blocks shared by the gfx950 kernels: element types, the 32x32 MFMA tile
// and its operand fragments, wave-level reductions.
//
// MFMA tile conventions (v_mfma_f32_32x32x16_bf16 and v_mfma_f32_32x32x2_f32, wave64):
//   operand fragments: lane l carries row/column (l % 32) of its operand and the K-half (l / 32);
//     for bf16 one K step covers 16 elements, lane half h holds elements [16 s + 8 h, 16 s + 8 h + 8);
//     for f32 one K step covers 2 elements; lane half h holds element h * (D / 2) + s, so every lane
//     reads D / 2 contiguous floats.  A and B use the same K mapping, so every pairing of lanes sums
//     a full dot product.
//   accumulator: lane l, register j holds D[8 (j / 4) + 4 (l / 32) + (j % 4)][l % 32].
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.h"

namespace kv {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int DT> struct Elem;
template <> struct Elem<kDtF32> { typedef float T; };
template <> struct Elem<kDtBf16> { typedef uint16_t T; };

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// Row of the 32x32 accumulator held by register j of lane l.
__device__ __forceinline__ int acc_row(int j, int lane) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

// All K-step fragments of one 32-wide operand slab (32 rows of D elements) for this lane.
template <int DT, int D> struct Frags;

template <int D> struct Frags<kDtBf16, D> {
  static constexpr int NS = D / 16;
  bf16x8_t v[NS];
  // row: pointer to this lane's row (D elements), half: lane / 32
  __device__ __forceinline__ void load_global(const uint16_t* row, int half) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      v[s] = *reinterpret_cast<const bf16x8_t*>(row + 16 * s + 8 * half);
  }
  __device__ __forceinline__ void load_lds(const uint16_t* row, int half) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      v[s] = *reinterpret_cast<const bf16x8_t*>(row + 16 * s + 8 * half);
  }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int s = 0; s < NS; ++s) v[s] = bf16x8_t{0, 0, 0, 0, 0, 0, 0, 0};
  }
};

template <int D> struct Frags<kDtF32, D> {
  static constexpr int NS = D / 2;
  float v[NS];
  __device__ __forceinline__ void load_global(const float* row, int half) {
    const float4* src = reinterpret_cast<const float4*>(row + half * (D / 2));
#pragma unroll
    for (int q = 0; q < NS / 4; ++q) {
      float4 x = src[q];
      v[4 * q + 0] = x.x;
      v[4 * q + 1] = x.y;
      v[4 * q + 2] = x.z;
      v[4 * q + 3] = x.w;
    }
  }
  __device__ __forceinline__ void load_lds(const float* row, int half) { load_global(row, half); }
  __device__ __forceinline__ void zero() {
#pragma unroll
    for (int s = 0; s < NS; ++s) v[s] = 0.f;
  }
};

__device__ __forceinline__ f32x16_t mfma_step(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16_t mfma_step(float a, float b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// acc = A * B^T over the full head dimension: A rows from `a`, B rows from `b`.
template <int DT, int D>
__device__ __forceinline__ f32x16_t mfma_tile(const Frags<DT, D>& a, const Frags<DT, D>& b) {
  f32x16_t acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < Frags<DT, D>::NS; ++s) acc = mfma_step(a.v[s], b.v[s], acc);
  return acc;
}

// Order-preserving 32-bit key of a float: a larger key means a larger value (-0 below +0; NaNs
// with the sign bit clear above +inf, with it set below -inf).
__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// The float whose order key is k (the inverse of order_key, bit for bit).
__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}

// Candidate entry: the order key of a base score and its position; a larger entry means a larger
// score, then a lower position (the selection's order and tie rule).  0 is no entry.
__device__ __forceinline__ uint64_t cand_entry(uint32_t okey, uint32_t pos) {
  return ((uint64_t)okey << 32) | (uint32_t)(0xFFFFFFFFu - pos);
}
__device__ __forceinline__ uint32_t cand_entry_pos(uint64_t e) { return 0xFFFFFFFFu - (uint32_t)e; }

// Add one to hist[digit] (LDS) for every active lane.  The digit of the first active lane is
// counted with one ballot and a single LDS add (the common case: most scores share their leading
// digits); lanes with other digits use LDS atomics, which handle scattered digits without
// conflicts.  Every lane of the wave must call it.
__device__ __forceinline__ void wave_hist_add(uint32_t* hist, uint32_t digit, bool active) {
  const uint64_t act = __ballot(active);
  if (act == 0) return;
  const int leader = __ffsll((unsigned long long)act) - 1;
  const uint32_t dl = __builtin_amdgcn_readlane(digit, leader);
  const uint64_t same = __ballot(active && digit == dl);
  if ((int)(threadIdx.x & 63) == leader) atomicAdd(&hist[dl], (uint32_t)__popcll(same));
  if (active && digit != dl) atomicAdd(&hist[digit], 1u);
}

// Ascending bitonic sort of v[0, n2) (n2 a power of two) by the nt threads of the workgroup; starts and ends with
// the workgroup synchronised.
template <typename V>
__device__ __forceinline__ void bitonic_sort(V* v, int n2, int tid, int nt) {
  for (int size = 2; size <= n2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < n2; i += nt) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const V a = v[i], b = v[j];
          if ((a > b) == up) {
            v[i] = b;
            v[j] = a;
          }
        }
      }
      __syncthreads();
    }
  }
}

// Value of the lane l ^ 32 (the other K-half / the other 16 accumulator rows).
__device__ __forceinline__ float swap_halves(float x) {
  return __shfl_xor(x, 32, 64);
}

// The largest value over the 64 lanes (quiet NaNs are ignored: NaN only if every lane holds NaN),
// as a uniform value: maxima within rows of 16 lanes, then across rows with row broadcasts into
// lane 63, each step one v_max_f32 with a DPP source (two wait states before each, for the VGPR it
// reads).
__device__ __forceinline__ float wave_max_uniform(float v) {
  asm("s_nop 1\n\t"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\t"
      "v_max_f32_dpp %0, %0, %0 quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\t"
      "v_max_f32_dpp %0, %0, %0 row_ror:4 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\t"
      "v_max_f32_dpp %0, %0, %0 row_ror:8 row_mask:0xf bank_mask:0xf\n\t"
      "s_nop 1\n\t"
      "v_max_f32_dpp %0, %0, %0 row_bcast:15 row_mask:0xa bank_mask:0xf\n\t"
      "s_nop 1\n\t"
      "v_max_f32_dpp %0, %0, %0 row_bcast:31 row_mask:0xc bank_mask:0xf\n\t"
      "s_nop 1"
      : "+v"(v));
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__float_as_uint(v), 63));
}

// Online-softmax pair merge in base-2 units: (m, z) represents z * 2^m.
__device__ __forceinline__ void merge_mz(float& m, float& z, float m2, float z2) {
  float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;  // both empty
  float a = (m == -INFINITY) ? 0.f : z * __builtin_amdgcn_exp2f(m - mn);
  float b = (m2 == -INFINITY) ? 0.f : z2 * __builtin_amdgcn_exp2f(m2 - mn);
  m = mn;
  z = a + b;
}

}  // namespace kv
