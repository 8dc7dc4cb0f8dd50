// Device helpers shared by the gfx950 kernels: int8 MFMA fragments, 16-lane DPP
// row reductions, the Eq. 2 quantiser and the softmax exponential.
//
// Fixed evaluation order used by every kernel (the paper fixes the fp32 precision
// of activations, scales and biases, Section 4.1, but not an order):
//   - sums over features are pairwise with stride halving: element c is first
//     added to element c + w/2, then the first half is reduced the same way;
//   - sums over attention neighbours and over tokens run in ascending index;
//   - only the multiply-adds written as fmaf are fused (built with
//     -ffp-contract=off), division and square root are correctly rounded.
#pragma once

#include <cstdint>

#include <hip/hip_runtime.h>

namespace aecct {

typedef int v4i __attribute__((ext_vector_type(4)));

// D(16x16 int32) += A(16x32 int8) * B(32x16 int8).  Lane l holds A row (l & 15),
// B column (l & 15), inputs k = 8 * (l >> 4) .. +7 (8 bytes); D rows 4 * (l >> 4) + i,
// column (l & 15).
__device__ __forceinline__ v4i mfma_i8_16x16x32(long a, long b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x32_i8(a, b, c, 0, 0, 0);
}

// Lane l of a 16-lane DPP row reads lane (l +- N) mod 16 of the same row.
template <int N>
__device__ __forceinline__ float row_rotate(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x120 + N, 0xf, 0xf, true));
}

// Pairwise (stride 8, 4, 2, 1) sum of the 16 values of a DPP row; every lane gets the
// result.  After a step with stride s each lane holds the partial for (lane mod s), so
// rotating by s/2 pairs exactly the partials the pairwise order pairs (addition
// commutes bit for bit).
__device__ __forceinline__ float row16_sum(float v) {
  v = v + row_rotate<8>(v);
  v = v + row_rotate<4>(v);
  v = v + row_rotate<2>(v);
  v = v + row_rotate<1>(v);
  return v;
}

__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, row_rotate<8>(v));
  v = fmaxf(v, row_rotate<4>(v));
  v = fmaxf(v, row_rotate<2>(v));
  v = fmaxf(v, row_rotate<1>(v));
  return v;
}

// Pairwise sum of T per-lane values (T a power of two), stride halving, in place.
template <int T>
__device__ __forceinline__ float lane_tree(float (&v)[T]) {
#pragma unroll
  for (int h = T / 2; h >= 1; h /= 2) {
#pragma unroll
    for (int t = 0; t < h; ++t) v[t] = v[t] + v[t + h];
  }
  return v[0];
}

// Eq. 2 code of one value: round-half-even(x * (127 / alpha)).  With alpha = max|x| the
// product is at most 127 (1 + 2^-23) in magnitude, so the code is already within
// [-127, 127] and the clip of Eq. 2 never changes it.
__device__ __forceinline__ int quant_code(float x, float inv) { return (int)__builtin_rintf(x * inv); }

// exp(x), x <= 0, for the attention softmax: Cody & Waite reduction x = k ln2 + r with
// ln2 split into a 16-bit head (k * head exact for |k| < 128) and an fp32 tail, the
// degree-7 Taylor polynomial of e^r (coefficients fp32(1/j!)) by Horner, and an exact
// scaling by 2^k.  Arguments below -80 give 0.
__device__ __forceinline__ float softmax_exp(float x) {
  if (x < -80.0f) return 0.0f;
  const float k = __builtin_rintf(x * 0x1.715476p+0f);
  float r = __builtin_fmaf(-k, 0x1.62e4p-1f, x);
  r = __builtin_fmaf(-k, 0x1.7f7d1cp-20f, r);
  float p = 0x1.a01a02p-13f;
  p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);
  p = __builtin_fmaf(p, r, 0x1.111112p-7f);
  p = __builtin_fmaf(p, r, 0x1.555556p-5f);
  p = __builtin_fmaf(p, r, 0x1.555556p-3f);
  p = __builtin_fmaf(p, r, 0.5f);
  p = __builtin_fmaf(p, r, 1.0f);
  p = __builtin_fmaf(p, r, 1.0f);
  return __builtin_ldexpf(p, (int)k);
}

// 8 ternary codes (2 bits each, 00 -> 0, 01 -> +1, 11 -> -1, code e in bits 2e..2e+1)
// to 8 int8 bytes, byte e = code e.
__device__ __forceinline__ uint64_t unpack_ternary8(uint32_t pk) {
  uint64_t out = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int v = ((int)(pk << (30 - 2 * e))) >> 30;   // sign-extended 2-bit field
    out |= (uint64_t)(uint8_t)(int8_t)v << (8 * e);
  }
  return out;
}

}  // namespace aecct
