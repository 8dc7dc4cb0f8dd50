// Device helpers shared by the gfx950 kernels: int8 MFMA fragments, 16-lane DPP
// row reductions, the Eq. 2 quantiser and the softmax exponential.
//
// Fixed evaluation order used by every kernel (the paper fixes the fp32 precision
// of activations, scales and biases, Section 4.1, but not an order):
//   - sums over features are pairwise with stride halving: element c is first
//     added to element c + w/2, then the first half is reduced the same way;
//   - sums over attention neighbours and over tokens run in ascending index;
//   - a head's dot product is a multiply then fused multiply-adds, ascending;
//   - the softmax is taken in base 2 on query rows pre-scaled by log2(e)/sqrt(d_h);
//   - only the multiply-adds written as fmaf are fused (built with
//     -ffp-contract=off), division is correctly rounded.
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

// Two k-steps of mfma_i8_16x16x32 as one v_mfma_i32_16x16x64_i8 (twice the k per instruction,
// the same issue cost): lane l passes its 8 A bytes of step 0 then those of step 1, and its B
// bytes the same way.  The instruction pairs A and B bytes of equal position within a lane, so
// the result is the sum of the two steps' products; int32 sums of int8 products are exact in
// any order.
__device__ __forceinline__ v4i mfma_i8_16x16x64(long a0, long a1, long b0, long b1, v4i c) {
  const v4i a = v4i{(int)a0, (int)(a0 >> 32), (int)a1, (int)(a1 >> 32)};
  const v4i b = v4i{(int)b0, (int)(b0 >> 32), (int)b1, (int)(b1 >> 32)};
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// c + the products of S k-steps, A and B fragments of step s from a(s) and b(s): pairs of steps
// on the 64-deep instruction, an odd last step on the 32-deep one.
template <int S, class FA, class FB>
__device__ __forceinline__ v4i mfma_i8_steps(FA a, FB b, v4i c) {
#pragma unroll
  for (int s = 0; s + 1 < S; s += 2) c = mfma_i8_16x16x64(a(s), a(s + 1), b(s), b(s + 1), c);
  if constexpr (S % 2 == 1) c = mfma_i8_16x16x32(a(S - 1), b(S - 1), c);
  return c;
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

// Eq. 2 code of one value: the exact product x * inv rounded once, half to even, to an
// integer.  fma(x, inv, 1.5 * 2^23) performs that rounding (the sum lies in [2^23, 2^24),
// where the fp32 spacing is 1, and 1.5 * 2^23 is even), and the code sits in the low
// bits: the low byte of the result's bit pattern is the int8 code.  With alpha = max|x|
// and inv = fp32(127 / alpha) the product is at most 127 (1 + 2^-23) in magnitude, so the
// code is already within [-127, 127] and the clip of Eq. 2 never changes it.
__device__ __forceinline__ uint32_t quant_bits(float x, float inv) {
  return __builtin_bit_cast(uint32_t, __builtin_fmaf(x, inv, 0x1.8p23f));
}
__device__ __forceinline__ int8_t quant_code(float x, float inv) { return (int8_t)quant_bits(x, inv); }

// Eq. 2 codes of four ReLU outputs from the code patterns of the pre-activations: the low 16
// bits of a quant_bits pattern are the code as an int16 (1.5 * 2^23 + c for |c| <= 127), so
// max(code, 0) on two codes at a time (v_pk_max_i16) equals the code of max(x, 0) (inv >= 0, and
// rounding is monotone); returns the four codes as bytes 0..3.
typedef short short2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack4_relu(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
  short2_t lo = __builtin_bit_cast(short2_t, __builtin_amdgcn_perm(b1, b0, 0x05040100u));
  short2_t hi = __builtin_bit_cast(short2_t, __builtin_amdgcn_perm(b3, b2, 0x05040100u));
  lo = __builtin_elementwise_max(lo, (short2_t){0, 0});
  hi = __builtin_elementwise_max(hi, (short2_t){0, 0});
  return __builtin_amdgcn_perm(__builtin_bit_cast(uint32_t, hi), __builtin_bit_cast(uint32_t, lo), 0x06040200u);
}

// 2^x for the base-2 attention softmax: clamp to [-125, 128] (the result stays a normal
// number, or is +inf from 2^128 on; a NaN argument gives 2^-125, since the median of three
// with a NaN operand is the minimum of the other two), split x = k + r with k = floor(x)
// and r = fract(x) = min(x - floor(x), 1 - 2^-24) in [0, 1) (v_fract_f32; v_cvt_flr_i32_f32
// gives k as an integer in one instruction), 2^r by p(r) = 1 + a1 r + ... + a5 r^5, the
// degree-5 polynomial with constant term 1 of least maximum relative error against 2^r on
// [0, 1] (5.2e-8 before rounding its coefficients to fp32), Horner, then an exact scaling by
// 2^k.  Relative error below 3e-7; exact at integers.
__device__ __forceinline__ float softmax_exp2(float x) {
  x = __builtin_amdgcn_fmed3f(x, -125.0f, 128.0f);
  const float r = __builtin_amdgcn_fractf(x);
  int k;
  asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(k) : "v"(x));
  float p = 0x1.f08ff4p-10f;
  p = __builtin_fmaf(p, r, 0x1.2552ccp-7f);
  p = __builtin_fmaf(p, r, 0x1.c98e60p-5f);
  p = __builtin_fmaf(p, r, 0x1.ebd24ep-3f);
  p = __builtin_fmaf(p, r, 0x1.62e4f0p-1f);
  p = __builtin_fmaf(p, r, 1.0f);
  return __builtin_ldexpf(p, k);
}

// 1/s correctly rounded for s in [2^-64, 2^64]: v_rcp_f32, then one Newton step with fused
// multiply-adds, r + r (1 - s r).  Checked on gfx950 against the IEEE division for every fp32
// s of that range (no difference).  The softmax sum S is always in it where it is inverted: the
// unshifted sums are kept only inside [2^-64, 2^64], and a shifted sum lies in [1, count].
__device__ __forceinline__ float recip_softmax_sum(float s) {
  const float r = __builtin_amdgcn_rcpf(s);
  return __builtin_fmaf(__builtin_fmaf(-s, r, 1.0f), r, r);
}

// The Eq. 2 scale factor fp32(127 / a) for a = alpha >= 0, and 0 for a = 0.  With a = m 2^e,
// m in [1/2, 1) (v_frexp_mant_f32 / v_frexp_exp_i32_f32, denormals included): q0 = 127
// v_rcp_f32(m), then the remainder correction q0 + r (127 - m q0) with fused multiply-adds, which
// equals the IEEE quotient 127 / m for every fp32 m of [2^-100, 2^100] (checked on gfx950), and
// 127 / a = (127 / m) 2^-e is an exact rescaling: 127 / a is never below 2^-122, so the result is
// normal or overflows to +inf exactly where the quotient does.
__device__ __forceinline__ float inv127(float a) {
  const float m = __builtin_amdgcn_frexp_mantf(a);
  const int e = __builtin_amdgcn_frexp_expf(a);
  const float r = __builtin_amdgcn_rcpf(m);
  const float q0 = 127.0f * r;
  const float q = __builtin_fmaf(__builtin_fmaf(-m, q0, 127.0f), r, q0);
  return a == 0.0f ? 0.0f : __builtin_ldexpf(q, -e);
}

// 1/sqrt(v), v > 0, for LayerNorm: seed 0x5F3759DF - (bits(v) >> 1) (Lomont 2003), then
// three Newton steps y <- y (3/2 - (v/2) y^2).
__device__ __forceinline__ float ln_rsqrt(float v) {
  const float h = 0.5f * v;
  float y = __builtin_bit_cast(float, 0x5F3759DFu - (__builtin_bit_cast(uint32_t, v) >> 1));
#pragma unroll
  for (int it = 0; it < 3; ++it) {
    float t = y * y;
    t = __builtin_fmaf(-h, t, 1.5f);
    y = y * t;
  }
  return y;
}

// A head's dot product: q[0] k[0], then fused multiply-adds in ascending order; a head of 16
// dimensions takes its two 8-dimension halves that way and adds them (low + high), the order
// in which two lanes that each hold one half combine them.
template <int W>
__device__ __forceinline__ float dot_seq(const float *q, const float *k) {
  float s = q[0] * k[0];
#pragma unroll
  for (int t = 1; t < W; ++t) s = __builtin_fmaf(q[t], k[t], s);
  return s;
}
template <int DH>
__device__ __forceinline__ float head_dot(const float (&q)[DH], const float *k) {
  if constexpr (DH == 16) return dot_seq<8>(q, k) + dot_seq<8>(q + 8, k + 8);
  else return dot_seq<DH>(q, k);
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
