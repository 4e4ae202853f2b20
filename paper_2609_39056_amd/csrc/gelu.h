// GELU in fp32 with a fixed operation sequence, and the STATIC 8-bit
// quantization of its bf16 output for the next linear.  The quantized DiT
// keeps GELU in bf16 between the MLP's up and down projections (App. D); the
// up projection's epilogue (kEpiGelu) and sq_gelu_bf16 both evaluate it here,
// one IEEE fp32 operation at a time (the library builds with fp contraction
// off and correctly rounded fp32 division), so every caller of these
// functions gets the same bits.
#pragma once

#include "sq_internal.h"

namespace sq {
namespace {

// erf(z) for z >= 0 by Abramowitz and Stegun 7.1.28 (absolute error below
// 3e-7): 1 - 1 / (1 + a1 z + a2 z^2 + ... + a6 z^6)^16.  The polynomial by
// Horner's rule from a6 down (a multiply and an add per coefficient), the
// 16th power by four squarings; where it overflows to infinity, 1 / p is 0.
// The coefficients are the table's decimal values rounded to double and then
// to float.
__device__ __forceinline__ float erf_as716(float z) {
  constexpr float a1 = static_cast<float>(0.0705230784), a2 = static_cast<float>(0.0422820123),
                  a3 = static_cast<float>(0.0092705272), a4 = static_cast<float>(0.0001520143),
                  a5 = static_cast<float>(0.0002765672), a6 = static_cast<float>(0.0000430638);
  float p = a6;
  p = p * z + a5;
  p = p * z + a4;
  p = p * z + a3;
  p = p * z + a2;
  p = p * z + a1;
  p = p * z + 1.0f;
  p = p * p;
  p = p * p;
  p = p * p;
  p = p * p;
  return 1.0f - 1.0f / p;
}

// GELU(x) = x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)): z = |x| * fp32(1/sqrt 2),
// e = erf(z), s = 1 + e for x >= 0 and 1 - e otherwise, then x * (s * 0.5)
// (the halving is exact and comes first, so x * s cannot overflow).
__device__ __forceinline__ float gelu_f32(float x) {
  constexpr float kInvSqrt2 = static_cast<float>(0.70710678118654752440);
  const float e = erf_as716(__builtin_fabsf(x) * kInvSqrt2);
  const float s = x >= 0.0f ? 1.0f + e : 1.0f - e;
  return x * (s * 0.5f);
}

// The next linear's STATIC quantizer (Eq. 1, 6 and 8 with the per-step
// threshold): per element x~ = g * D^-1[n], t = (x~ * gamma) * (1 / Delta),
// clamped to [-127, 127] and rounded to even; returns the code's byte.
__device__ __forceinline__ uint32_t static_code8(float g, float dinv, float gain, float inv) {
  float t = ((g * dinv) * gain) * inv;
  t = __builtin_fminf(__builtin_fmaxf(t, -127.0f), 127.0f);
  return __float_as_uint(t + 12582912.0f) & 0xFFu;  // 1.5 * 2^23 + t: the low byte is the rounded code
}

// Four outputs y (fp32, one row, consecutive columns) of the up projection ->
// bf16 -> GELU -> bf16 -> four code bytes of the next layer, packed low
// column first.  The bf16 conversions (two values per instruction) round to
// nearest even.
typedef float f2v_gelu __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v_gelu __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void bf16_round2(float& a, float& b) {
  const uint32_t u = __builtin_bit_cast(uint32_t, __builtin_convertvector((f2v_gelu){a, b}, bf2v_gelu));
  a = __uint_as_float(u << 16);
  b = __uint_as_float(u & 0xFFFF0000u);
}
__device__ __forceinline__ uint32_t gelu_codes4(const float (&y)[4], const float (&dinv)[4], float gain, float inv) {
  float v[4] = {y[0], y[1], y[2], y[3]};
  bf16_round2(v[0], v[1]);
  bf16_round2(v[2], v[3]);
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = gelu_f32(v[j]);
  bf16_round2(v[0], v[1]);
  bf16_round2(v[2], v[3]);
  uint32_t w = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) w |= static_code8(v[j], dinv[j], gain, inv) << (8 * j);
  return w;
}

// The next linear's STATIC 4-bit step and its reciprocal (the first kernel's
// arithmetic: Delta rounded to fp16 before use; an infinite 1 / Delta gives 0).
__device__ __forceinline__ uint32_t static_step4(float clip, float& delta, float& inv) {
  const uint32_t bits = f32_to_f16(clip / 7.0f);
  delta = f16_to_f32(bits);
  inv = 1.0f / delta;
  if (__builtin_isinf(inv)) inv = 0.0f;
  return bits;
}

// Four outputs y (fp32, one row, consecutive columns) of the up projection ->
// bf16 -> GELU -> bf16 -> the next layer's STATIC 4-bit quantizer (t = ((g *
// D^-1) * gain) * (1 / Delta) clamped to [-7, 7], rounded to even).  Returns
// per element the bits of t + 1.5 * 2^23 (the low nibble is the two's
// complement code) and in neg the sign bit of t (the fp8 form's sign: a code
// 0 of negative t is -0).
__device__ __forceinline__ void gelu_codes4_a4(const float (&y)[4], const float (&dinv)[4], float gain, float inv,
                                               uint32_t (&bits)[4], uint32_t (&neg)[4]) {
  float v[4] = {y[0], y[1], y[2], y[3]};
  bf16_round2(v[0], v[1]);
  bf16_round2(v[2], v[3]);
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = gelu_f32(v[j]);
  bf16_round2(v[0], v[1]);
  bf16_round2(v[2], v[3]);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float t = ((v[j] * dinv[j]) * gain) * inv;
    t = __builtin_fminf(__builtin_fmaxf(t, -7.0f), 7.0f);
    bits[j] = __float_as_uint(t + 12582912.0f);
    neg[j] = __float_as_uint(t) >> 31;
  }
}

// The fp8 form of a code (e4m3 byte of code * 2^-9: sign and magnitude) and
// the code's value, from gelu_codes4_a4's bits and sign: |code| = rne(|t|) =
// |rne(t)|, the rounding being symmetric.
__device__ __forceinline__ uint32_t fp8_code_byte(uint32_t bits, uint32_t neg, int& code) {
  const int c = static_cast<int>(static_cast<int8_t>(static_cast<uint8_t>(bits & 0xFFu)));
  const uint32_t mag = static_cast<uint32_t>(c < 0 ? -c : c);
  code = c;
  return mag | (neg << 7);
}

}  // namespace
}  // namespace sq
