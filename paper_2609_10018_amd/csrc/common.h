// Shared device-side helpers of the gfx950 kernels: bf16 conversion, vector
// types, wave reductions.  Host code does not include this file.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace elasto {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// Round to nearest, ties to even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 b = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, b);
}

// Two values rounded to bf16 like f32_to_bf16 and packed, lo in bits 0-15
// (one packed conversion instead of two conversions and a merge).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Exact GELU, z * Phi(z), with the device library's erff.
__device__ __forceinline__ float gelu_erf(float z) {
  return 0.5f * z * (1.0f + erff(z * 0.70710678118654752f));
}

// GELU for the bf16 path, without transcendental instructions:
// GELU(z) = z * Phi(z) with Phi(z) - 1/2 ~= s q(s^2), s = clamp(z / kGeluZ, -1, 1),
// q a polynomial of degree 9 in s^2 (near-minimax fit; gelu_fit.py makes the
// coefficients).
// |error| <= 1e-4 absolute for |z| <= 12 and <= 1e-4 relative where
// |GELU(z)| > 0.1: below the bf16 rounding of the result (relative 2^-9).
constexpr float kGeluZ = 4.5f;
constexpr float kGeluC[10] = {1.795161009e+00f, -6.052584648e+00f, 1.825310516e+01f,
                              -4.269977188e+01f, 7.698018646e+01f, -1.044052124e+02f,
                              1.017403946e+02f, -6.639614868e+01f, 2.573282433e+01f,
                              -4.447952271e+00f};
__device__ __forceinline__ float gelu_poly(float z) {
  const float s = __builtin_amdgcn_fmed3f(z * (1.0f / kGeluZ), -1.0f, 1.0f);
  const float s2 = s * s;
  float q = kGeluC[9];
#pragma unroll
  for (int k = 8; k >= 0; --k) q = fmaf(q, s2, kGeluC[k]);
  return z * fmaf(s, q, 0.5f);
}

// d/dz of gelu_poly: with s = z/Z inside (-Z, Z),
// (z (0.5 + s q(s^2)))' = 0.5 + s q + s (q + 2 s^2 q'(s^2)); outside, s is
// constant and only 0.5 + s q remains.
__device__ __forceinline__ float gelu_poly_grad(float z) {
  const float s = __builtin_amdgcn_fmed3f(z * (1.0f / kGeluZ), -1.0f, 1.0f);
  const float s2 = s * s;
  float q = kGeluC[9], dq = 9.0f * kGeluC[9];
#pragma unroll
  for (int k = 8; k >= 0; --k) q = fmaf(q, s2, kGeluC[k]);
#pragma unroll
  for (int k = 8; k >= 1; --k) dq = fmaf(dq, s2, (float)k * kGeluC[k]);
  const float inner = fabsf(z) < kGeluZ ? s * fmaf(2.0f * s2, dq, q) : 0.0f;
  return fmaf(s, q, 0.5f) + inner;
}

}  // namespace elasto
