// Device-side types and helpers for the gfx950 kernels.
//
// Activations and weights are stored as bf16 bit patterns (uint16_t) in HBM;
// all arithmetic is fp32 (MFMA accumulates in fp32).  Conversions to bf16
// use the hardware's round-to-nearest-even (v_cvt_pk_bf16_f32).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace surge {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
// Native 16-byte vector (HIP's uint4 is a union-based struct, which keeps
// LLVM from turning register arrays of it into registers).
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

// Two floats -> packed bf16 pair (low half = a).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2 v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

// Eight bf16 in a uint4 -> eight floats.
__device__ __forceinline__ void unpack8(const uint4& u, float* f) {
  f[0] = __uint_as_float(u.x << 16);
  f[1] = __uint_as_float(u.x & 0xffff0000u);
  f[2] = __uint_as_float(u.y << 16);
  f[3] = __uint_as_float(u.y & 0xffff0000u);
  f[4] = __uint_as_float(u.z << 16);
  f[5] = __uint_as_float(u.z & 0xffff0000u);
  f[6] = __uint_as_float(u.w << 16);
  f[7] = __uint_as_float(u.w & 0xffff0000u);
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  uint4 u;
  u.x = pack_bf16x2(f[0], f[1]);
  u.y = pack_bf16x2(f[2], f[3]);
  u.z = pack_bf16x2(f[4], f[5]);
  u.w = pack_bf16x2(f[6], f[7]);
  return u;
}

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// GELU, z Phi(z) = 0.5 z (1 + erf(z / sqrt 2)), with erf by Abramowitz &
// Stegun, Handbook of Mathematical Functions, formula 7.1.26: for x >= 0,
// erf(x) = 1 - t (a1 + a2 t + ... + a5 t^4) exp(-x^2), t = 1 / (1 + p x),
// absolute error <= 1.5e-7 (about 6e-7 evaluated in fp32 with the hardware
// reciprocal and exp2), far below the bf16 rounding of the outputs it
// feeds.  With q = 0.5 |z| t (a1 + ... + a5 t^4) exp(-z^2 / 2), both signs
// of z give GELU(z) = max(z, 0) - q (for z < 0, 1 + erf = 1 - (1 - 2q/|z|)),
// so the 0.5 and 1/sqrt 2 fold into the constants and no sign fix-up is
// needed.
__device__ __forceinline__ float gelu_erf(float z) {
  constexpr float P = 0.3275911f * 0.70710678118654752f;
  constexpr float A1 = 0.5f * 0.254829592f, A2 = 0.5f * -0.284496736f, A3 = 0.5f * 1.421413741f,
                  A4 = 0.5f * -1.453152027f, A5 = 0.5f * 1.061405429f;
  const float az = fabsf(z);
  const float t = __builtin_amdgcn_rcpf(fmaf(P, az, 1.0f));
  float poly = fmaf(A5, t, A4);
  poly = fmaf(poly, t, A3);
  poly = fmaf(poly, t, A2);
  poly = fmaf(poly, t, A1);
  const float e = __builtin_amdgcn_exp2f(z * z * -0.72134752044448170f);  // exp(-z^2 / 2)
  return fmaf(-(az * poly) * t, e, fmaxf(z, 0.0f));
}

}  // namespace surge
