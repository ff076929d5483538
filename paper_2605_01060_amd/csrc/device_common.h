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
typedef short i16x4 __attribute__((ext_vector_type(4)));
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

// LDS rows of CPR 16-byte chunks (CPR = 8: 64 bf16, CPR = 4: 32 bf16); the
// logical chunk c of row r is stored at position c ^ f(r), with
//   CPR = 8: f(r) = (r & 7) ^ ((r >> 3) & 1),
//   CPR = 4: f(r) = ((r >> 1) & 3) ^ ((r >> 3) & 1).
// Reading one logical chunk from 32 consecutive rows, any 8 aligned rows
// fall on 8 different 16-byte slots of a 128-byte window and any 16 aligned
// rows on 16 different slots of a 256-byte window: free of bank conflicts
// whether the LDS serves a 16-byte read 8 lanes at a time over 32 banks or
// 16 lanes at a time over 64 banks.  Returns the slot index (16-byte units).
template <int CPR>
__device__ __forceinline__ int swz(int row, int chunk) {
  static_assert(CPR == 8 || CPR == 4, "LDS rows of 64 or 32 bf16");
  if (CPR == 8) return row * 8 + (chunk ^ (row & 7) ^ ((row >> 3) & 1));
  return row * 4 + (chunk ^ ((row >> 1) & 3) ^ ((row >> 3) & 1));
}

// A wave copy instruction (below) fills 64 consecutive slots: lane l's slot
// is row l / CPR (+ 64/CPR per further copy), stored position l % CPR.  The
// logical chunk that belongs there, the same for every further copy when
// the copies of a wave start at rows that are multiples of 16:
//   CPR = 8: (l & 7) ^ (l >> 3) ^ (copy & 1)    (rows 8 apart per copy),
//   CPR = 4: (l & 3) ^ ((l >> 3) & 3) ^ (l >> 5).
template <int CPR>
__device__ __forceinline__ int copy_chunk(int lane, int copy) {
  if (CPR == 8) return (lane & 7) ^ (lane >> 3) ^ (copy & 1);
  return (lane & 3) ^ ((lane >> 3) & 3) ^ (lane >> 5);
}

// Direct global -> LDS copy of 16 bytes per lane (gfx950 global_load_lds):
// the wave's 64 lanes land contiguously at LDS byte address `lds` (wave
// uniform, passed in M0).  Inline assembly, so the waits are placed by the
// kernel itself; the compiler does not track these loads.
__device__ __forceinline__ void copy_to_lds16(const void* g, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, off"
      :
      : "v"(g), "s"(lds)
      : "memory", "m0");
}

// The same copy from sbase + voff: sbase wave-uniform (scalar registers),
// voff a 32-bit byte offset per lane.
__device__ __forceinline__ void copy_to_lds16_at(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      :
      : "v"(voff), "s"(sbase), "s"(lds)
      : "memory", "m0");
}

// The same copy from a wave-uniform base: lane l fetches the 16 bytes at
// base + 16 l (a 32-bit lane offset added to a scalar base, computed inside
// the statement so that no per-lane address has to stay live around it).
// `lds` must be wave-uniform.
__device__ __forceinline__ void copy_lanes_to_lds16(const void* base, uint32_t lds) {
  uint32_t voff;
  asm volatile(
      "v_mbcnt_lo_u32_b32 %0, -1, 0\n\t"
      "v_mbcnt_hi_u32_b32 %0, -1, %0\n\t"
      "v_lshlrev_b32 %0, 4, %0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1"
      : "=&v"(voff)
      : "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory", "m0");
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

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
// Stegun, Handbook of Mathematical Functions, formula 7.1.28: for x >= 0,
// erf(x) = 1 - (1 + a1 x + ... + a6 x^6)^-16, absolute error <= 3e-7
// (about 7e-7 for GELU evaluated in fp32), far below the bf16 rounding of
// the outputs it feeds; it needs one reciprocal and no exponential.  With
// q = 0.5 |z| (1 + c1 |z| + ... + c6 |z|^6)^-16 (c_i = a_i / sqrt(2)^i),
// both signs of z give GELU(z) = max(z, 0) - q, so no sign fix-up is needed.
// The factor 0.5 is folded into the polynomial: scaled by k = 2^(1/16), its
// -16th power carries the 1/2.
__device__ __forceinline__ float gelu_erf(float z) {
  constexpr float K = 1.0442737824274138f;  // 2^(1/16)
  constexpr float C1 = 0.0705230784f * 0.70710678118654752f * K;
  constexpr float C2 = 0.0422820123f * 0.5f * K;
  constexpr float C3 = 0.0092705272f * 0.35355339059327376f * K;
  constexpr float C4 = 0.0001520143f * 0.25f * K;
  constexpr float C5 = 0.0002765672f * 0.17677669529663688f * K;
  constexpr float C6 = 0.0000430638f * 0.125f * K;
  const float az = fabsf(z);
  float p = fmaf(C6, az, C5);
  p = fmaf(p, az, C4);
  p = fmaf(p, az, C3);
  p = fmaf(p, az, C2);
  p = fmaf(p, az, C1);
  p = fmaf(p, az, K);
  const float r = __builtin_amdgcn_rcpf(p);
  const float r2 = r * r;
  const float r4 = r2 * r2;
  const float r8 = r4 * r4;
  return fmaf(-az, r8 * r8, fmaxf(z, 0.0f));
}

}  // namespace surge
