// Device helpers for the gfx950 kernels: bf16 bit handling, cross-lane
// exchange through DPP, bf16 dot/MFMA wrappers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "plan.hpp"

namespace cpattn {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
// Lazy rescaling: the running max only moves when a score exceeds it by more
// than this many powers of two, so unnormalised weights stay below 2^8.
constexpr float kRescaleThreshold = 8.0f;

__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  bf16x2_t v;
  v[0] = (__bf16)a;
  v[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t to_bf16(float a) {
  return __builtin_bit_cast(uint16_t, (__bf16)a);
}

// a.lo*b.lo + a.hi*b.hi + c, bf16 pairs, fp32 accumulate (v_dot2_f32_bf16)
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// DPP lane exchange inside rows of 16 lanes.
//   kXor1: quad_perm [1,0,3,2]     partner lane ^ 1
//   kXor2: quad_perm [2,3,0,1]     partner lane ^ 2
//   kMirror8: row_half_mirror      partner 7 - i inside each group of 8
//   kXor8: row_ror:8               partner lane ^ 8 inside each row of 16
enum DppPartner : int { kXor1 = 0xB1, kXor2 = 0x4E, kMirror8 = 0x141, kXor8 = 0x128 };

template <int Ctrl>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), Ctrl, 0xF, 0xF, false));
}

// Partner whose lane index differs in bit `Bit` (1, 2, 4, 8) and, for Bit 4,
// also in the bits below it (a perfect matching of the 0/1 halves either way).
template <int Bit>
__device__ __forceinline__ float lane_partner(float x) {
  if constexpr (Bit == 1) return dpp<kXor1>(x);
  else if constexpr (Bit == 2) return dpp<kXor2>(x);
  else if constexpr (Bit == 4) return dpp<kMirror8>(x);
  else return dpp<kXor8>(x);
}

__device__ __forceinline__ float shfl_xor_f(float x, int m) { return __shfl_xor(x, m, 64); }

// max over all 64 lanes (every lane receives it)
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dpp<kXor1>(x));
  x = fmaxf(x, dpp<kXor2>(x));
  x = fmaxf(x, dpp<kMirror8>(x));
  x = fmaxf(x, dpp<kXor8>(x));
  x = fmaxf(x, shfl_xor_f(x, 16));
  x = fmaxf(x, shfl_xor_f(x, 32));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
  x += dpp<kXor1>(x);
  x += dpp<kXor2>(x);
  x += dpp<kMirror8>(x);
  x += dpp<kXor8>(x);
  x += shfl_xor_f(x, 16);
  x += shfl_xor_f(x, 32);
  return x;
}

__device__ __forceinline__ f32x16_t mfma32x32x16(uint4 a, uint4 b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint4 ld_global16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 ld_global16_nt(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(v[0], v[1], v[2], v[3]);
}

}  // namespace cpattn
