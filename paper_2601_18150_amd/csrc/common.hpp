// Small device utilities shared by the fp8rl kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp8rl {

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Per-half unsigned max of two packed u16 pairs (v_pk_max_u16).
__device__ __forceinline__ uint32_t max_u16x2(uint32_t a, uint32_t b) {
  u16x2 x = __builtin_bit_cast(u16x2, a);
  u16x2 y = __builtin_bit_cast(u16x2, b);
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(x, y));
}

// Largest bf16 magnitude (15 bits, as u16 pattern) among the 8 bf16 of a uint4.
// Non-negative floats order like their bit patterns, so the integer max is the
// float max of |x|.
__device__ __forceinline__ uint32_t amax16_of(const uint4& v) {
  uint32_t m = max_u16x2(max_u16x2(v.x & 0x7FFF7FFFu, v.y & 0x7FFF7FFFu),
                         max_u16x2(v.z & 0x7FFF7FFFu, v.w & 0x7FFF7FFFu));
  return max(m & 0xFFFFu, m >> 16);
}

// Max over the 16 lanes of each row of a wave (lanes 16r .. 16r+15), returned to
// all 16 lanes, using DPP row operations (no LDS traffic).
__device__ __forceinline__ uint32_t row16_max(uint32_t v) {
  // quad_perm [1,0,3,2] : swap neighbours
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
  // quad_perm [2,3,0,1] : swap pairs
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
  // row_half_mirror : lane i <-> 7-i within each half row
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
  // row_mirror : lane i <-> 15-i within the row
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
  return v;
}

// Max over all 64 lanes of the wave, returned as a wave-uniform value.
__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  v = row16_max(v);
  uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)v, 0);
  uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)v, 16);
  uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)v, 32);
  uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)v, 48);
  return max(max(a, b), max(c, d));
}

// fp32 -> bf16 bits, round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

}  // namespace fp8rl
