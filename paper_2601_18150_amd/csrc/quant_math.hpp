// Scale and quotient arithmetic of the blockwise E4M3 quantiser, shared by the
// weight and activation kernels.  Everything here is __host__ __device__ so the
// same sequence can also be compiled for the CPU and checked there against
// plain IEEE division.
//
// Quantisation rule (paper section 2.1.1, Eq. (1): divide by the block scale,
// round to FP8; the scale comes from the block's largest magnitude):
//   scale = fl32(amax / 448)            (1.0 for an all-zero block)
//   code  = E4M3_rne_sat(fl32(x / scale)), sign of x kept
// (the rounding to E4M3 itself is done by the kernels).
//
// The per-element quotient avoids a full IEEE division per element: with the
// block reciprocal r = fl32(1/scale) (itself correctly rounded), the sequence
//   q0 = fl32(a * r);  e = fma(-q0, scale, a) (exact);  q = fl32(q0 + e * r)
// is Markstein's correction step, which returns the correctly rounded quotient
// a / scale when r is correctly rounded and no intermediate is subnormal or
// infinite.  Blocks with amax < 2^-82 (where the residual could fall into the
// fp32 subnormal range, and for the smallest blocks 1/scale would overflow) are
// handled by scaling a and scale by 2^64 first, which leaves the real quotient
// unchanged.  Quotients below 2^-11 may differ in the last bit (the residual of
// an fp32-subnormal x is not exact), but every value below 2^-10 rounds to an
// E4M3 zero, so the codes are unaffected.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#include <hip/hip_runtime.h>
#define FP8RL_HD __host__ __device__ __forceinline__
#else
#include <math.h>
#include <string.h>
#define FP8RL_HD static inline
#endif

namespace fp8rl {
namespace qmath {

constexpr float kE4M3Max = 448.0f;
// amax below 2^-82 takes the pre-scaled path (bf16 magnitude bits < 45 << 7).
// Above it, scale >= 2^-91, so every x whose quotient reaches 2^-11 is at least
// 2^-102 and the residual x - q0 * scale of the correction step is an exact
// (normal) fp32 number.
constexpr uint32_t kSmallAmaxBits16 = 45u << 7;
constexpr float kPrescale = 18446744073709551616.0f;   // 2^64

FP8RL_HD float as_float(uint32_t u) {
#if defined(__HIPCC__)
  return __uint_as_float(u);
#else
  float f; memcpy(&f, &u, 4); return f;
#endif
}

FP8RL_HD uint32_t as_uint(float f) {
#if defined(__HIPCC__)
  return __float_as_uint(f);
#else
  uint32_t u; memcpy(&u, &f, 4); return u;
#endif
}

FP8RL_HD float fma_f32(float a, float b, float c) {
#if defined(__HIPCC__)
  return __builtin_fmaf(a, b, c);
#else
  return fmaf(a, b, c);
#endif
}

// Per-block constants derived from the block's largest bf16 magnitude
// (amax16 = the 15 magnitude bits of the largest |x|).
struct BlockScale {
  float scale;     // stored scale: fl32(amax / 448), or 1.0 for amax == 0
  float s;         // divisor used in the element map (scale, or scale * 2^64)
  float r;         // fl32(1 / s)
  bool prescaled;  // elements must be multiplied by 2^64 before the map
};

FP8RL_HD BlockScale block_scale(uint32_t amax16) {
  BlockScale b;
  const float amax = as_float(amax16 << 16);
  // IEEE fp32 division, correctly rounded (HIP's default for '/').
  b.scale = (amax16 == 0u) ? 1.0f : amax / kE4M3Max;
  b.prescaled = amax16 < kSmallAmaxBits16 && amax16 != 0u;
  b.s = b.prescaled ? b.scale * kPrescale : b.scale;   // exact: power-of-two product
  b.r = 1.0f / b.s;
  return b;
}

// Power-of-two (UE8M0) variant (section 2.4.3): scale = 2^k with k the smallest
// integer such that amax <= 448 * 2^k, clamped below at -127 (the smallest UE8M0
// value); 1.0 for an all-zero block.  With amax = 1.m * 2^e (a normal bf16),
// amax / 448 = (1.m / 1.75) * 2^(e - 8), so k = e - 8, plus one when the 7-bit
// mantissa m exceeds 0x60 (1.m > 1.75).  Subnormal amax gives k < -127 before
// the clamp.  The element map is then the exact product x * 2^-k: s and r below
// are 2^k and 2^-k, prescaled is false.
FP8RL_HD int pow2_exponent(uint32_t amax16) {
  if (amax16 == 0u) return 0;
  const int ef = (int)(amax16 >> 7);
  if (ef == 0) return -127;
  const int k = ef - 127 - 8 + ((amax16 & 0x7Fu) > 0x60u ? 1 : 0);
  return k < -127 ? -127 : k;
}

FP8RL_HD BlockScale block_scale_pow2(uint32_t amax16) {
  const int k = pow2_exponent(amax16);                  // -127 .. 120
  BlockScale b;
  b.scale = as_float(k >= -126 ? (uint32_t)(k + 127) << 23 : 0x00400000u);   // 2^k (2^-127 is subnormal)
  b.s = b.scale;
  b.r = as_float((uint32_t)(127 - k) << 23);            // 2^-k, a normal number for every k here
  b.prescaled = false;
  return b;
}

// Correctly rounded fl32(a / s) for finite a (either sign), given r = fl32(1/s);
// an exact -0 result may come back as +0 (the kernels restore the sign).
FP8RL_HD float quotient(float a, float s, float r) {
  const float q0 = a * r;
  const float e = fma_f32(-q0, s, a);
  return fma_f32(e, r, q0);
}

}  // namespace qmath
}  // namespace fp8rl
