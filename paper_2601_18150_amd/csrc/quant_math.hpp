// Element arithmetic of the blockwise E4M3 quantiser, shared by the weight and
// activation kernels.  Everything here is __host__ __device__ so the exact same
// instruction sequence can also be compiled for the CPU and swept exhaustively.
//
// Quantisation rule (paper section 2.1.1, Eq. (1): divide by the block scale,
// round to FP8; the scale comes from the block's largest magnitude):
//   scale = fl32(amax / 448)            (1.0 for an all-zero block)
//   code  = E4M3_rne_sat(fl32(x / scale)), sign of x kept.
//
// The per-element quotient avoids a full IEEE division per element: with the
// block reciprocal r = fl32(1/scale) (itself correctly rounded), the sequence
//   q0 = fl32(a * r);  e = fma(-q0, scale, a) (exact);  q = fl32(q0 + e * r)
// is Markstein's correction step, which returns the correctly rounded quotient
// a / scale when r is correctly rounded and no intermediate is subnormal or
// infinite.  Blocks with amax < 2^-100 (where 1/scale would overflow) are
// handled by scaling a and scale by 2^64 first, which leaves the real quotient
// unchanged.  Quotients that do fall in the fp32 subnormal range are below the
// smallest E4M3 magnitude (2^-9) by far and encode as +-0 either way.
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
// amax below 2^-100 takes the pre-scaled path (bf16 magnitude bits < 27 << 7)
constexpr uint32_t kSmallAmaxBits16 = 27u << 7;
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

// Correctly rounded fl32(a / s) for a >= 0 finite, given r = fl32(1/s).
FP8RL_HD float quotient(float a, float s, float r) {
  const float q0 = a * r;
  const float e = fma_f32(-q0, s, a);
  return fma_f32(e, r, q0);
}

// 7-bit E4M3 magnitude code of q >= 0 (q <= 448 * (1 + 2^-22) here):
// round to nearest even on the E4M3 grid, saturating at 0x7E.
FP8RL_HD uint32_t e4m3_mag(float q) {
  const uint32_t b = as_uint(q);
  // normal range [2^-6, 448]: keep 3 mantissa bits with RNE on the fp32 bits,
  // then rebias the exponent from 127 to 7 (subtract 120 << 3 from the code).
  const uint32_t lsb = (b >> 20) & 1u;
  const uint32_t normal = (b + (0x7FFFFu - (120u << 23)) + lsb) >> 20;
  // subnormal range [0, 2^-6): adding 2^14 (ulp 2^-9) rounds q to a multiple of
  // 2^-9 with RNE; the low bits of the sum are then that multiple.
  const uint32_t sub = as_uint(q + 16384.0f) - 0x46800000u;
  uint32_t code = (b < 0x3C800000u) ? sub : normal;
  return code < 0x7Eu ? code : 0x7Eu;
}

// Full element map for one bf16 input (bit pattern h) of a block.
template <bool kPrescaled>
FP8RL_HD uint32_t quant_elem(uint32_t h, const BlockScale& bs) {
  float a = as_float((h & 0x7FFFu) << 16);
  if (kPrescaled) a *= kPrescale;
  const uint32_t mag = e4m3_mag(quotient(a, bs.s, bs.r));
  return mag | ((h >> 8) & 0x80u);
}

}  // namespace qmath
}  // namespace fp8rl
