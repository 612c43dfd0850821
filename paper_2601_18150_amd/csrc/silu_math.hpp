// h = bf16(SiLU(g) * u) for bf16 g, u, correctly rounded from the exact value
// (the gated MLP's down-projection input; paper section 2.1.1 quantises that
// layer like every other linear).
//
// Fast path, fp32:
//   e = 2^(-g log2 e) = E (1 + c) with E = v_exp_f32(g * H) (H: -log2 e to 16
//       significant bits, so the product with an 8-bit bf16 g is exact) and
//       c = g * L ln 2 (L = -log2 e - H, |L| < 2^-17), so 1 + e = fma(E, c, 1 + E);
//   q = g * rcp(1 + e)  (v_rcp_f32);   r = q * u.
// The relative errors (in units of 2^-24: E 2, the dropped c^2 / 2 term at most
// 1.6 for |g| <= 88 beyond which 1 + e overflows, 1 + E and the fma 1 each, rcp
// 2, the two products 1 each) stay below 10, so r lies within 10 ulps of the
// exact value whenever q is a normal number well above the subnormal range and
// r is finite; an exhaustive check over every gate bit pattern and up
// significand measures the actual maximum.  r then rounds to the same bf16 as
// the exact value unless its 16 discarded bits lie within kTieGuard ulps of the
// half-way point 0x8000.  The rounding itself is v_cvt_pk_bf16_f32 (nearest
// even).
//
// Exact path (those few elements, and every element with a tiny, zero,
// infinite or NaN quotient): for g != 0 the exact value is never a bf16 tie,
// but in two limits it lies closer to an exactly representable product than
// fp64 can resolve, so the product is rounded with the side of the tie given
// by the sign of the deviation:
//   |g| <= 2^-20: SiLU(g) u = (g u / 2)(1 + tanh(g / 2)), within 2^-21 of the
//                 16-bit product g u / 2: a tie goes away from zero for g > 0,
//                 toward zero for g < 0;
//   g >= 16:      SiLU(g) u = g u (1 - 1 / (1 + e^g)), within 2^-23 of g u: a
//                 tie goes toward zero.
// Between them the fp64 evaluation is never within 2^-48 of a bf16 rounding
// boundary (checked over every gate bit pattern and up significand), far
// beyond its few-ulp error, so its nearest-even rounding is the exact one.
// NaN gives 0x7FC0.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp8rl {
namespace silu {

constexpr float kNegLog2eHi = -0x1.7154p+0f;            // -log2(e) to 16 significant bits (-1.44268798828125)
constexpr float kNegLog2eLoLn2 = -0x1.480fb6p-18f;     // (-log2(e) - kNegLog2eHi) * ln 2, to fp32
constexpr uint32_t kTieGuard = 12;                      // fp32 ulps around the bf16 half-way point
constexpr float kMinQuotient = 0x1p-100f;              // fast path only for |q| at or above

// The fast path's fp32 result r (and the quotient q it came from).
__device__ __forceinline__ float fast(float g, float u, float& q) {
  const float big_e = __builtin_amdgcn_exp2f(g * kNegLog2eHi);    // exact argument
  const float c = g * kNegLog2eLoLn2;
  const float d = __builtin_fmaf(big_e, c, 1.0f + big_e);          // 1 + e
  q = g * __builtin_amdgcn_rcpf(d);
  return q * u;
}

// Whether r certainly rounds like the exact value.
__device__ __forceinline__ bool fast_ok(float q, float r) {
  const uint32_t low = __float_as_uint(r) & 0xFFFFu;
  return (low - (0x8000u - kTieGuard) > 2u * kTieGuard) & (fabsf(q) >= kMinQuotient) &
         (fabsf(r) <= 0x1.fffffep127f);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 -> two packed bf16, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// x rounded to bf16 from fp64, once: to nearest; an exact tie away from zero
// (tie > 0), toward zero (tie < 0) or to even (tie == 0).  NaN gives 0x7FC0.
__device__ inline uint32_t f64_to_bf16_tie(double x, int tie) {
  if (x != x) return 0x7FC0u;
  const uint32_t sign = __double_as_longlong(x) < 0 ? 0x8000u : 0u;
  const double a = fabs(x);
  if (a == 0.0) return sign;
  if (a >= 0x1p128) return sign | 0x7F80u;
  int e;
  frexp(a, &e);                                          // a in [2^(e-1), 2^e)
  const int qe = max(e - 1, -126) - 7;                   // bf16 spacing near a is 2^qe
  const double t = ldexp(a, -qe);                        // exact
  const double lo = floor(t);
  const double fr = t - lo;
  double n = fr > 0.5 ? lo + 1.0 : lo;
  if (fr == 0.5) n = tie > 0 ? lo + 1.0 : tie < 0 ? lo : (fmod(lo, 2.0) == 0.0 ? lo : lo + 1.0);
  const double r = ldexp(n, qe);
  if (r >= 0x1p128) return sign | 0x7F80u;
  return sign | (__float_as_uint((float)r) >> 16);      // exact: at most 8 significant bits
}

__device__ __noinline__ uint32_t exact(float g, float u) {
  const double gd = g, ud = u;
  if (fabsf(g) <= 0x1p-20f) return f64_to_bf16_tie(gd * ud * 0.5, g > 0.0f ? 1 : g < 0.0f ? -1 : 0);
  if (g >= 16.0f) return f64_to_bf16_tie(gd * ud, -1);
  return f64_to_bf16_tie(gd / (1.0 + exp(-gd)) * ud, 0);
}

// Eight packed bf16 pairs (one uint4 of gate, one of up) -> eight packed bf16 h.
__device__ __forceinline__ uint4 silu_mul8(const uint4& vg, const uint4& vu) {
  const uint32_t gw[4] = {vg.x, vg.y, vg.z, vg.w};
  const uint32_t uw[4] = {vu.x, vu.y, vu.z, vu.w};
  float gs[8], us[8], rs[8];
  uint32_t slow = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    gs[i] = __uint_as_float(i & 1 ? gw[i >> 1] & 0xFFFF0000u : gw[i >> 1] << 16);
    us[i] = __uint_as_float(i & 1 ? uw[i >> 1] & 0xFFFF0000u : uw[i >> 1] << 16);
    float q;
    rs[i] = fast(gs[i], us[i], q);
    slow |= fast_ok(q, rs[i]) ? 0u : 1u << i;
  }
  uint32_t hw[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) hw[j] = bf16x2_rne(rs[2 * j], rs[2 * j + 1]);
  if (slow) {                                            // replace what the fast path could not certify
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (slow & (1u << i)) {
        const uint32_t b = exact(gs[i], us[i]);
        hw[i >> 1] = i & 1 ? (hw[i >> 1] & 0xFFFFu) | (b << 16) : (hw[i >> 1] & 0xFFFF0000u) | b;
      }
  }
  return make_uint4(hw[0], hw[1], hw[2], hw[3]);
}

}  // namespace silu
}  // namespace fp8rl
