// Measurement probes, not part of the FP8 linear-layer path, built into their
// own library (libfp8rl_probe.so):
//  * a loop of independent v_mfma_f32_16x16x128_f8f6f4 instructions fed from
//    registers, which gives the FP8 MFMA rate this GPU sustains (at the clock
//    its power limit allows for pure MFMA work) as a measured reference next to
//    the spec peak;
//  * the fp32 fast path of the SiLU * up evaluation (silu_math.hpp, the same
//    code the fused down-projection kernel runs) element by element, so that
//    its error can be measured against the exact value for every input.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "silu_math.hpp"

namespace {

typedef int v8i32 __attribute__((ext_vector_type(8)));
typedef float v4f32 __attribute__((ext_vector_type(4)));

// 256 threads; each wave runs `iters` rounds of four independent MFMAs.
// clk[2b], clk[2b+1]: shader-clock and 100 MHz real-time ticks of workgroup b.
__global__ __launch_bounds__(256) void mfma_rate_kernel(float* __restrict__ out, int iters,
                                                        unsigned long long* __restrict__ clk) {
  const int t = threadIdx.x;
  v8i32 a, b;
  for (int i = 0; i < 8; ++i) {
    a[i] = (int)(0x3C3A3836u + 0x01010101u * (unsigned)((t + i) & 7));
    b[i] = (int)(0x38363C3Au + 0x01010101u * (unsigned)((3 * t + i) & 7));
  }
  v4f32 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = c0, c2 = c0, c3 = c0;
  const unsigned long long s0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c0, 0, 0, 0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c1, 0, 0, 0, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c2, 0, 0, 0, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, c3, 0, 0, 0, 0, 0, 0);
  }
  const unsigned long long s1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float acc = 0.f;
  for (int i = 0; i < 4; ++i) acc += c0[i] + c1[i] + c2[i] + c3[i];
  out[blockIdx.x * 256 + t] = acc;
  if (t == 0) {
    clk[2 * blockIdx.x] = s1 - s0;
    clk[2 * blockIdx.x + 1] = r1 - r0;
  }
}

// One thread per element: r = the fast path's fp32 result, q its quotient.
__global__ __launch_bounds__(256) void silu_fast_kernel(const uint16_t* __restrict__ g, const uint16_t* __restrict__ u,
                                                        float* __restrict__ r, float* __restrict__ q, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float qi;
  r[i] = fp8rl::silu::fast(__uint_as_float((uint32_t)g[i] << 16), __uint_as_float((uint32_t)u[i] << 16), qi);
  q[i] = qi;
}

}  // namespace

// Enqueue the probe: `blocks` workgroups of 256 threads; out holds blocks*256
// floats, clk 2*blocks counters (device pointers).  Returns a hipError_t value.
extern "C" int fp8rl_probe_mfma_rate(float* out, unsigned long long* clk, int blocks, int iters, void* stream) {
  if (!out || !clk || blocks <= 0 || iters <= 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_rate_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, out, iters, clk);
  return (int)hipGetLastError();
}

// g, u: n bf16 bit patterns each; r, q: n floats.  n < 2^31.
extern "C" int fp8rl_probe_silu_fast(const uint16_t* g, const uint16_t* u, float* r, float* q, long long n,
                                     void* stream) {
  if (n < 0 || n >= (1ll << 31)) return 1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(silu_fast_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), g, u, r, q, (int64_t)n);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}
