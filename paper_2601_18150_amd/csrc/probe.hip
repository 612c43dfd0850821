// Measurement probe, not part of the FP8 linear-layer path: a loop of
// independent v_mfma_f32_16x16x128_f8f6f4 instructions fed from registers,
// which gives the FP8 MFMA rate this GPU sustains (at the clock its power limit
// allows for pure MFMA work) as a measured reference next to the spec peak.
// Built into its own library (libfp8rl_probe.so) for bench.py.
#include <hip/hip_runtime.h>
#include <stdint.h>

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

}  // namespace

// Enqueue the probe: `blocks` workgroups of 256 threads; out holds blocks*256
// floats, clk 2*blocks counters (device pointers).  Returns a hipError_t value.
extern "C" int fp8rl_probe_mfma_rate(float* out, unsigned long long* clk, int blocks, int iters, void* stream) {
  if (!out || !clk || blocks <= 0 || iters <= 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(mfma_rate_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, out, iters, clk);
  return (int)hipGetLastError();
}
