// Token-level truncated importance-sampling weights and mismatch-KL sums
// (paper section 2.1.3, Eq. (2)-(3); the mismatch KL of section 2.2):
//   d = logp_train - logp_rollout (exact in fp64), w = e^d,
//   w_TIS = min(w, C) rounded to fp32 (0 outside the response mask),
//   stats = (sum of -d, sum of expm1(d) - d, valid tokens, tokens with w > C).
// HBM-bound: 9 bytes read and 4 written per token.  The sums are fp64 and
// deterministic: each thread walks a fixed token set, the wave and workgroup
// reductions run in a fixed order, and a second kernel adds the per-workgroup
// partials (in the caller's workspace) in order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "launch.hpp"

namespace fp8rl {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double shfl_xor_f64(double v, int m) {
  const long long b = __double_as_longlong(v);
  const int lo = __shfl_xor((int)(b & 0xFFFFFFFFll), m, 64);
  const int hi = __shfl_xor((int)(b >> 32), m, 64);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor_f64(v, m);
  return v;                                     // every lane holds the same, identically ordered sum
}

// Sum of the four statistics over the workgroup; thread 0 gets the result.
__device__ __forceinline__ void block_sum4(double (&s)[4], double* red) {
  const int t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < 4; ++j) s[j] = wave_sum_f64(s[j]);
  if ((t & 63) == 0)
#pragma unroll
    for (int j = 0; j < 4; ++j) red[(t >> 6) * 4 + j] = s[j];
  __syncthreads();
  if (t == 0)
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] = (red[j] + red[4 + j]) + (red[8 + j] + red[12 + j]);
}

// One token's contribution.
__device__ __forceinline__ float tis_token(float lt, float lr, bool valid, double c, double (&s)[4]) {
  const double d = (double)lt - (double)lr;
  const double w = exp(d);
  if (!valid) return 0.0f;
  s[0] -= d;
  s[1] += expm1(d) - d;
  s[2] += 1.0;
  s[3] += w > c ? 1.0 : 0.0;
  return (float)fmin(w, c);
}

// Thread j of the grid handles the 4-token chunks j, j + stride, ... (16-byte loads
// of both log-probability arrays, 4-byte loads of the mask, two chunks in flight per
// step); the n % 4 tail tokens go to the first threads of workgroup 0.
__global__ __launch_bounds__(kThreads) void tis_partial_kernel(const float* __restrict__ lt,
                                                              const float* __restrict__ lr,
                                                              const uint8_t* __restrict__ mask, int64_t n,
                                                              double c, float* __restrict__ w_tis,
                                                              double* __restrict__ partial) {
  __shared__ double red[16];
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  const int64_t chunks = n / 4;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  const float4* lt4 = reinterpret_cast<const float4*>(lt);
  const float4* lr4 = reinterpret_cast<const float4*>(lr);
  const uint32_t* m4 = reinterpret_cast<const uint32_t*>(mask);
  float4* w4 = reinterpret_cast<float4*>(w_tis);
  int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  for (; i + stride < chunks; i += 2 * stride) {
    const float4 a0 = lt4[i], b0 = lr4[i], a1 = lt4[i + stride], b1 = lr4[i + stride];
    const uint32_t v0 = mask ? m4[i] : 0x01010101u, v1 = mask ? m4[i + stride] : 0x01010101u;
    float4 o;
    o.x = tis_token(a0.x, b0.x, (v0 & 0xFFu) != 0, c, s);
    o.y = tis_token(a0.y, b0.y, (v0 & 0xFF00u) != 0, c, s);
    o.z = tis_token(a0.z, b0.z, (v0 & 0xFF0000u) != 0, c, s);
    o.w = tis_token(a0.w, b0.w, (v0 & 0xFF000000u) != 0, c, s);
    w4[i] = o;
    o.x = tis_token(a1.x, b1.x, (v1 & 0xFFu) != 0, c, s);
    o.y = tis_token(a1.y, b1.y, (v1 & 0xFF00u) != 0, c, s);
    o.z = tis_token(a1.z, b1.z, (v1 & 0xFF0000u) != 0, c, s);
    o.w = tis_token(a1.w, b1.w, (v1 & 0xFF000000u) != 0, c, s);
    w4[i + stride] = o;
  }
  if (i < chunks) {
    const float4 a0 = lt4[i], b0 = lr4[i];
    const uint32_t v0 = mask ? m4[i] : 0x01010101u;
    float4 o;
    o.x = tis_token(a0.x, b0.x, (v0 & 0xFFu) != 0, c, s);
    o.y = tis_token(a0.y, b0.y, (v0 & 0xFF00u) != 0, c, s);
    o.z = tis_token(a0.z, b0.z, (v0 & 0xFF0000u) != 0, c, s);
    o.w = tis_token(a0.w, b0.w, (v0 & 0xFF000000u) != 0, c, s);
    w4[i] = o;
  }
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const int64_t t = chunks * 4 + threadIdx.x;
    w_tis[t] = tis_token(lt[t], lr[t], mask == nullptr || mask[t] != 0, c, s);
  }
  block_sum4(s, red);
  if (threadIdx.x == 0)
#pragma unroll
    for (int j = 0; j < 4; ++j) partial[(int64_t)blockIdx.x * 4 + j] = s[j];
}

// One workgroup: lane-strided fixed-order sums of the partials, then the tree.
__global__ __launch_bounds__(kThreads) void tis_final_kernel(const double* __restrict__ partial, int blocks,
                                                            double* __restrict__ stats) {
  __shared__ double red[16];
  double s[4] = {0.0, 0.0, 0.0, 0.0};
  for (int b = threadIdx.x; b < blocks; b += kThreads)
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] += partial[(int64_t)b * 4 + j];
  block_sum4(s, red);
  if (threadIdx.x == 0)
#pragma unroll
    for (int j = 0; j < 4; ++j) stats[j] = s[j];
}

}  // namespace

int tis_blocks(int64_t n) {
  constexpr int64_t kMaxBlocks = 2048;      // 8 workgroups per CU
  const int64_t b = (n / 4 + 2 * kThreads - 1) / (2 * kThreads);   // two 4-token chunks per thread and step
  return (int)(b < 1 ? 1 : (b > kMaxBlocks ? kMaxBlocks : b));
}

hipError_t launch_tis_weights_kl(const float* logp_train, const float* logp_rollout, const uint8_t* mask, int64_t n,
                                 float clip_c, float* w_tis, double* stats, double* partial, hipStream_t stream) {
  const int blocks = tis_blocks(n);
  hipLaunchKernelGGL(tis_partial_kernel, dim3(blocks), dim3(kThreads), 0, stream, logp_train, logp_rollout, mask, n,
                     (double)clip_c, w_tis, partial);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(tis_final_kernel, dim3(1), dim3(kThreads), 0, stream, partial, blocks, stats);
  return hipGetLastError();
}

}  // namespace fp8rl
