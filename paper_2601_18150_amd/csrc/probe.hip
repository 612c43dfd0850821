// Measurement probes, not part of the FP8 linear-layer path, built into their
// own library (libfp8rl_probe.so):
//  * a loop of independent v_mfma_f32_16x16x128_f8f6f4 instructions fed from
//    registers, which gives the FP8 MFMA rate this GPU sustains (at the clock
//    its power limit allows for pure MFMA work) as a measured reference next to
//    the spec peak;
//  * the fp32 fast path of the SiLU * up evaluation (silu_math.hpp, the same
//    code the fused down-projection kernel runs) element by element, so that
//    its error can be measured against the exact value for every input;
//  * single v_mfma_f32_16x16x128_f8f6f4 instructions on operands given by the
//    host, so that the instruction's summation of its 128 products (and of the
//    accumulator input) can be compared with the exact sums;
//  * the global-to-LDS DMA the GEMMs feed their operand tiles with, alone (no
//    compute), streaming regions of chosen sizes, so that the rate one CU can
//    pull from L1-, L2- or HBM-resident data is measured directly;
//  * the GEMM K step's inner loop without its memory traffic: per step each of
//    8 waves reads its wave tile's fragments from LDS and issues its MFMAs,
//    optionally with the per-K-block scale FMAs and a workgroup barrier, so
//    that what each costs the MFMA pipes is measured on its own.
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

// Workgroup b streams region b of src ([b * region, (b + 1) * region)) into LDS
// with 16-byte-per-lane DMA instructions (1 KiB per wave instruction, as the
// GEMM K loop issues them), or (kToLds false) into registers with the same
// 16-byte loads: each wave issues kInflight instructions, waits for
// them, and moves on, `iters` rounds, walking the region's 1 KiB chunks
// cyclically.  The buffer resource spans exactly the region, so an offset past
// it would read zeros rather than leave it (the host also checks the regions
// fit in src).  clk[2b], clk[2b+1]: shader-clock and 100 MHz real-time ticks.
typedef __attribute__((address_space(3))) void lds_void_t;
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
template <int kInflight, bool kToLds>
__global__ __launch_bounds__(1024) void dma_rate_kernel(const uint8_t* __restrict__ src, uint32_t region, int iters,
                                                        float* __restrict__ sink, unsigned long long* __restrict__ clk) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[64 * 1024];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int waves = blockDim.x >> 6;
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(src + (int64_t)blockIdx.x * region), (short)0, (int)region, 0x00020000);
  const uint32_t chunks = region >> 10;
  uint32_t c = (uint32_t)(wave * kInflight) % chunks;          // every offset below stays < region
  const uint32_t step = (uint32_t)(waves * kInflight) % chunks;
  uint32_t x = 0;
  const unsigned long long s0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < kInflight; ++i) {
      const uint32_t ci = (c + i) % chunks;
      if constexpr (kToLds) {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)(lds + ((wave * kInflight + i) & 63) * 1024), 16,
                                                 (ci << 10) + lane * 16, 0, 0, 0);
      } else {
        const v4u32 v = __builtin_amdgcn_raw_buffer_load_b128(r, (ci << 10) + lane * 16, 0, 0);
        x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
      }
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);    // vmcnt(0)
    c = (c + step) % chunks;
  }
  const unsigned long long s1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  __syncthreads();
  sink[(int64_t)blockIdx.x * blockDim.x + t] = (float)lds[(t * 16) & (64 * 1024 - 1)] + (float)x;
  if (t == 0) {
    clk[2 * blockIdx.x] = s1 - s0;
    clk[2 * blockIdx.x + 1] = r1 - r0;
  }
}

// Inner loop of one K step, 8 waves (two per SIMD), wave tile (16 TN) n x
// (16 TM) m as the GEMMs lay it out: per step TM + TN fragments of 32 bytes per
// lane read from LDS (two ds_read_b128 each) and TN x TM MFMAs.  kFma: MFMA
// into a zero accumulator, then acc += p * scale (four FMAs per MFMA, as the
// fp32-scale GEMM); else the MFMA accumulates in place.  kBarrier: s_barrier
// after every step, as the GEMM's LDS ring needs.  The fragments are fixed
// data; nothing is written to LDS after the start.
typedef int v8i32p __attribute__((ext_vector_type(8)));
typedef float v4f32p __attribute__((ext_vector_type(4)));
template <int TN, int TM, bool kFma, bool kBarrier>
__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, float* __restrict__ out,
                                                        unsigned long long* __restrict__ clk) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[96 * 1024];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  for (int i = t; i < 96 * 1024 / 16; i += blockDim.x)
    reinterpret_cast<v4u32*>(lds)[i] = (v4u32){0x38383838u + (unsigned)(i & 7), 0x3A3A3A3Au, 0x34343434u, 0x36363636u};
  __syncthreads();
  // wave w: n half (w & 1) of the W fragments, m quarter (w >> 1) of the A fragments
  const int wbase = (wave & 1) * TN * 2048;                       // < 2 * 8 * 2048 = 32 KiB
  const int abase = 32 * 1024 + (wave >> 1) * TM * 2048;          // < 32 KiB + 4 * 4 * 2048 = 64 KiB
  const int lo = lane * 16;
  v4f32p acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = (v4f32p){0.f, 0.f, 0.f, 0.f};
  float sc[TM];
#pragma unroll
  for (int j = 0; j < TM; ++j) sc[j] = 1.0f + (float)j * 0.25f;
  auto frag = [&](int off) {
    const v4u32 u0 = *reinterpret_cast<const v4u32*>(lds + off + lo);
    const v4u32 u1 = *reinterpret_cast<const v4u32*>(lds + off + 1024 + lo);
    return (v8i32p){(int)u0[0], (int)u0[1], (int)u0[2], (int)u0[3], (int)u1[0], (int)u1[1], (int)u1[2], (int)u1[3]};
  };
  const unsigned long long s0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
    v8i32p bf[TM];
#pragma unroll
    for (int tm = 0; tm < TM; ++tm) bf[tm] = frag(abase + tm * 2048);
#pragma unroll
    for (int tn = 0; tn < TN; ++tn) {
      const v8i32p af = frag(wbase + tn * 2048);
      if constexpr (kFma) {
        v4f32p p[TM];
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          p[tm] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf[tm], (v4f32p){0.f, 0.f, 0.f, 0.f}, 0, 0, 0,
                                                                   0, 0, 0);
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[tn][tm][r] = __builtin_fmaf(p[tm][r], sc[tm], acc[tn][tm][r]);
      } else {
#pragma unroll
        for (int tm = 0; tm < TM; ++tm)
          acc[tn][tm] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf[tm], acc[tn][tm], 0, 0, 0, 0, 0, 0);
      }
    }
    if constexpr (kBarrier) __syncthreads();
#pragma unroll
    for (int j = 0; j < TM; ++j) sc[j] = sc[j] * 0.999f + 1e-7f;     // a new scale per step
  }
  const unsigned long long s1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  float f = 0.f;
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) f += acc[i][j][0] + acc[i][j][3];
  out[(int64_t)blockIdx.x * blockDim.x + t] = f;
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

// One wave per case: d = c + A . B^T for one 16x16x128 E4M3 tile, computed by
// exactly one v_mfma_f32_16x16x128_f8f6f4.  a, b: [cases][16][128] codes (row i
// of A, row j of B); c, d: [cases][16][16] fp32, element [i][j].  Lane L feeds
// row L % 16 of each operand, K bytes 32 (L / 16) .. +31, and holds the results
// [4 (L / 16) + r][L % 16], r = 0..3.
__global__ __launch_bounds__(64) void mfma_tile_kernel(const uint8_t* __restrict__ a, const uint8_t* __restrict__ b,
                                                       const float* __restrict__ c, float* __restrict__ d) {
  const int64_t cs = blockIdx.x;
  const int lane = threadIdx.x;
  const int row = lane & 15, g = lane >> 4;
  const uint4* pa = reinterpret_cast<const uint4*>(a + cs * 2048 + row * 128 + g * 32);
  const uint4* pb = reinterpret_cast<const uint4*>(b + cs * 2048 + row * 128 + g * 32);
  const uint4 a0 = pa[0], a1 = pa[1], b0 = pb[0], b1 = pb[1];
  v8i32 fa, fb;
  fa[0] = (int)a0.x; fa[1] = (int)a0.y; fa[2] = (int)a0.z; fa[3] = (int)a0.w;
  fa[4] = (int)a1.x; fa[5] = (int)a1.y; fa[6] = (int)a1.z; fa[7] = (int)a1.w;
  fb[0] = (int)b0.x; fb[1] = (int)b0.y; fb[2] = (int)b0.z; fb[3] = (int)b0.w;
  fb[4] = (int)b1.x; fb[5] = (int)b1.y; fb[6] = (int)b1.z; fb[7] = (int)b1.w;
  v4f32 acc;
  for (int r = 0; r < 4; ++r) acc[r] = c[cs * 256 + (4 * g + r) * 16 + row];
  acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(fa, fb, acc, 0, 0, 0, 0, 0, 0);
  for (int r = 0; r < 4; ++r) d[cs * 256 + (4 * g + r) * 16 + row] = acc[r];
}

}  // namespace

// a, b: cases x 2048 codes; c, d: cases x 256 floats (device pointers, 16-byte
// aligned).  0 on success, 1 for a bad argument, 4 for a launch error.
extern "C" int fp8rl_probe_mfma_tile(const uint8_t* a, const uint8_t* b, const float* c, float* d, long long cases,
                                     void* stream) {
  if (cases < 0 || cases >= (1ll << 31) || (cases > 0 && (!a || !b || !c || !d))) return 1;
  if (cases == 0) return 0;
  hipLaunchKernelGGL(mfma_tile_kernel, dim3((unsigned)cases), dim3(64), 0, static_cast<hipStream_t>(stream), a, b, c,
                     d);
  return hipGetLastError() == hipSuccess ? 0 : 4;
}

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

// DMA-rate probe.  src: src_bytes of device memory; region: bytes streamed by
// each workgroup, a multiple of 1024 below 2^31, blocks * region <= src_bytes;
// waves: 1..16 per workgroup; inflight: 1, 2, 4 or 8 instructions per wave
// between waits; to_lds: 1 for the DMA into LDS, 0 for loads into registers; sink: blocks * waves * 64 floats; clk: 2 * blocks.  Moves
// iters * blocks * waves * inflight KiB.  0 on success, 1 on a bad argument,
// 4 on a launch failure.
extern "C" int fp8rl_probe_dma_rate(const uint8_t* src, long long src_bytes, long long region, int blocks, int waves,
                                    int inflight, int to_lds, int iters, float* sink, unsigned long long* clk,
                                    void* stream) {
  if (!src || !sink || !clk || blocks < 1 || waves < 1 || waves > 16 || iters < 1) return 1;
  if (region < 1024 || region % 1024 || region >= (1ll << 31) || src_bytes < 0 || (long long)blocks > src_bytes / region)
    return 1;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)blocks), block((unsigned)(64 * waves));
  const uint32_t reg = (uint32_t)region;
#define FP8RL_DMA(N)                                                                                            \
  if (inflight == N) {                                                                                          \
    if (to_lds)                                                                                                 \
      hipLaunchKernelGGL((dma_rate_kernel<N, true>), grid, block, 0, st, src, reg, iters, sink, clk);           \
    else                                                                                                        \
      hipLaunchKernelGGL((dma_rate_kernel<N, false>), grid, block, 0, st, src, reg, iters, sink, clk);          \
    return hipGetLastError() == hipSuccess ? 0 : 4;                                                             \
  }
  FP8RL_DMA(1)
  FP8RL_DMA(2)
  FP8RL_DMA(4)
  FP8RL_DMA(8)
#undef FP8RL_DMA
  return 1;
}

// K-step inner-loop probe: blocks workgroups of 512 threads (8 waves); tile 0 =
// wave tile 128n x 64m (the prefill GEMM's), 1 = 64n x 64m (the decode and MoE
// tiles'); fma, barrier: 0 or 1 (see mfma_loop_kernel).  out: blocks * 512
// floats; clk: 2 * blocks.  Each wave issues iters * TN * TM MFMAs.  0 on
// success, 1 on a bad argument, 4 on a launch failure.
extern "C" int fp8rl_probe_mfma_loop(int tile, int fma, int barrier, int blocks, int iters, float* out,
                                     unsigned long long* clk, void* stream) {
  if (!out || !clk || blocks < 1 || iters < 1 || tile < 0 || tile > 1 || fma < 0 || fma > 1 || barrier < 0 ||
      barrier > 1)
    return 1;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)blocks), block(512);
#define FP8RL_LOOP(TN, TM, F, B) \
  hipLaunchKernelGGL((mfma_loop_kernel<TN, TM, F, B>), grid, block, 0, st, iters, out, clk)
  const int sel = tile * 4 + fma * 2 + barrier;
  switch (sel) {
    case 0: FP8RL_LOOP(8, 4, false, false); break;
    case 1: FP8RL_LOOP(8, 4, false, true); break;
    case 2: FP8RL_LOOP(8, 4, true, false); break;
    case 3: FP8RL_LOOP(8, 4, true, true); break;
    case 4: FP8RL_LOOP(4, 4, false, false); break;
    case 5: FP8RL_LOOP(4, 4, false, true); break;
    case 6: FP8RL_LOOP(4, 4, true, false); break;
    default: FP8RL_LOOP(4, 4, true, true); break;
  }
#undef FP8RL_LOOP
  return hipGetLastError() == hipSuccess ? 0 : 4;
}
