// Dense and grouped (MoE) blockwise-scaled FP8 GEMM kernels and launchers.
// The tile computation lives in gemm_core.hpp; this file maps workgroups to
// tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gemm_core.hpp"
#include "launch.hpp"

namespace fp8rl {
namespace {

// Tile configurations.
// (measured on MI355X: 256x128 tiles with 3 slots and 128x128 tiles with 3
// slots were both slower than these two on every configured shape; 128x128
// with 2 slots fits two workgroups per CU, which is what small-M and MoE
// shapes need to fill the 256 CUs)
using CfgLarge = GemmCfg<256, 256, 2, 4, 2>;   // 512 threads, wave tile 128(n) x 64(m), 130 KiB LDS
using CfgSmall = GemmCfg<128, 128, 2, 2, 2>;   // 256 threads, wave tile 64 x 64, 65 KiB LDS

constexpr int kXcds = 8;        // MI355X: workgroup i is dispatched to XCD i % 8
constexpr int kGroupM = 8;      // m tiles per band of the grouped raster order

// Workgroup id -> output tile (encoded tile_n * tiles_m + tile_m).
// 1. Renumber so that the workgroups one XCD receives (ids x, x+8, x+16, ...)
//    walk one contiguous range of tile numbers.
// 2. Walk tile numbers in bands of kGroupM m tiles, m fastest: the tiles an XCD
//    runs at the same time share a few A row blocks and W row blocks, which
//    then stay in that XCD's L2.
// Renumber workgroup ids so that the ids one XCD receives (x, x+8, x+16, ...)
// map to one contiguous range of [0, total).
__device__ __forceinline__ int xcd_contiguous(int id, int total) {
  const int q = total / kXcds, r = total % kXcds;
  const int x = id % kXcds, j = id / kXcds;
  return x * q + min(x, r) + j;
}

__device__ __forceinline__ int band_tile(int t, int tiles_m, int tiles_n) {
  const int band = t / (kGroupM * tiles_n);
  const int first_m = band * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int in_band = t - band * kGroupM * tiles_n;
  const int tile_m = first_m + in_band % gm;
  const int tile_n = in_band / gm;
  return tile_n * tiles_m + tile_m;
}

__device__ __forceinline__ int xcd_grouped_tile(int id, int tiles_m, int tiles_n) {
  return band_tile(xcd_contiguous(id, tiles_m * tiles_n), tiles_m, tiles_n);
}

template <class C>
__global__ __launch_bounds__(C::kThreads) void gemm_w8a8_block_kernel(
    const uint8_t* __restrict__ qa, int64_t lda, const float* __restrict__ sa, int64_t ld_sa,
    const uint8_t* __restrict__ qw, int64_t ldw, const float* __restrict__ sw,
    uint16_t* __restrict__ y, int64_t ldy, int64_t M, int64_t N, int KB, int tiles_m) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes];
  const int tile = xcd_grouped_tile(blockIdx.x, tiles_m, (int)gridDim.x / tiles_m);
  const int tile_m = tile % tiles_m;
  const int tile_n = tile / tiles_m;
  const int64_t row_lo = (int64_t)tile_m * C::BM;
  const int64_t row_hi = min(row_lo + C::BM, M);
  gemm_tile<C>(qa, lda, sa, ld_sa, qw, ldw, sw, KB, y, ldy, nullptr, 0, row_lo, row_hi, (int64_t)tile_n * C::BN,
               N, KB, lds);
}

// Split-K dense GEMM, for shapes whose tiles alone cannot fill the GPU (decode:
// M = 256 gives 64-96 tiles of 128x128 for the narrow layers).  Workgroup v
// runs K range `split` of one tile and writes its fp32 sums to
// part[split][M][N]; splitk_reduce_kernel adds the ranges in order.  Ids are
// renumbered as in the dense kernel, split slowest, so the tiles an XCD runs
// together share their weight rows.
template <class C>
__global__ __launch_bounds__(C::kThreads) void gemm_w8a8_block_splitk_kernel(
    const uint8_t* __restrict__ qa, int64_t lda, const float* __restrict__ sa, int64_t ld_sa,
    const uint8_t* __restrict__ qw, int64_t ldw, const float* __restrict__ sw,
    float* __restrict__ part, int64_t M, int64_t N, int KB, int tiles_m, int tiles_n, int splits) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes];
  const int total = tiles_m * tiles_n;
  const int v = xcd_contiguous(blockIdx.x, total * splits);
  const int split = v / total;
  const int tile = band_tile(v - split * total, tiles_m, tiles_n);
  const int tile_m = tile % tiles_m;
  const int tile_n = tile / tiles_m;
  const int kb0 = (int)(((int64_t)split * KB) / splits);
  const int kb1 = (int)(((int64_t)(split + 1) * KB) / splits);
  const int64_t row_lo = (int64_t)tile_m * C::BM;
  const int64_t row_hi = min(row_lo + C::BM, M);
  gemm_tile<C, true>(qa + (int64_t)kb0 * 128, lda, sa + (int64_t)kb0 * ld_sa, ld_sa, qw + (int64_t)kb0 * 128, ldw,
                     sw + kb0, KB, nullptr, 0, part + (int64_t)split * M * N, N, row_lo, row_hi,
                     (int64_t)tile_n * C::BN, N, kb1 - kb0, lds);
}

// y[m][n] = bf16_rne(part[0][m][n] + part[1][m][n] + ... ), eight n per thread.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, int64_t M, int64_t N,
                                                            int splits, uint16_t* __restrict__ y, int64_t ldy) {
  const int64_t chunks = N / 8;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= M * chunks) return;
  const int64_t m = i / chunks;
  const int64_t c = i - m * chunks;
  const float* p = part + m * N + c * 8;
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  for (int s = 1; s < splits; ++s) {
    const float4 u = *reinterpret_cast<const float4*>(p + (int64_t)s * M * N);
    const float4 w = *reinterpret_cast<const float4*>(p + (int64_t)s * M * N + 4);
    a.x += u.x; a.y += u.y; a.z += u.z; a.w += u.w;
    b.x += w.x; b.y += w.y; b.z += w.z; b.w += w.w;
  }
  uint4 o;
  o.x = f32_to_bf16_rne(a.x) | (f32_to_bf16_rne(a.y) << 16);
  o.y = f32_to_bf16_rne(a.z) | (f32_to_bf16_rne(a.w) << 16);
  o.z = f32_to_bf16_rne(b.x) | (f32_to_bf16_rne(b.y) << 16);
  o.w = f32_to_bf16_rne(b.z) | (f32_to_bf16_rne(b.w) << 16);
  *reinterpret_cast<uint4*>(y + m * ldy + c * 8) = o;
}

// Grouped GEMM: a 1-D grid of max_tiles_m x tiles_n workgroups.  The m tile
// index counts over all experts in order (expert e owns ceil(rows_e / BM)
// consecutive m tiles); the grid is sized for the worst case
// (total_rows / BM + num_groups) and workgroups past the last real tile exit at
// once.  Ids are renumbered so that each XCD walks a contiguous range, m tile
// fastest: the m tiles of one expert that share a weight slab run on the same
// XCD and read it from its L2.
template <class C>
__global__ __launch_bounds__(C::kThreads) void grouped_gemm_w8a8_block_kernel(
    const uint8_t* __restrict__ qa, const float* __restrict__ sa, int64_t ld_sa,
    const uint8_t* __restrict__ qw, const float* __restrict__ sw,
    const int32_t* __restrict__ offsets, int G, uint16_t* __restrict__ y, int64_t N, int64_t K,
    int max_tiles_m) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes];
  __shared__ int found[2];
  const int t = threadIdx.x;
  const int lin = xcd_contiguous(blockIdx.x, (int)gridDim.x);
  const int target = lin % max_tiles_m;
  const int tile_n = lin / max_tiles_m;
  if (t == 0) found[0] = -1;
  __syncthreads();
  if (t < 64) {
    // wave 0 scans the experts 64 at a time: inclusive prefix sum of tile counts
    int base = 0;
    for (int e0 = 0; e0 < G; e0 += 64) {
      const int e = e0 + t;
      int cnt = 0;
      if (e < G) cnt = (offsets[e + 1] - offsets[e] + C::BM - 1) / C::BM;
      int incl = cnt;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int v = __shfl_up(incl, d, 64);
        if (t >= d) incl += v;
      }
      const int excl = incl - cnt;
      if (cnt > 0 && target >= base + excl && target < base + incl) {
        found[0] = e;
        found[1] = target - base - excl;
      }
      base += __shfl(incl, 63, 64);
      if (target < base) break;
    }
  }
  __syncthreads();
  const int e = found[0];
  if (e < 0) return;                       // uniform: past the last real tile
  const int mt = found[1];
  const int KB = (int)(K / 128);
  const int64_t row_lo = (int64_t)offsets[e] + (int64_t)mt * C::BM;
  const int64_t row_hi = min(row_lo + C::BM, (int64_t)offsets[e + 1]);
  gemm_tile<C>(qa, K, sa, ld_sa, qw + (int64_t)e * N * K, K, sw + (int64_t)e * (N / 128) * KB, KB, y, N,
               nullptr, 0, row_lo, row_hi, (int64_t)tile_n * C::BN, N, KB, lds);
}

template <class C>
hipError_t launch_dense(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa, const uint8_t* qw,
                        int64_t ldw, const float* sw, uint16_t* y, int64_t ldy, int64_t m, int64_t n,
                        int64_t k, hipStream_t stream) {
  const int tiles_m = (int)((m + C::BM - 1) / C::BM);
  const int tiles_n = (int)((n + C::BN - 1) / C::BN);
  hipLaunchKernelGGL(gemm_w8a8_block_kernel<C>, dim3((unsigned)(tiles_m * tiles_n)), dim3(C::kThreads), 0,
                     stream, qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, (int)(k / 128), tiles_m);
  return hipGetLastError();
}

template <class C>
hipError_t launch_grouped(const uint8_t* qa, const float* sa, int64_t ld_sa, const uint8_t* qw,
                          const float* sw, const int32_t* offsets, int64_t g, int64_t rows, uint16_t* y,
                          int64_t n, int64_t k, hipStream_t stream) {
  const int64_t max_tiles_m = rows / C::BM + g;
  const int64_t tiles_n = (n + C::BN - 1) / C::BN;
  hipLaunchKernelGGL(grouped_gemm_w8a8_block_kernel<C>, dim3((unsigned)(max_tiles_m * tiles_n)),
                     dim3(C::kThreads), 0, stream, qa, sa, ld_sa, qw, sw, offsets, (int)g, y, n, k,
                     (int)max_tiles_m);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_w8a8_block(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                  const uint8_t* qw, int64_t ldw, const float* sw, uint16_t* y, int64_t ldy,
                                  int64_t m, int64_t n, int64_t k, hipStream_t stream) {
  if (m >= 2048 && n >= 2048)
    return launch_dense<CfgLarge>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream);
  return launch_dense<CfgSmall>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream);
}

int splitk_factor(int64_t m, int64_t n, int64_t k) {
  // Split K only when the 128x128 tiles cover less than half of MI355X's 256
  // CUs, into the largest power of two of ranges that keeps tiles x splits
  // within 256, each range at least 4 K blocks long.  (Measured on the decode
  // linears, M = 256: more ranges lose to the fp32 partial-sum traffic, which
  // grows with the split.)
  constexpr int64_t kCus = 256;
  if (m <= 0 || n <= 0 || k <= 0 || (m >= 2048 && n >= 2048)) return 1;
  const int64_t tiles = ((m + 127) / 128) * (n / 128);
  if (2 * tiles >= kCus) return 1;
  int64_t s = 1;
  while (2 * s * tiles <= kCus) s *= 2;
  const int64_t by_k = (k / 128) / 4;
  if (s > by_k) s = by_k;
  return s > 1 ? (int)s : 1;
}

hipError_t launch_gemm_w8a8_block_splitk(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                         const uint8_t* qw, int64_t ldw, const float* sw, uint16_t* y,
                                         int64_t ldy, int64_t m, int64_t n, int64_t k, float* part, int splits,
                                         hipStream_t stream) {
  using C = CfgSmall;
  const int tiles_m = (int)((m + C::BM - 1) / C::BM);
  const int tiles_n = (int)(n / C::BN);
  hipLaunchKernelGGL(gemm_w8a8_block_splitk_kernel<C>, dim3((unsigned)(tiles_m * tiles_n * splits)),
                     dim3(C::kThreads), 0, stream, qa, lda, sa, ld_sa, qw, ldw, sw, part, m, n, (int)(k / 128),
                     tiles_m, tiles_n, splits);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t chunks = m * (n / 8);
  hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, stream, part, m,
                     n, splits, y, ldy);
  return hipGetLastError();
}

hipError_t launch_grouped_gemm_w8a8_block(const uint8_t* qa, const float* sa, int64_t ld_sa,
                                          const uint8_t* qw, const float* sw, const int32_t* group_offsets,
                                          int64_t num_groups, int64_t total_rows, uint16_t* y, int64_t n,
                                          int64_t k, hipStream_t stream) {
  return launch_grouped<CfgSmall>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups, total_rows, y, n, k,
                                  stream);
}

}  // namespace fp8rl
