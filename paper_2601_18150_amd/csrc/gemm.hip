// Dense and grouped (MoE) blockwise-scaled FP8 GEMM kernels and launchers.
// The tile computation lives in gemm_core.hpp; this file maps workgroups to
// tiles.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "gemm_core.hpp"
#include "launch.hpp"

namespace fp8rl {
namespace {

// Tile configurations (BN x BM, waves, LDS ring depth), measured on MI355X:
// - M and N >= 2048: 256x256, 8 waves, 2 slots (one workgroup per CU).
// - other M > 256, and the grouped GEMM with K > 1024: 128x128, 4 waves, 2
//   slots: two workgroups per CU walking their tiles as one pipeline.  Deeper
//   rings with one tile per workgroup were slower (MoE gate_up 270 vs 205 us).
// - the grouped GEMM with K <= 1024: 256n x 128m, 8 waves, 2 slots, one
//   workgroup per CU walking its tiles as one pipeline: half as many tiles, so
//   short K loops pay fewer tile ends (Qwen3-30B-A3B down, K = 768: 104-106 vs
//   118-120 us; gate_up, K = 2048, is 2-4% slower with it).
// - 128 < M <= 256 (decode batches): 64x64 tiles, 4 waves, 3 slots, one tile per
//   workgroup, when they number at most 512 (Qwen3-8B at M = 256: qkv 21.6 vs
//   24.0 us, o_proj 17.0 vs 21.3 us for split-K 128x128 tiles); otherwise one
//   256-token tile, 128x256, 8 waves, 3 slots (gate_up: 44 vs 48 us for 128x128,
//   59 us for 64x64).
// - split-K ranges: 128x128, 3 slots (decode linears 123 vs 129 us per layer).
using CfgLarge = GemmCfg<256, 256, 2, 4, 2>;   // 512 threads, wave tile 128(n) x 64(m), 130 KiB LDS
using CfgSmall = GemmCfg<128, 128, 2, 2, 2>;   // 256 threads, wave tile 64 x 64, 65 KiB LDS
using CfgDecode = GemmCfg<128, 256, 2, 4, 3>;  // 512 threads, wave tile 64 x 64, 147 KiB LDS
using CfgDecodeNarrow = GemmCfg<64, 64, 2, 2, 3>;   // 256 threads, wave tile 32 x 32, 49 KiB LDS
using CfgSplitK = GemmCfg<128, 128, 2, 2, 3>;  // one tile per workgroup, 2 K steps in flight, 98 KiB LDS
using CfgGroupedShortK = GemmCfg<256, 128, 4, 2, 2>;   // 512 threads, wave tile 64 x 64, 97 KiB LDS
using CfgGrouped = CfgSmall;

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

__device__ __forceinline__ int band_tile(int t, int tiles_m, int tiles_n, int group_m = kGroupM) {
  const int band = t / (group_m * tiles_n);
  const int first_m = band * group_m;
  const int gm = min(tiles_m - first_m, group_m);
  const int in_band = t - band * group_m * tiles_n;
  const int tile_m = first_m + in_band % gm;
  const int tile_n = in_band / gm;
  return tile_n * tiles_m + tile_m;
}

__device__ __forceinline__ int xcd_grouped_tile(int id, int tiles_m, int tiles_n) {
  return band_tile(xcd_contiguous(id, tiles_m * tiles_n), tiles_m, tiles_n);
}

// The cross-tile pipeline (next tile's first load during this tile's last
// step) for the 128x128 and 256x128 tiles with a 2-slot ring; the 256x256 tile
// has no registers to spare for the next tile's load plan and runs one tile per
// workgroup.
template <class C>
constexpr bool kCrossTiles = C::BN * C::BM <= 256 * 128 && C::STAGES == 2;

// Job providers for gemm_tiles (see gemm_core.hpp): wave-uniform, no LDS
// writes, no synchronisation.

// Dense: a persistent grid; workgroup b runs tiles v = b, b + gridDim.x, ... of
// the renumbered order above (with gridDim.x a multiple of 8 every tile a
// workgroup runs is in its own XCD's range).
template <class C>
struct DenseJobs {
  int v, stride, tiles_m, tiles_n, M;
  __device__ bool next(TileJob& j) {
    if (v >= tiles_m * tiles_n) return false;
    const int tile = xcd_grouped_tile(v, tiles_m, tiles_n);
    v += stride;
    const int tile_m = tile % tiles_m;
    j.row_lo = tile_m * C::BM;
    j.m_valid = min(C::BM, M - j.row_lo);
    j.n0 = (tile / tiles_m) * C::BN;
    j.qw_off = 0;
    j.sw_off = 0;
    return true;
  }
};

// A single given tile.
struct OneJob {
  TileJob job;
  bool done;
  __device__ bool next(TileJob& j) {
    if (done) return false;
    j = job;
    done = true;
    return true;
  }
};

// kMx: power-of-two scales through the MX-scaled MFMA (gemm_core.hpp).
template <class C, bool kMx>
__global__ __launch_bounds__(C::kThreads) void gemm_w8a8_block_kernel(
    const uint8_t* __restrict__ qa, int64_t lda, const float* __restrict__ sa, int64_t ld_sa,
    const uint8_t* __restrict__ qw, int64_t ldw, const float* __restrict__ sw,
    uint16_t* __restrict__ y, int64_t ldy, int64_t M, int64_t N, int KB, int tiles_m, int tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes];
  DenseJobs<C> jobs{(int)blockIdx.x, (int)gridDim.x, tiles_m, tiles_n, (int)M};
  gemm_tiles<C, false, kCrossTiles<C>, DenseJobs<C>, kMx>(qa, lda, sa, ld_sa, qw, ldw, sw, KB, y, ldy, nullptr,
                                                          (int)N, KB, jobs, lds);
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
  const int kb0 = (int)(((int64_t)split * KB) / splits);
  const int kb1 = (int)(((int64_t)(split + 1) * KB) / splits);
  OneJob jobs;
  jobs.done = false;
  jobs.job.row_lo = tile_m * C::BM;
  jobs.job.m_valid = (int)min((int64_t)C::BM, M - jobs.job.row_lo);
  jobs.job.n0 = (tile / tiles_m) * C::BN;
  jobs.job.qw_off = (int64_t)kb0 * 128;
  jobs.job.sw_off = kb0;
  gemm_tiles<C, true, false>(qa + (int64_t)kb0 * 128, lda, sa + (int64_t)kb0 * ld_sa, ld_sa, qw, ldw, sw, KB, nullptr, 0,
                      part + (int64_t)split * M * N, (int)N, kb1 - kb0, jobs, lds);
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

// Grouped GEMM: m tiles are numbered over all experts in order (expert e owns
// ceil(rows_e / BM) consecutive m tiles, empty experts none).  Each workgroup
// first builds, in LDS, the first m tile and the first row of every expert
// from the device offsets (one prefix scan by wave 0), then runs tiles
// v = b, b + gridDim.x, ... of the (m tile, n tile) grid, renumbered so that
// each XCD walks a contiguous range in bands of kGroupMoe m tiles (m fastest
// inside a band): an XCD's concurrent tiles share their activation rows across
// the n tiles and, within an expert, its weight slab, both from its L2.
constexpr int kMaxExperts = 1024;          // table capacity (LDS: 8 KiB)
constexpr int kGroupMoe = 2;               // m tiles per band (measured: 2-4 best, 6-10% over m-fastest)

template <class C>
struct GroupedJobs {
  int v, stride, real_m, tiles_n, G;
  const int* tstart;                       // LDS [G+1]: first m tile of expert e
  const int* rstart;                       // LDS [G+1]: first row of expert e
  int64_t N, K;
  __device__ bool next(TileJob& j) {
    if (v >= real_m * tiles_n) return false;
    const int bt = band_tile(xcd_contiguous(v, real_m * tiles_n), real_m, tiles_n, kGroupMoe);
    v += stride;
    const int target = bt % real_m;
    const int tile_n = bt / real_m;
    // e = (number of experts whose first m tile is <= target) - 1: the last
    // such expert owns the tile (empty experts share their start with the next)
    const int lane = threadIdx.x & 63;
    int cnt = 0;
    for (int e0 = 0; e0 <= G; e0 += 64) {
      const int e = e0 + lane;
      const bool le = e <= G && tstart[e] <= target;
      const unsigned long long mask = __ballot(le);
      cnt += __popcll(mask);
      if (~mask) break;
    }
    // (the table entries are wave-uniform: keep them in scalar registers)
    const int e = __builtin_amdgcn_readfirstlane(cnt - 1);
    const int mt = target - __builtin_amdgcn_readfirstlane(tstart[e]);
    j.row_lo = __builtin_amdgcn_readfirstlane(rstart[e]) + mt * C::BM;
    j.m_valid = min(C::BM, __builtin_amdgcn_readfirstlane(rstart[e + 1]) - j.row_lo);
    j.n0 = tile_n * C::BN;
    j.qw_off = (int64_t)e * N * K;
    j.sw_off = (int64_t)e * (N / 128) * (K / 128);
    return true;
  }
};

// kGather: output row r takes its activation row from source row gidx[r] of qa
// ([src_rows][lda]) and sa ([K/128][ld_sa]); otherwise qa is [rows][K].
template <class C, bool kMx, bool kGather>
__global__ __launch_bounds__(C::kThreads) void grouped_gemm_w8a8_block_kernel(
    const uint8_t* __restrict__ qa, const float* __restrict__ sa, int64_t ld_sa,
    const uint8_t* __restrict__ qw, const float* __restrict__ sw,
    const int32_t* __restrict__ offsets, int G, uint16_t* __restrict__ y, int64_t N, int64_t K, int tiles_n,
    const int32_t* __restrict__ gidx, int src_rows, int64_t lda) {
  // one LDS object: the ring, then the two expert tables
  __shared__ __attribute__((aligned(16))) uint8_t lds[C::kLdsBytes + 2 * 4 * (kMaxExperts + 1)];
  int* tstart = reinterpret_cast<int*>(lds + C::kLdsBytes);
  int* rstart = tstart + (kMaxExperts + 1);
  const int t = threadIdx.x;
  if (t < 64) {
    // wave 0: exclusive prefix sum of the experts' m-tile counts, 64 at a time
    int base = 0;
    for (int e0 = 0; e0 <= G; e0 += 64) {
      const int e = e0 + t;
      int cnt = 0, r0 = 0;
      if (e <= G) r0 = offsets[e];
      if (e < G) cnt = (offsets[e + 1] - r0 + C::BM - 1) / C::BM;
      int incl = cnt;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int u = __shfl_up(incl, d, 64);
        if (t >= d) incl += u;
      }
      if (e <= G) {
        tstart[e] = base + incl - cnt;
        rstart[e] = r0;
      }
      base += __shfl(incl, 63, 64);
    }
  }
  __syncthreads();
  GroupedJobs<C> jobs{(int)blockIdx.x, (int)gridDim.x, __builtin_amdgcn_readfirstlane(tstart[G]), tiles_n, G,
                      tstart, rstart, N, K};
  const int KB = (int)(K / 128);
  gemm_tiles<C, false, kCrossTiles<C>, GroupedJobs<C>, kMx, kGather>(qa, kGather ? lda : K, sa, ld_sa, qw, K, sw, KB,
                                                                     y, N, nullptr, (int)N, KB, jobs, lds, gidx,
                                                                     src_rows);
}

// Workgroups that stay resident on one CU for a configuration (LDS-limited).
template <class C, int kExtraLds = 0>
constexpr int per_cu() { return (160 * 1024) / (C::kLdsBytes + kExtraLds); }

constexpr int kCus = 256;     // MI355X; grids of kCus * per_cu() are multiples of 8 (one per XCD)

template <class C, bool kMx>
hipError_t launch_dense(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa, const uint8_t* qw,
                        int64_t ldw, const float* sw, uint16_t* y, int64_t ldy, int64_t m, int64_t n,
                        int64_t k, hipStream_t stream) {
  const int tiles_m = (int)((m + C::BM - 1) / C::BM);
  const int tiles_n = (int)((n + C::BN - 1) / C::BN);
  const int64_t total = (int64_t)tiles_m * tiles_n;
  // persistent grid with the cross-tile pipeline, else one workgroup per tile
  // (a persistent grid without it measured no faster)
  const int64_t slots = kCrossTiles<C> ? (int64_t)kCus * per_cu<C>() : total;
  hipLaunchKernelGGL((gemm_w8a8_block_kernel<C, kMx>), dim3((unsigned)(total < slots ? total : slots)),
                     dim3(C::kThreads), 0, stream, qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n,
                     (int)(k / 128), tiles_m, tiles_n);
  return hipGetLastError();
}

template <class C, bool kMx, bool kGather = false>
hipError_t launch_grouped(const uint8_t* qa, const float* sa, int64_t ld_sa, const uint8_t* qw,
                          const float* sw, const int32_t* offsets, int64_t g, int64_t rows, uint16_t* y,
                          int64_t n, int64_t k, hipStream_t stream, const int32_t* gidx = nullptr,
                          int64_t src_rows = 0, int64_t lda = 0) {
  const int64_t max_tiles_m = rows / C::BM + g;        // upper bound on the real m tiles
  const int64_t tiles_n = (n + C::BN - 1) / C::BN;
  const int64_t total = max_tiles_m * tiles_n;
  // persistent grid with the cross-tile pipeline, else one workgroup per tile
  const int64_t slots = kCrossTiles<C> ? (int64_t)kCus * per_cu<C, 2 * 4 * (kMaxExperts + 1)>() : total;
  hipLaunchKernelGGL((grouped_gemm_w8a8_block_kernel<C, kMx, kGather>),
                     dim3((unsigned)(total < slots ? total : slots)), dim3(C::kThreads), 0, stream, qa, sa, ld_sa, qw,
                     sw, offsets, (int)g, y, n, k, (int)tiles_n, gidx, (int)src_rows, lda);
  return hipGetLastError();
}

}  // namespace

// Decode batches (128 < M <= 256) whose 64x64 tiles number at most 512 (two per CU).
static bool decode_narrow_tiles(int64_t m, int64_t n) { return ((m + 63) / 64) * (n / 64) <= 512; }

hipError_t launch_gemm_w8a8_block(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                  const uint8_t* qw, int64_t ldw, const float* sw, uint16_t* y, int64_t ldy,
                                  int64_t m, int64_t n, int64_t k, hipStream_t stream, bool pow2_scales) {
  const bool large = m >= 2048 && n >= 2048;
  const bool decode = !large && m > 128 && m <= 256;
  const bool narrow = decode && decode_narrow_tiles(m, n);
  if (pow2_scales)
    return large    ? launch_dense<CfgLarge, true>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream)
           : narrow ? launch_dense<CfgDecodeNarrow, true>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream)
           : decode ? launch_dense<CfgDecode, true>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream)
                    : launch_dense<CfgSmall, true>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream);
  return large    ? launch_dense<CfgLarge, false>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream)
         : narrow ? launch_dense<CfgDecodeNarrow, false>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream)
         : decode ? launch_dense<CfgDecode, false>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream)
                  : launch_dense<CfgSmall, false>(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, stream);
}

int splitk_factor(int64_t m, int64_t n, int64_t k) {
  // Split K only when the 128x128 tiles cover less than half of MI355X's 256
  // CUs, into the largest power of two of ranges that keeps tiles x splits
  // within 256, each range at least 4 K blocks long.  (Measured on the decode
  // linears, M = 256: more ranges lose to the fp32 partial-sum traffic, which
  // grows with the split.)
  constexpr int64_t kCus = 256;
  if (m <= 0 || n <= 0 || k <= 0 || (m >= 2048 && n >= 2048)) return 1;
  // decode batches run unsplit on 64x64 tiles when K is short enough for one
  // workgroup's K loop (Qwen3-8B qkv, o_proj: K = 4096; down, K = 12288, splits)
  if (m > 128 && m <= 256 && k <= 4096 && decode_narrow_tiles(m, n)) return 1;
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
  using C = CfgSplitK;
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

// Split-K partial sums for callers that cannot allocate: a file-scope device
// array (each GPU the library runs on holds its own copy until the process
// ends).  In host code `scratch` only names the symbol; its device address on
// the current device comes from hipGetSymbolAddress, fetched once per device.
static __device__ __align__(256) float scratch[kSplitKScratchBytes / 4];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<float*> scratch_ptr[kMaxDevices];
}  // namespace

hipError_t splitk_scratch(float** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  float* p = scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    void* q = nullptr;
    e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    p = static_cast<float*>(q);
    scratch_ptr[dev].store(p, std::memory_order_release);   // racing first calls store the same address
  }
  *out = p;
  return hipSuccess;
}

hipError_t launch_grouped_gemm_w8a8_block(const uint8_t* qa, const float* sa, int64_t ld_sa,
                                          const uint8_t* qw, const float* sw, const int32_t* group_offsets,
                                          int64_t num_groups, int64_t total_rows, uint16_t* y, int64_t n,
                                          int64_t k, hipStream_t stream, bool pow2_scales) {
  const bool short_k = k <= 1024;
  if (pow2_scales)
    return short_k ? launch_grouped<CfgGroupedShortK, true>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups,
                                                             total_rows, y, n, k, stream)
                   : launch_grouped<CfgGrouped, true>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups, total_rows,
                                                      y, n, k, stream);
  return short_k ? launch_grouped<CfgGroupedShortK, false>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups,
                                                            total_rows, y, n, k, stream)
                 : launch_grouped<CfgGrouped, false>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups, total_rows, y,
                                                     n, k, stream);
}

hipError_t launch_grouped_gemm_w8a8_block_gathered(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                                   int64_t src_rows, const int32_t* row_index, const uint8_t* qw,
                                                   const float* sw, const int32_t* group_offsets, int64_t num_groups,
                                                   int64_t total_rows, uint16_t* y, int64_t n, int64_t k,
                                                   hipStream_t stream) {
  if (k <= 1024)
    return launch_grouped<CfgGroupedShortK, false, true>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups,
                                                         total_rows, y, n, k, stream, row_index, src_rows, lda);
  return launch_grouped<CfgGrouped, false, true>(qa, sa, ld_sa, qw, sw, group_offsets, num_groups, total_rows, y,
                                                 n, k, stream, row_index, src_rows, lda);
}

}  // namespace fp8rl
