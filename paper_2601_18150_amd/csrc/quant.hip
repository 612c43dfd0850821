// Blockwise (128x128) weight and per-token 1x128 activation quantisation to
// OCP E4M3 with fp32 scales (paper section 2.1.1, Eq. (1); section 3.1).
//
// Both kernels are HBM-bound streaming kernels: 16-byte loads of 8 bf16 per
// lane, an integer max over the bf16 magnitudes (packed u16 max), a DPP
// reduction inside each 16-lane row, the per-block scale, the quotient of
// quant_math.hpp and the hardware E4M3 conversion, then 8-byte stores of 8
// codes per lane.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "launch.hpp"
#include "quant_math.hpp"
#include "silu_math.hpp"

#pragma clang fp contract(off)

namespace fp8rl {
namespace {

using qmath::BlockScale;

// 8 bf16 (one uint4) -> 8 E4M3 codes (one uint2), all with the same block scale.
//
// The signed quotient fl32(x / s) is rounded to E4M3 by the hardware conversion
// (v_cvt_pk_fp8_f32: OCP E4M3, round to nearest even).  |quotient| never
// exceeds 448 * (1 + 2^-22) here, which rounds to 448, so the conversion never
// overflows.  The only input whose quotient loses its sign is x = -0 (the
// Markstein step turns -0 into +0); OR-ing the sign bit of every input into its
// code restores 0x80 there and changes nothing elsewhere.  The exhaustive
// (x, amax) sweep of the tests checks this path against the oracle bit for bit.
// How an element's quotient x / scale is formed.
enum QuotientMode : int {
  kMarkstein = 0,      // correctly rounded division (quant_math.hpp)
  kMarksteinPre = 1,   // the same, block pre-scaled by 2^64 (amax < 2^-82)
  kPow2 = 2,           // power-of-two scale: the exact product x * 2^-k
};

template <int kMode>
__device__ __forceinline__ float quotient_of(uint32_t f32_bits, const BlockScale& bs) {
  float x = __uint_as_float(f32_bits);
  if (kMode == kPow2) return x * bs.r;
  if (kMode == kMarksteinPre) x *= qmath::kPrescale;
  return qmath::quotient(x, bs.s, bs.r);
}

template <int kMode>
__device__ __forceinline__ uint32_t quant4(uint32_t w0, uint32_t w1, const BlockScale& bs) {
  const float q0 = quotient_of<kMode>(w0 << 16, bs);
  const float q1 = quotient_of<kMode>(w0 & 0xFFFF0000u, bs);
  const float q2 = quotient_of<kMode>(w1 << 16, bs);
  const float q3 = quotient_of<kMode>(w1 & 0xFFFF0000u, bs);
  int c = __builtin_amdgcn_cvt_pk_fp8_f32(q0, q1, 0, false);   // bytes 0, 1
  c = __builtin_amdgcn_cvt_pk_fp8_f32(q2, q3, c, true);        // bytes 2, 3
  // sign bits of the four bf16 inputs (bit 15 of each half word) -> bit 7 of each byte
  const uint32_t signs = __builtin_amdgcn_perm(w1, w0, 0x07050301u) & 0x80808080u;
  return (uint32_t)c | signs;
}

template <int kMode>
__device__ __forceinline__ uint2 quant8(const uint4& v, const BlockScale& bs) {
  return make_uint2(quant4<kMode>(v.x, v.y, bs), quant4<kMode>(v.z, v.w, bs));
}

// 8 elements with the block's scale: the fp32 scale's two quotient paths, or the
// power-of-two product.
template <bool kPow2Scale>
__device__ __forceinline__ uint2 quant8_block(const uint4& v, const BlockScale& bs) {
  if (kPow2Scale) return quant8<kPow2>(v, bs);
  return bs.prescaled ? quant8<kMarksteinPre>(v, bs) : quant8<kMarkstein>(v, bs);
}

template <bool kPow2Scale>
__device__ __forceinline__ BlockScale scale_of(uint32_t amax16) {
  return kPow2Scale ? qmath::block_scale_pow2(amax16) : qmath::block_scale(amax16);
}

// Streaming (non-temporal) 16-byte load / 8-byte store: the weight re-quantisation
// touches every byte once, so its traffic should not displace cached data
// (measured: the 144-matrix resync pass runs about 10% faster this way).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint4 load_stream16(const uint16_t* p) {
  const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(t[0], t[1], t[2], t[3]);
}

__device__ __forceinline__ void store_stream8(uint8_t* p, const uint2& v) {
  const u32x2_t t = {v.x, v.y};
  __builtin_nontemporal_store(t, reinterpret_cast<u32x2_t*>(p));
}

// ---------------------------------------------------------------------------
// Weight: one 256-thread workgroup per 128x128 block.  Thread t owns the 16-byte
// column chunk (t & 15) of rows (t >> 4) + 16 i, i = 0..7: every load instruction
// of a wave reads four 256-byte row segments.
// ---------------------------------------------------------------------------
template <bool kPow2Scale>
__device__ __forceinline__ void quant_weight_block(const uint16_t* __restrict__ w, int64_t ldw,
                                                   uint8_t* __restrict__ q, int64_t ldq,
                                                   float* __restrict__ scale, int nbk, int blk, uint32_t* red) {
  const int bi = blk / nbk;
  const int bj = blk - bi * nbk;
  const int t = threadIdx.x;
  const int chunk = t & 15;
  const int r0 = t >> 4;

  const uint16_t* src = w + (int64_t)(bi * 128 + r0) * ldw + bj * 128 + chunk * 8;
  uint4 v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = load_stream16(src + (int64_t)(16 * i) * ldw);

  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = max(m, amax16_of(v[i]));
  m = wave_max(m);
  if ((t & 63) == 0) red[t >> 6] = m;
  __syncthreads();
  m = max(max(red[0], red[1]), max(red[2], red[3]));

  const BlockScale bs = scale_of<kPow2Scale>(m);
  if (t == 0) scale[blk] = bs.scale;

  uint8_t* dst = q + (int64_t)(bi * 128 + r0) * ldq + bj * 128 + chunk * 8;
  if (kPow2Scale) {
#pragma unroll
    for (int i = 0; i < 8; ++i) store_stream8(dst + (int64_t)(16 * i) * ldq, quant8<kPow2>(v[i], bs));
  } else if (bs.prescaled) {
#pragma unroll
    for (int i = 0; i < 8; ++i) store_stream8(dst + (int64_t)(16 * i) * ldq, quant8<kMarksteinPre>(v[i], bs));
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) store_stream8(dst + (int64_t)(16 * i) * ldq, quant8<kMarkstein>(v[i], bs));
  }
}

template <bool kPow2Scale>
__global__ __launch_bounds__(256) void quant_weight_block128_kernel(
    const uint16_t* __restrict__ w, int64_t ldw, uint8_t* __restrict__ q, int64_t ldq,
    float* __restrict__ scale, int nbk) {
  __shared__ uint32_t red[4];
  quant_weight_block<kPow2Scale>(w, ldw, q, ldq, scale, nbk, blockIdx.x, red);
}

// Many matrices in one launch: the job table travels in the kernel arguments
// (constant memory, read with scalar loads); workgroup b quantises block
// b - first_block of the last job whose first_block <= b.  One launch keeps the
// memory pipeline full across matrices: a launch per matrix pays its ramp-up and
// drain each time (about 2.5 us, measured on the 144-matrix resync pass).
struct WeightJobArg {
  const uint16_t* w;
  uint8_t* q;
  float* scale;
  int64_t ldw, ldq;
  int nbk;                 // k / 128
  int first_block;         // blocks of the jobs before this one in the launch
};

struct WeightBatchArg {
  WeightJobArg job[kWeightBatchJobs];
  int count;
};

__global__ __launch_bounds__(256) void quant_weight_block128_batched_kernel(const WeightBatchArg b) {
  __shared__ uint32_t red[4];
  const int blk = blockIdx.x;
  // binary search (wave-uniform) for the last job with first_block <= blk
  int lo = 0, hi = b.count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (b.job[mid].first_block <= blk) lo = mid; else hi = mid - 1;
  }
  const WeightJobArg& j = b.job[lo];
  quant_weight_block<false>(j.w, j.ldw, j.q, j.ldq, j.scale, j.nbk, blk - j.first_block, red);
}

// ---------------------------------------------------------------------------
// Activation: 16 lanes per (token, group); a 256-thread workgroup covers 16
// consecutive tokens of one 128-wide group, so its 16 scale stores (scales are
// token-contiguous per group) are one 64-byte run instead of 16 floats ld_scale
// apart.  Plain (cached) loads: the activations usually come straight from the
// previous kernel and still sit in the memory-side cache.
// ---------------------------------------------------------------------------
template <bool kPow2Scale>
__global__ __launch_bounds__(256) void quant_act_token_group128_kernel(
    const uint16_t* __restrict__ a, int64_t lda, uint8_t* __restrict__ q, int64_t ldq,
    float* __restrict__ scale, int64_t ld_scale, uint32_t m, uint32_t ng) {
  const int t = threadIdx.x;
  const int chunk = t & 15;
  const uint32_t rb = blockIdx.x / ng;             // block of 16 tokens
  const uint32_t g = blockIdx.x - rb * ng;         // 128-wide group
  const uint32_t r = rb * 16u + (uint32_t)(t >> 4);
  const bool valid = r < m;
  const int64_t row = valid ? r : m - 1;           // rows past the end re-read the last row (in bounds)

  const uint4 v = *reinterpret_cast<const uint4*>(a + row * lda + g * 128 + chunk * 8);
  const uint32_t mx = row16_max(amax16_of(v));
  const BlockScale bs = scale_of<kPow2Scale>(mx);
  const uint2 c = quant8_block<kPow2Scale>(v, bs);
  if (valid) {
    *reinterpret_cast<uint2*>(q + row * ldq + g * 128 + chunk * 8) = c;
    if (chunk == 0) scale[(int64_t)g * ld_scale + row] = bs.scale;
  }
}

// ---------------------------------------------------------------------------
// Down-projection input of the gated MLP: h = bf16(SiLU(gate) * up) from the
// fused gate_up output [gate | up] (silu_math.hpp: correctly rounded), then the
// same 1x128 group quantisation.  16 lanes per (token, group), each lane 8
// elements of gate and the matching 8 of up.  A workgroup covers 16 * kUnits
// consecutive tokens of one 128-wide group, so its scale stores (scales are
// token-contiguous per group) fill whole cache lines inside one workgroup
// instead of single floats scattered over many.  gate and up are read once:
// streaming loads.  h is written out only when asked for.
// ---------------------------------------------------------------------------
template <int kUnits>
__global__ __launch_bounds__(256) void silu_mul_quant_group128_kernel(
    const uint16_t* __restrict__ gu, int64_t ld_gu, int64_t inter, uint8_t* __restrict__ q, int64_t ldq,
    float* __restrict__ scale, int64_t ld_scale, uint16_t* __restrict__ h, int64_t ldh, uint32_t m, uint32_t ng) {
  const int t = threadIdx.x;
  const int chunk = t & 15;
  const uint32_t rb = blockIdx.x / ng;            // block of 16 * kUnits tokens
  const uint32_t g = blockIdx.x - rb * ng;        // 128-wide group
  uint32_t row[kUnits];
  bool valid[kUnits];
  uint4 vg[kUnits], vu[kUnits];
#pragma unroll
  for (int k = 0; k < kUnits; ++k) {
    const uint32_t r = rb * (16u * kUnits) + 16u * k + (t >> 4);
    valid[k] = r < m;
    row[k] = valid[k] ? r : m - 1;                // rows past the end re-read the last row (in bounds)
    const uint16_t* src = gu + (int64_t)row[k] * ld_gu + g * 128 + chunk * 8;
    vg[k] = load_stream16(src);
    vu[k] = load_stream16(src + inter);
  }
#pragma unroll
  for (int k = 0; k < kUnits; ++k) {
    const uint4 v = silu::silu_mul8(vg[k], vu[k]);
    const uint32_t mx = row16_max(amax16_of(v));
    const BlockScale bs = qmath::block_scale(mx);
    const uint2 c = quant8_block<false>(v, bs);
    if (valid[k]) {
      *reinterpret_cast<uint2*>(q + (int64_t)row[k] * ldq + g * 128 + chunk * 8) = c;
      if (chunk == 0) scale[(int64_t)g * ld_scale + row[k]] = bs.scale;
      if (h) *reinterpret_cast<uint4*>(h + (int64_t)row[k] * ldh + g * 128 + chunk * 8) = v;
    }
  }
}

// ---------------------------------------------------------------------------
// Gather of quantised activation rows: dst row r = src row index[r] (codes and
// the row's group scales).  One thread per 16-byte chunk of a row; the thread
// holding the first chunk of a 128-wide group also copies its scale.  Indices
// outside [0, src_rows) are clamped (a violated precondition, but never an
// out-of-bounds read).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gather_rows_fp8_kernel(
    const uint8_t* __restrict__ q_src, int64_t ldq_src, const float* __restrict__ s_src, int64_t ld_s_src,
    const int32_t* __restrict__ index, int64_t src_rows, int64_t rows, int64_t chunks,
    uint8_t* __restrict__ q_dst, int64_t ldq_dst, float* __restrict__ s_dst, int64_t ld_s_dst) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * chunks) return;
  const int64_t r = i / chunks;
  const int64_t c = i - r * chunks;
  const int64_t src = min(max((int64_t)index[r], (int64_t)0), src_rows - 1);
  *reinterpret_cast<uint4*>(q_dst + r * ldq_dst + c * 16) =
      *reinterpret_cast<const uint4*>(q_src + src * ldq_src + c * 16);
  if ((c & 7) == 0) s_dst[(c >> 3) * ld_s_dst + r] = s_src[(c >> 3) * ld_s_src + src];
}

}  // namespace

hipError_t launch_silu_mul_quant_group128(const uint16_t* gu, int64_t m, int64_t inter, int64_t ld_gu,
                                          uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                          uint16_t* h, int64_t ldh, hipStream_t stream) {
  const uint32_t ng = (uint32_t)(inter / 128);      // m * ng < 2^28 (checked by the caller)
  // tokens per workgroup: 64 while that still gives 2048 workgroups (eight per
  // CU), else 32, else 16.  Measured (us, 8192 x 12288 / 32768 x 768 / 256 x
  // 12288): 64 tokens 93.5 / 29.9 / 9.8, 32 tokens 97.5 / 30.6 / 8.6, 16 tokens
  // 96.9 / 30.6 / 7.9; 128 tokens 103.5 at the first shape.
  const auto blocks_for = [&](int64_t tokens) { return (uint32_t)((m + tokens - 1) / tokens) * ng; };
  constexpr uint32_t kMinBlocks = 2048;
  const uint32_t b4 = blocks_for(64), b2 = blocks_for(32), b1 = blocks_for(16);
  if (b4 >= kMinBlocks)
    hipLaunchKernelGGL(silu_mul_quant_group128_kernel<4>, dim3(b4), dim3(256), 0, stream, gu, ld_gu, inter, q, ldq,
                       scale, ld_scale, h, ldh, (uint32_t)m, ng);
  else if (b2 >= kMinBlocks)
    hipLaunchKernelGGL(silu_mul_quant_group128_kernel<2>, dim3(b2), dim3(256), 0, stream, gu, ld_gu, inter, q, ldq,
                       scale, ld_scale, h, ldh, (uint32_t)m, ng);
  else
    hipLaunchKernelGGL(silu_mul_quant_group128_kernel<1>, dim3(b1), dim3(256), 0, stream, gu, ld_gu, inter, q, ldq,
                       scale, ld_scale, h, ldh, (uint32_t)m, ng);
  return hipGetLastError();
}

hipError_t launch_gather_rows_fp8(const uint8_t* q_src, int64_t ldq_src, const float* s_src, int64_t ld_s_src,
                                  const int32_t* index, int64_t src_rows, int64_t rows, int64_t k,
                                  uint8_t* q_dst, int64_t ldq_dst, float* s_dst, int64_t ld_s_dst,
                                  hipStream_t stream) {
  const int64_t chunks = k / 16;
  const int64_t blocks = (rows * chunks + 255) / 256;
  hipLaunchKernelGGL(gather_rows_fp8_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, q_src, ldq_src, s_src,
                     ld_s_src, index, src_rows, rows, chunks, q_dst, ldq_dst, s_dst, ld_s_dst);
  return hipGetLastError();
}

hipError_t launch_quant_weight_block128(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                                        uint8_t* q, int64_t ldq, float* scale, hipStream_t stream,
                                        bool pow2_scale) {
  const int nbn = (int)(n / 128), nbk = (int)(k / 128);
  const int64_t blocks = (int64_t)nbn * nbk;
  if (pow2_scale)
    hipLaunchKernelGGL(quant_weight_block128_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       w, ldw, q, ldq, scale, nbk);
  else
    hipLaunchKernelGGL(quant_weight_block128_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       w, ldw, q, ldq, scale, nbk);
  return hipGetLastError();
}

hipError_t launch_quant_weight_block128_batched(const WeightJob* jobs, int count, hipStream_t stream) {
  WeightBatchArg b;
  b.count = 0;
  int64_t blocks = 0;
  for (int i = 0; i < count; ++i) {
    const int64_t nb = (jobs[i].n / 128) * (jobs[i].k / 128);
    if (nb == 0) continue;
    WeightJobArg& j = b.job[b.count++];
    j.w = jobs[i].w;
    j.q = jobs[i].q;
    j.scale = jobs[i].scale;
    j.ldw = jobs[i].ldw;
    j.ldq = jobs[i].ldq;
    j.nbk = (int)(jobs[i].k / 128);
    j.first_block = (int)blocks;
    blocks += nb;
  }
  if (b.count == 0) return hipSuccess;
  hipLaunchKernelGGL(quant_weight_block128_batched_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, b);
  return hipGetLastError();
}

hipError_t launch_quant_act_token_group128(const uint16_t* a, int64_t m, int64_t k, int64_t lda,
                                           uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                           hipStream_t stream, bool pow2_scale) {
  // m * (k / 128) < 2^28 (checked by the caller), so the grid fits 32 bits.  Measured
  // on 8192 x 4096 inside the prefill step (weight requant, this, GEMM): 20.7 us,
  // against 22.0 us for workgroups over 16 consecutive (token, group) units in
  // row-major order, and 24.6 / 27.8 us with streaming loads (which pay off only
  // when the input is not in any cache: 24.1 vs 32.8 us after a cache flush).
  const uint32_t ng = (uint32_t)(k / 128);
  const uint32_t blocks = (uint32_t)((m + 15) / 16) * ng;
  if (pow2_scale)
    hipLaunchKernelGGL(quant_act_token_group128_kernel<true>, dim3(blocks), dim3(256), 0, stream,
                       a, lda, q, ldq, scale, ld_scale, (uint32_t)m, ng);
  else
    hipLaunchKernelGGL(quant_act_token_group128_kernel<false>, dim3(blocks), dim3(256), 0, stream,
                       a, lda, q, ldq, scale, ld_scale, (uint32_t)m, ng);
  return hipGetLastError();
}

}  // namespace fp8rl
