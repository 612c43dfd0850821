// Blockwise-scaled FP8 GEMM tile for gfx950 (CDNA4) MFMA.
//
// Computes one BN x BM output tile of  Y^T = W . A^T  over the whole K range:
// the weight tile provides the MFMA "A" operand (16 rows of n per instruction)
// and the activation tile the "B" operand (16 rows of m), so each lane's four
// fp32 results are four consecutive n of one token m -- an 8-byte bf16 store.
//
// K is walked in 128-wide steps, one per scale block (section 2.1.1: weight
// scales per 128x128 block, activation scales per 1x128 group).  A single
// v_mfma_f32_16x16x128_f8f6f4 covers exactly one K block of a 16x16 sub-tile,
// so its fp32 result is that block's partial sum; it is folded into the
// accumulator with one FMA by the combined scale sA[m, kb] * sW[nb, kb]:
//     acc += P_kb * (sA * sW)
// i.e. the per-K-block scale is applied in the epilogue of each K step.
//
// Data movement per K step: the block's W and A tiles (BN x 128 and BM x 128
// bytes) go global -> registers -> LDS (double-buffered), rows of 128 bytes
// with the 16-byte chunk index XOR-swizzled by (row & 7) so that the fragment
// reads (ds_read_b128) of 8 consecutive rows hit 8 distinct bank groups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace fp8rl {

typedef int v8i32 __attribute__((ext_vector_type(8)));
typedef float v4f32 __attribute__((ext_vector_type(4)));

template <int BN_, int BM_, int WN_, int WM_>
struct GemmCfg {
  static constexpr int BN = BN_;            // tile extent along n (weight rows)
  static constexpr int BM = BM_;            // tile extent along m (tokens)
  static constexpr int WN = WN_;            // waves along n
  static constexpr int WM = WM_;            // waves along m
  static constexpr int kWaves = WN * WM;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int WTN = BN / WN;       // wave tile along n
  static constexpr int WTM = BM / WM;       // wave tile along m
  static constexpr int TN = WTN / 16;       // 16x16 sub-tiles per wave along n
  static constexpr int TM = WTM / 16;       // ... along m
  static constexpr int kWBytes = BN * 128;  // one K step of the W tile
  static constexpr int kABytes = BM * 128;
  static constexpr int kStageBytes = kWBytes + kABytes;
  static constexpr int kLdsBytes = 2 * kStageBytes;
  static constexpr int kRowStep = kThreads / 8;           // rows covered by one load sweep
  static constexpr int kWLoads = BN / kRowStep;           // 16-byte loads per thread per K step
  static constexpr int kALoads = BM / kRowStep;
  static_assert(WTN % 16 == 0 && WTM % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(WTN <= 128 && 128 % WTN == 0, "a wave's n range must sit inside one 128-row scale block");
  static_assert(BN % kRowStep == 0 && BM % kRowStep == 0, "tile rows must be a multiple of the load sweep");
};

// Byte offset of 16-byte chunk `c` of row `r` in a swizzled 128-byte-row tile.
__device__ __forceinline__ int swz(int r, int c) { return r * 128 + ((c ^ (r & 7)) << 4); }

// 32-byte MFMA operand of one lane: two 16-byte chunks at byte offsets o0, o1.
__device__ __forceinline__ v8i32 lds_frag2(const uint8_t* base, int o0, int o1) {
  const uint4 lo = *reinterpret_cast<const uint4*>(base + o0);
  const uint4 hi = *reinterpret_cast<const uint4*>(base + o1);
  v8i32 f;
  f[0] = (int)lo.x; f[1] = (int)lo.y; f[2] = (int)lo.z; f[3] = (int)lo.w;
  f[4] = (int)hi.x; f[5] = (int)hi.y; f[6] = (int)hi.z; f[7] = (int)hi.w;
  return f;
}

__device__ __forceinline__ v4f32 mfma_fp8_16x16x128(const v8i32& a, const v8i32& b) {
  const v4f32 zero = {0.f, 0.f, 0.f, 0.f};
  // format codes 0/0 = E4M3 for both operands; scale operands 0 select the
  // plain (unscaled) v_mfma_f32_16x16x128_f8f6f4
  return __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, zero, 0, 0, 0, 0, 0, 0);
}

// One output tile.  Rows row_lo .. row_hi-1 of A / Y are valid for this tile
// (row_hi - row_lo may be less than BM: loads clamp to the last valid row, stores
// are masked).  n0 .. n0+BN-1 are the tile's weight rows; rows >= N are clamped
// on load and masked on store.  sw points at this weight's [N/128][KB] scales.
template <class C>
__device__ __forceinline__ void gemm_tile(const uint8_t* __restrict__ qa, int64_t lda,
                                          const float* __restrict__ sa, int64_t ld_sa,
                                          const uint8_t* __restrict__ qw, int64_t ldw,
                                          const float* __restrict__ sw,
                                          uint16_t* __restrict__ y, int64_t ldy,
                                          int64_t row_lo, int64_t row_hi, int64_t n0, int64_t N,
                                          int KB, uint8_t* lds) {
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wn = wave % C::WN;
  const int wm = wave / C::WN;
  const int n_valid = (int)min((int64_t)C::BN, N - n0);        // >= 1
  const int m_valid = (int)(row_hi - row_lo);                  // >= 1

  // ---- global -> LDS copy plan: thread t moves 16-byte chunk (t & 7) of tile
  //      rows (t >> 3) + i * kRowStep.  Since kRowStep is a multiple of 8,
  //      (row & 7) and hence the swizzled LDS chunk are fixed per thread.
  //      Global addresses are a wave-uniform 64-bit base (advanced by 128 bytes
  //      per K step) plus a 32-bit per-lane offset.
  const int c8 = t & 7;
  const int r8 = t >> 3;
  uint32_t ow[C::kWLoads];
  uint32_t oa[C::kALoads];
#pragma unroll
  for (int i = 0; i < C::kWLoads; ++i)
    ow[i] = (uint32_t)(min(r8 + i * C::kRowStep, n_valid - 1) * ldw + c8 * 16);
#pragma unroll
  for (int i = 0; i < C::kALoads; ++i)
    oa[i] = (uint32_t)(min(r8 + i * C::kRowStep, m_valid - 1) * lda + c8 * 16);
  const int lds_st = swz(r8, c8);           // + i * kRowStep * 128 for load i
  const uint8_t* wbase = qw + n0 * ldw;
  const uint8_t* abase = qa + row_lo * lda;

  uint4 rw[C::kWLoads];
  uint4 ra[C::kALoads];

  // ---- scales: this lane's tokens (one per 16-row m sub-tile) and this wave's
  //      128-row weight scale block
  uint32_t osa[C::TM];
#pragma unroll
  for (int tm = 0; tm < C::TM; ++tm) osa[tm] = (uint32_t)min(wm * C::WTM + tm * 16 + (lane & 15), m_valid - 1);
  const float* sabase = sa + row_lo;
  // a wave whose n range lies past N (tail tile) reads the last block's scales
  // and stores nothing
  const float* swrow = sw + ((min(n0 + wn * C::WTN, N - 1) >> 7) * KB);
  const bool wave_active_n = wn * C::WTN < n_valid;

  v4f32 acc[C::TN][C::TM];
#pragma unroll
  for (int i = 0; i < C::TN; ++i)
#pragma unroll
    for (int j = 0; j < C::TM; ++j) acc[i][j] = (v4f32){0.f, 0.f, 0.f, 0.f};

  const int frow = lane & 15;
  const int fg = lane >> 4;
  // fragment byte offsets inside a tile: row frow (+16 per sub-tile), chunks 2g, 2g+1
  const int f0 = frow * 128 + (((2 * fg) ^ (frow & 7)) << 4);
  const int f1 = frow * 128 + (((2 * fg + 1) ^ (frow & 7)) << 4);

  // prologue: K step 0 into stage 0
#pragma unroll
  for (int i = 0; i < C::kWLoads; ++i) rw[i] = *reinterpret_cast<const uint4*>(wbase + ow[i]);
#pragma unroll
  for (int i = 0; i < C::kALoads; ++i) ra[i] = *reinterpret_cast<const uint4*>(abase + oa[i]);
#pragma unroll
  for (int i = 0; i < C::kWLoads; ++i)
    *reinterpret_cast<uint4*>(lds + lds_st + i * C::kRowStep * 128) = rw[i];
#pragma unroll
  for (int i = 0; i < C::kALoads; ++i)
    *reinterpret_cast<uint4*>(lds + C::kWBytes + lds_st + i * C::kRowStep * 128) = ra[i];
  __syncthreads();

  for (int kb = 0; kb < KB; ++kb) {
    // next K step's tiles into registers (the last step reloads itself; the
    // copy then goes to the idle stage and is never read)
    {
      const int kn = min(kb + 1, KB - 1);
      const uint8_t* wb = wbase + kn * 128;
      const uint8_t* ab = abase + kn * 128;
#pragma unroll
      for (int i = 0; i < C::kWLoads; ++i) rw[i] = *reinterpret_cast<const uint4*>(wb + ow[i]);
#pragma unroll
      for (int i = 0; i < C::kALoads; ++i) ra[i] = *reinterpret_cast<const uint4*>(ab + oa[i]);
    }

    const float swv = swrow[kb];
    const float* sak = sabase + (int64_t)kb * ld_sa;
    float sc[C::TM];
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) sc[tm] = sak[osa[tm]] * swv;

    const uint8_t* st = lds + (kb & 1) * C::kStageBytes;
    const uint8_t* sta = st + C::kWBytes + wm * C::WTM * 128;
    const uint8_t* stw = st + wn * C::WTN * 128;
    v8i32 bf[C::TM];
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) bf[tm] = lds_frag2(sta + tm * 16 * 128, f0, f1);
#pragma unroll
    for (int tn = 0; tn < C::TN; ++tn) {
      const v8i32 af = lds_frag2(stw + tn * 16 * 128, f0, f1);
#pragma unroll
      for (int tm = 0; tm < C::TM; ++tm) {
        const v4f32 p = mfma_fp8_16x16x128(af, bf[tm]);
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[tn][tm][r] = __builtin_fmaf(p[r], sc[tm], acc[tn][tm][r]);
      }
    }

    {
      uint8_t* sn = lds + ((kb + 1) & 1) * C::kStageBytes;
#pragma unroll
      for (int i = 0; i < C::kWLoads; ++i) *reinterpret_cast<uint4*>(sn + lds_st + i * C::kRowStep * 128) = rw[i];
#pragma unroll
      for (int i = 0; i < C::kALoads; ++i)
        *reinterpret_cast<uint4*>(sn + C::kWBytes + lds_st + i * C::kRowStep * 128) = ra[i];
    }
    __syncthreads();
  }

  // ---- epilogue: fp32 -> bf16 (RNE), four consecutive n per lane
  if (!wave_active_n) return;
#pragma unroll
  for (int tn = 0; tn < C::TN; ++tn) {
    const int nl = wn * C::WTN + tn * 16 + 4 * fg;
    if (nl >= n_valid) continue;
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) {
      const int ml = wm * C::WTM + tm * 16 + frow;
      if (ml >= m_valid) continue;
      uint2 o;
      o.x = f32_to_bf16_rne(acc[tn][tm][0]) | (f32_to_bf16_rne(acc[tn][tm][1]) << 16);
      o.y = f32_to_bf16_rne(acc[tn][tm][2]) | (f32_to_bf16_rne(acc[tn][tm][3]) << 16);
      *reinterpret_cast<uint2*>(y + (row_lo + ml) * ldy + n0 + nl) = o;
    }
  }
}

}  // namespace fp8rl
