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
// bytes) go straight from global memory into an LDS ring (global_load_lds,
// no register staging), rows of 128 bytes with the 16-byte chunk index
// XOR-swizzled by (row & 7) so that the fragment reads (ds_read_b128) of 8
// consecutive rows hit 8 distinct bank groups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace fp8rl {

typedef int v8i32 __attribute__((ext_vector_type(8)));
typedef float v4f32 __attribute__((ext_vector_type(4)));

template <int BN_, int BM_, int WN_, int WM_, int STAGES_>
struct GemmCfg {
  static constexpr int BN = BN_;            // tile extent along n (weight rows)
  static constexpr int BM = BM_;            // tile extent along m (tokens)
  static constexpr int WN = WN_;            // waves along n
  static constexpr int WM = WM_;            // waves along m
  static constexpr int STAGES = STAGES_;    // LDS ring depth (K steps in flight)
  static constexpr int kWaves = WN * WM;
  static constexpr int kThreads = kWaves * 64;
  static constexpr int WTN = BN / WN;       // wave tile along n
  static constexpr int WTM = BM / WM;       // wave tile along m
  static constexpr int TN = WTN / 16;       // 16x16 sub-tiles per wave along n
  static constexpr int TM = WTM / 16;       // ... along m
  static constexpr int kWBytes = BN * 128;  // one K step of the W tile
  static constexpr int kABytes = BM * 128;
  static constexpr int kStageBytes = kWBytes + kABytes;
  static constexpr int kLdsBytes = STAGES * kStageBytes;
  // one direct-to-LDS wave instruction moves 8 rows x 128 bytes (1 KiB)
  static constexpr int kOctets = (BN + BM) / 8;
  static constexpr int kLoadsPerWave = kOctets / kWaves;
  static_assert(WTN % 16 == 0 && WTM % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(WTN <= 128 && 128 % WTN == 0, "a wave's n range must sit inside one 128-row scale block");
  static_assert(kOctets % kWaves == 0, "row octets must divide evenly among the waves");
  static_assert(STAGES >= 2, "need at least double buffering");
  static_assert(kLdsBytes <= 160 * 1024, "LDS is 160 KiB per CU");
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

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) const void global_void_t;

// 16 bytes per lane, global -> LDS without passing through registers
// (global_load_lds_dwordx4): lane L of the wave writes LDS bytes
// [lds_wave_base + 16 L, +16).  lds_wave_base must be wave-uniform.
__device__ __forceinline__ void lds_dma16(const uint8_t* gptr, uint8_t* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((global_void_t*)gptr, (lds_void_t*)lds_wave_base, 16, 0, 0);
}

// s_waitcnt vmcnt(n) only (expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// One output tile.  Rows row_lo .. row_hi-1 of A / Y are valid for this tile
// (row_hi - row_lo may be less than BM: loads clamp to the last valid row, stores
// are masked).  n0 .. n0+BN-1 are the tile's weight rows; rows >= N are clamped
// on load and masked on store.  sw points at this weight's [N/128][KB] scales.
//
// Pipeline (STAGES-deep LDS ring, one barrier per K step):
//   prologue: DMA K steps 0 .. STAGES-2
//   step kb:  wait for this wave's DMA of step kb; barrier (all waves' DMA of
//             step kb landed, all waves done reading step kb-1's slot);
//             prefetch next step's scales; DMA step kb+STAGES-1 into the slot
//             freed by step kb-1; MFMA + scale-FMA on slot kb % STAGES.
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

  // ---- DMA plan: wave w moves row octets w, w + kWaves, ...  In an octet,
  //      lane L lands at row 8o + (L >> 3), physical chunk (L & 7), which holds
  //      logical chunk (L & 7) ^ (row & 7) of the swizzled layout.
  const int lrow = lane >> 3;
  const int lchunk = (lane & 7) ^ lrow;
  uint32_t goff[C::kLoadsPerWave];
  bool is_w[C::kLoadsPerWave];
#pragma unroll
  for (int i = 0; i < C::kLoadsPerWave; ++i) {
    const int o = wave + i * C::kWaves;                 // wave-uniform
    is_w[i] = o < C::BN / 8;
    const int r = (is_w[i] ? o : o - C::BN / 8) * 8 + lrow;
    goff[i] = is_w[i] ? (uint32_t)(min(r, n_valid - 1) * ldw + lchunk * 16)
                      : (uint32_t)(min(r, m_valid - 1) * lda + lchunk * 16);
  }
  const uint8_t* wbase = qw + n0 * ldw;
  const uint8_t* abase = qa + row_lo * lda;

  auto dma_stage = [&](int kb, int slot) {
    uint8_t* sbase = lds + slot * C::kStageBytes;
    const uint8_t* wb = wbase + kb * 128;
    const uint8_t* ab = abase + kb * 128;
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) {
      const int o = wave + i * C::kWaves;
      lds_dma16((is_w[i] ? wb : ab) + goff[i], sbase + o * 1024);
    }
  };

  // ---- scales: this lane's tokens (one per 16-row m sub-tile) and this wave's
  //      128-row weight scale block (a wave past N reads the last block and
  //      stores nothing)
  uint32_t osa[C::TM];
#pragma unroll
  for (int tm = 0; tm < C::TM; ++tm) osa[tm] = (uint32_t)min(wm * C::WTM + tm * 16 + (lane & 15), m_valid - 1);
  const float* sabase = sa + row_lo;
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

  // prologue
  float sa_cur[C::TM];
#pragma unroll
  for (int tm = 0; tm < C::TM; ++tm) sa_cur[tm] = sabase[osa[tm]];
  float sw_cur = swrow[0];
#pragma unroll
  for (int s = 0; s < C::STAGES - 1; ++s) dma_stage(min(s, KB - 1), s);

  for (int kb = 0; kb < KB; ++kb) {
    // step kb's DMA is the oldest still outstanding: STAGES-2 younger stages may stay in flight
    wait_vmcnt<(C::STAGES - 2) * C::kLoadsPerWave>();
    __syncthreads();

    // next step's scales (clamped: the last step reloads its own)
    const int kn = min(kb + 1, KB - 1);
    float sa_nxt[C::TM];
    const float* sak = sabase + (int64_t)kn * ld_sa;
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) sa_nxt[tm] = sak[osa[tm]];
    const float sw_nxt = swrow[kn];

    // refill the slot released by step kb-1 (past the end: reload the last step)
    dma_stage(min(kb + C::STAGES - 1, KB - 1), (kb + C::STAGES - 1) % C::STAGES);

    float sc[C::TM];
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) sc[tm] = sa_cur[tm] * sw_cur;

    const uint8_t* st = lds + (kb % C::STAGES) * C::kStageBytes;
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

#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) sa_cur[tm] = sa_nxt[tm];
    sw_cur = sw_nxt;
  }
  // drain the trailing (redundant) DMA before the workgroup may exit
  wait_vmcnt<0>();

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
