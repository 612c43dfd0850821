// Blockwise-scaled FP8 GEMM tile for gfx950 (CDNA4) MFMA.
//
// Computes one BN x BM output tile of  Y^T = W . A^T  over the whole K range:
// the weight tile provides the MFMA "A" operand (16 rows of n per instruction)
// and the activation tile the "B" operand (16 rows of m), so each lane's four
// fp32 results are four consecutive n of one token m.
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
// XOR-swizzled so that the fragment reads (ds_read_b128) are free of bank
// conflicts.  The finished tile is converted to bf16, staged in LDS and written
// as whole output rows.
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
  static constexpr int kSBytes = BM * 4;    // one K step of the activation scales
  static constexpr int kStageBytes = kWBytes + kABytes + kSBytes;
  static constexpr int kLdsBytes = STAGES * kStageBytes;
  // one direct-to-LDS wave instruction moves 8 rows x 128 bytes (1 KiB)
  static constexpr int kOctets = (BN + BM) / 8;
  static constexpr int kLoadsPerWave = kOctets / kWaves;
  // activation scales: 64 tokens (one dword each) per wave instruction
  static constexpr int kScaleLoads = BM / 64;
  static_assert(BM % 64 == 0 && kScaleLoads <= kWaves, "one scale DMA per wave at most");
  static_assert(WTN % 16 == 0 && WTM % 16 == 0, "wave tile must be a multiple of 16");
  static_assert(WTN <= 128 && 128 % WTN == 0, "a wave's n range must sit inside one 128-row scale block");
  static_assert(kOctets % kWaves == 0, "row octets must divide evenly among the waves");
  static_assert(STAGES >= 2, "need at least double buffering");
  static_assert(kLdsBytes <= 160 * 1024, "LDS is 160 KiB per CU");
};

// LDS tile layout: rows of 128 bytes (one K step), eight 16-byte chunks per
// row; logical chunk c of row r is stored at physical chunk c ^ swz_key(r).
// A fragment read (ds_read_b128) has 16 lanes reading the same logical chunk
// of 16 consecutive rows.  With 64 banks of 4 bytes, row r's physical chunk p
// lands on banks 32 (r & 1) + 4p .. +3, so the 16 rows need distinct
// (r & 1, p): the key below is a permutation of 0..7 over the even rows and
// over the odd rows of any 16-row group (and over any 8 consecutive rows,
// which also keeps a 32-bank LDS conflict-free).
__device__ __forceinline__ int swz_key(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ int swz(int r, int c) { return r * 128 + ((c ^ swz_key(r)) << 4); }

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

// 4 bytes per lane, global -> LDS (global_load_lds_dword): lane L writes
// LDS bytes [lds_wave_base + 4 L, +4).
__device__ __forceinline__ void lds_dma4(const float* gptr, uint8_t* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((global_void_t*)gptr, (lds_void_t*)lds_wave_base, 4, 0, 0);
}

// 16-byte streaming (non-temporal) store of eight bf16
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store_stream16(uint16_t* p, const uint4& v) {
  const u32x4_t w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
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
// on load and masked on store.  The tile sums KB K blocks starting where qa, sa,
// qw and sw point; sw rows (one per 128 weight rows) are sw_ld floats apart.
// kPartial: write the fp32 sums to part (row stride ldp) instead of bf16 to y
// (one K range of a split-K product; the caller adds the ranges).
//
// Pipeline (STAGES-deep LDS ring, one barrier per K step):
//   prologue: DMA K steps 0 .. STAGES-2
//   step kb:  wait for this wave's DMA of step kb; barrier (all waves' DMA of
//             step kb landed, all waves done reading step kb-1's slot);
//             MFMA + scale-FMA on slot kb % STAGES, with the DMA of step
//             kb+STAGES-1 into the slot freed by step kb-1 interleaved.
// A slot holds the W tile, the A tile and the tile's BM activation scales of
// one K step; the weight scale is a wave-uniform scalar load.  The DMA is then
// the only vector-memory traffic of the loop, so the one explicit vmcnt wait
// per step is the only wait on global memory.
template <class C, bool kPartial = false>
__device__ __forceinline__ void gemm_tile(const uint8_t* __restrict__ qa, int64_t lda,
                                          const float* __restrict__ sa, int64_t ld_sa,
                                          const uint8_t* __restrict__ qw, int64_t ldw,
                                          const float* __restrict__ sw, int sw_ld,
                                          uint16_t* __restrict__ y, int64_t ldy,
                                          float* __restrict__ part, int64_t ldp,
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
  //      logical chunk (L & 7) ^ swz_key(row) of the swizzled layout.
  const int lrow = lane >> 3;
  uint32_t goff[C::kLoadsPerWave];
  bool is_w[C::kLoadsPerWave];
#pragma unroll
  for (int i = 0; i < C::kLoadsPerWave; ++i) {
    const int o = wave + i * C::kWaves;                 // wave-uniform
    is_w[i] = o < C::BN / 8;
    const int r = (is_w[i] ? o : o - C::BN / 8) * 8 + lrow;
    const int lchunk = (lane & 7) ^ swz_key(r);
    goff[i] = is_w[i] ? (uint32_t)(min(r, n_valid - 1) * ldw + lchunk * 16)
                      : (uint32_t)(min(r, m_valid - 1) * lda + lchunk * 16);
  }
  const uint8_t* wbase = qw + n0 * ldw;
  const uint8_t* abase = qa + row_lo * lda;

  // ---- scales: wave w < kScaleLoads DMAs tokens 64w .. 64w+63 of the tile
  //      (clamped to the last valid row); this wave's 128-row weight scale
  //      block is read with scalar loads (a wave past N reads the last block
  //      and stores nothing)
  const bool sdma = wave < C::kScaleLoads;
  const float* sa_lane = sa + row_lo + min(wave * 64 + lane, m_valid - 1);
  const float* swrow = sw + ((min(n0 + wn * C::WTN, N - 1) >> 7) * sw_ld);
  auto dma_stage = [&](int kb, int slot) {
    uint8_t* sbase = lds + slot * C::kStageBytes;
    const uint8_t* wb = wbase + kb * 128;
    const uint8_t* ab = abase + kb * 128;
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) {
      const int o = wave + i * C::kWaves;
      lds_dma16((is_w[i] ? wb : ab) + goff[i], sbase + o * 1024);
    }
    if (sdma) lds_dma4(sa_lane + (int64_t)kb * ld_sa, sbase + C::kWBytes + C::kABytes + wave * 256);
  };

  v4f32 acc[C::TN][C::TM];
#pragma unroll
  for (int i = 0; i < C::TN; ++i)
#pragma unroll
    for (int j = 0; j < C::TM; ++j) acc[i][j] = (v4f32){0.f, 0.f, 0.f, 0.f};

  const int frow = lane & 15;
  const int fg = lane >> 4;
  // fragment byte offsets inside a tile: row frow (+16 per sub-tile), chunks 2g, 2g+1
  // (sub-tiles start at multiples of 16 rows, so swz_key(row) = swz_key(frow))
  const int f0 = swz(frow, 2 * fg);
  const int f1 = swz(frow, 2 * fg + 1);

  // prologue
#pragma unroll
  for (int s = 0; s < C::STAGES - 1; ++s)
    if (s < KB) dma_stage(s, s);

  for (int kb = 0; kb < KB; ++kb) {
    // step kb's DMA is the oldest still outstanding: up to STAGES-2 younger
    // stages (kLoadsPerWave tile loads + at most one scale load each) may stay
    // in flight; near the end of K fewer were issued, so wait for everything
    if (kb + C::STAGES - 2 < KB) {
      if (sdma)
        wait_vmcnt<(C::STAGES - 2) * (C::kLoadsPerWave + 1)>();
      else
        wait_vmcnt<(C::STAGES - 2) * C::kLoadsPerWave>();
    } else {
      wait_vmcnt<0>();
    }
    __syncthreads();

    // refill the slot released by step kb-1 with step kb+STAGES-1 (none past
    // the end of K).  With 8 sub-tile rows per wave the DMA instructions are
    // spread over the first half of the sub-tile loop below (issued all at once
    // they stall the wave on a full address queue, issued later they arrive
    // after the next barrier); with fewer, all are issued with the first one
    // (measured fastest for the 128x128 tiles).
    const bool refill = kb + C::STAGES - 1 < KB;
    const int kd = min(kb + C::STAGES - 1, KB - 1);   // (only used when refill)
    uint8_t* dslot = lds + ((kb + C::STAGES - 1) % C::STAGES) * C::kStageBytes;
    const uint8_t* dwb = wbase + kd * 128;
    const uint8_t* dab = abase + kd * 128;

    constexpr int kDmaSpread = C::TN >= 8 ? C::TN / 2 : 1;   // sub-tile rows that carry DMA issue
    const uint8_t* st = lds + (kb % C::STAGES) * C::kStageBytes;
    const float* sts = reinterpret_cast<const float*>(st + C::kWBytes + C::kABytes) + wm * C::WTM + (lane & 15);
    const float swv = swrow[kb];
    float sc[C::TM];
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) sc[tm] = sts[tm * 16] * swv;

    const uint8_t* sta = st + C::kWBytes + wm * C::WTM * 128;
    const uint8_t* stw = st + wn * C::WTN * 128;
    // first weight fragment, then the activation fragments in the order the
    // first MFMAs consume them (LDS returns in order, so each MFMA waits only
    // for its own operands); weight fragments are double-buffered: the next
    // sub-tile's read is in flight while this one's MFMAs run
    v8i32 af = lds_frag2(stw, f0, f1);
    v8i32 bf[C::TM];
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) bf[tm] = lds_frag2(sta + tm * 16 * 128, f0, f1);
#pragma unroll
    for (int tn = 0; tn < C::TN; ++tn) {
#pragma unroll
      for (int i = 0; i < C::kLoadsPerWave; ++i) {
        if ((i * kDmaSpread) / C::kLoadsPerWave == tn && refill) {
          const int o = wave + i * C::kWaves;
          lds_dma16((is_w[i] ? dwb : dab) + goff[i], dslot + o * 1024);
        }
      }
      if (tn == 0 && sdma && refill) lds_dma4(sa_lane + (int64_t)kd * ld_sa, dslot + C::kWBytes + C::kABytes + wave * 256);
      v8i32 af_next = af;
      if (tn + 1 < C::TN) af_next = lds_frag2(stw + (tn + 1) * 16 * 128, f0, f1);
      // all MFMAs of the sub-tile row first (independent results in flight),
      // then their scale FMAs
      v4f32 p[C::TM];
#pragma unroll
      for (int tm = 0; tm < C::TM; ++tm) p[tm] = mfma_fp8_16x16x128(af, bf[tm]);
#pragma unroll
      for (int tm = 0; tm < C::TM; ++tm)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[tn][tm][r] = __builtin_fmaf(p[tm][r], sc[tm], acc[tn][tm][r]);
      af = af_next;
    }

  }
  // (the last iteration waited for every DMA: nothing is in flight here)

  if constexpr (kPartial) {
    // ---- split-K partial: the fp32 sums, four consecutive n per lane (16 bytes)
#pragma unroll
    for (int tn = 0; tn < C::TN; ++tn) {
      const int nl = wn * C::WTN + tn * 16 + 4 * fg;
#pragma unroll
      for (int tm = 0; tm < C::TM; ++tm) {
        const int ml = wm * C::WTM + tm * 16 + frow;
        if (ml < m_valid && nl < n_valid)
          *reinterpret_cast<v4f32*>(part + (row_lo + ml) * ldp + n0 + nl) = acc[tn][tm];
      }
    }
    return;
  }

  // ---- epilogue: fp32 -> bf16 (RNE) into a copy of the whole tile in LDS (the
  //      ring is free once every wave is past its last K step), then each
  //      workgroup writes full 16-byte chunks of whole output rows with
  //      streaming stores.  Direct 8-byte stores from the MFMA layout wrote
  //      partial cache lines (1.6x the output bytes reached HBM) and let the
  //      output displace the operands in the memory-side cache.
  //      LDS layout: BM rows of BN bf16; 16-byte chunk c of row r sits at
  //      c ^ (r & 15), so the 16 rows of one fragment store, and the two rows
  //      of one read-back wave instruction, spread evenly over the 64 banks.
  constexpr int kRowBytes = C::BN * 2;
  constexpr int kChunks = kRowBytes / 16;
  static_assert(kChunks >= 16 && C::BM * kRowBytes <= C::kLdsBytes, "the bf16 tile must fit in the LDS ring");
  __syncthreads();
#pragma unroll
  for (int tn = 0; tn < C::TN; ++tn) {
    const int nl = wn * C::WTN + tn * 16 + 4 * fg;
#pragma unroll
    for (int tm = 0; tm < C::TM; ++tm) {
      const int ml = wm * C::WTM + tm * 16 + frow;
      uint2 o;
      o.x = f32_to_bf16_rne(acc[tn][tm][0]) | (f32_to_bf16_rne(acc[tn][tm][1]) << 16);
      o.y = f32_to_bf16_rne(acc[tn][tm][2]) | (f32_to_bf16_rne(acc[tn][tm][3]) << 16);
      *reinterpret_cast<uint2*>(lds + ml * kRowBytes + (((nl >> 3) ^ (ml & 15)) << 4) + ((nl >> 2) & 1) * 8) = o;
    }
  }
  __syncthreads();
  const int c = t % kChunks;                    // this thread's chunk of every row it writes
#pragma unroll 4
  for (int r = t / kChunks; r < C::BM; r += C::kThreads / kChunks) {
    if (r < m_valid && c * 8 < n_valid) {
      const uint4 v = *reinterpret_cast<const uint4*>(lds + r * kRowBytes + ((c ^ (r & 15)) << 4));
      store_stream16(y + (row_lo + r) * ldy + n0 + c * 8, v);
    }
  }
}

}  // namespace fp8rl
