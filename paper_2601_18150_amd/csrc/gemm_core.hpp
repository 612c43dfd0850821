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
// With power-of-two (UE8M0) scales (section 2.4.3) the MX-scaled form of the
// same instruction applies 2^(eA + eW) to the products itself and accumulates
// straight into acc: no per-step scale arithmetic (kMx).
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

// Raw buffer resource at base (stride 0, range 4 GiB - 1, so no offset used
// here is clamped: the DMA offsets are relative to a tile's first row, at most
// 256 rows x a leading dimension below 2^24 plus K).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, -1, 0x00020000);
}

// The 16-byte DMA through a buffer resource (buffer_load_dwordx4 ... lds): lane
// address = base + voff + soff, with a 32-bit per-lane offset (one VGPR) and a
// wave-uniform one (an SGPR).  Used in the K loop, where the 64-bit per-lane
// addresses of global_load_lds would hold two VGPRs per load.
__device__ __forceinline__ void lds_dma16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                          uint8_t* lds_wave_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds_wave_base, 16, voff, soff, 0, 0);
}

// 16-byte streaming (non-temporal) store of eight bf16
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store_stream16(uint16_t* p, const uint4& v) {
  const u32x4_t w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4_t*>(p));
}

// Workgroup barrier for data shared through LDS only: waits for this wave's
// LDS operations (lgkmcnt(0)), then s_barrier.  Unlike __syncthreads() it does
// not wait for outstanding global stores or DMA loads (their vmcnt waits are
// explicit); the empty asm statements keep the compiler from moving memory
// operations across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14));   // lgkmcnt(0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt vmcnt(n) only (expcnt and lgkmcnt left at their maxima)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// At the top of a K step with `later` further steps' DMA already issued behind
// it (kPer wave instructions each), wait until this step's DMA has landed.
// Loads complete in issue order, so vmcnt(later * kPer) suffices; the count
// must be an immediate, hence the branches (later <= S - 2).
template <int S, int kPer>
__device__ __forceinline__ void wait_dma_step(int later) {
  static_assert(S >= 2 && S <= 4, "ring depth 2..4");
  if constexpr (S == 2) {
    wait_vmcnt<0>();
  } else if constexpr (S == 3) {
    if (later >= 1) wait_vmcnt<kPer>(); else wait_vmcnt<0>();
  } else {
    if (later >= 2) wait_vmcnt<2 * kPer>(); else if (later == 1) wait_vmcnt<kPer>(); else wait_vmcnt<0>();
  }
}

// One output tile to compute (wave-uniform values, produced by a job provider).
struct TileJob {
  int row_lo;              // first row of A / Y
  int m_valid;             // rows of the tile that exist, 1 .. BM
  int n0;                  // first weight row (output column)
  int64_t qw_off;          // weight codes of this tile's matrix: qw + qw_off, [N][ldw]
  int64_t sw_off;          // its block scales: sw + sw_off, rows of sw_ld floats
  // (offsets rather than pointers: addresses derived from the kernel's
  // __restrict__ arguments keep their no-alias, read-only provenance, so the
  // compiler neither orders the output stores after the operand loads nor turns
  // the scale reads into vector loads)
};

// Tiles of  Y^T = W . A^T  computed by one workgroup, one after another; the
// job provider `jobs` hands them out (jobs.next(j) returns false at the end; it
// must not touch LDS or synchronise).  Rows >= M of a tile are clamped on load
// and masked on store, weight rows >= N likewise.  Each tile sums KB K blocks
// starting where qa, sa, qw + qw_off and sw + sw_off point; sw rows (one per
// 128 weight rows) are sw_ld floats apart.  kPartial: write the fp32 sums to part (rows of
// N floats) instead of bf16 to y (one K range of a split-K product).
//
// Pipeline (S-slot LDS ring, S = C::STAGES, one barrier per K step):
//   prologue: the DMA of steps 0 .. S-2 into slots 0 .. S-2.
//   step s:  wait for this wave's DMA of step s; barrier (all waves' DMA of step
//            s landed, all waves done reading step s-1's slot); MFMA + scale-FMA
//            on slot s % S, with the DMA of step s+S-1 into the slot of step s-1
//            interleaved.  S - 1 K steps are in flight while one is computed.
//   kCross (2-slot ring only): after a tile's last K block, step s+1 is the
//            first K block of the workgroup's next tile, so consecutive tiles
//            form one pipeline and the next tile's first load overlaps this
//            tile's last step and output.  Without it the workgroup computes its
//            first tile only (the 256x256 tile, whose registers are full, runs
//            one tile per workgroup).
//   tile end: the bf16 tile is staged through the slot of its last step (in
//            row groups that fit one slot) and written as whole output rows.
// A slot holds the W tile, the A tile and the tile's BM activation scales of
// one K step; the weight scale is a wave-uniform scalar load.  The DMA is then
// the only vector-memory traffic of the loop, so the one explicit vmcnt wait
// per step is the only wait on global memory (at a tile's first step it also
// covers the previous tile's output stores).
//
// kGather: row r of a tile (output row row_lo + r) takes its activation codes
// and scales from source row gidx[row_lo + r] of qa / sa (clamped into
// [0, src_rows)), so a gather of quantised rows (MoE dispatch) needs no copy.
// The row indices of the next tile are loaded when that tile is picked, one
// tile ahead, and turned into DMA offsets at the current tile's last step,
// after the per-step vmcnt(0) waits have retired them (2-slot ring only).
template <class C, bool kPartial, bool kCross, class Jobs, bool kMx = false, bool kGather = false>
__device__ __forceinline__ void gemm_tiles(const uint8_t* __restrict__ qa, int64_t lda,
                                           const float* __restrict__ sa, int64_t ld_sa,
                                           const uint8_t* __restrict__ qw, int64_t ldw,
                                           const float* __restrict__ sw, int sw_ld,
                                           uint16_t* __restrict__ y, int64_t ldy, float* __restrict__ part,
                                           int N, int KB, Jobs& jobs, uint8_t* lds,
                                           const int32_t* __restrict__ gidx = nullptr, int src_rows = 0) {
  constexpr int S = C::STAGES;
  static_assert(S == 2 || !kCross, "the cross-tile pipeline is written for a 2-slot ring");
  static_assert(!kGather || (S == 2 && kCross && !kPartial), "row gather: 2-slot cross-tile pipeline only");
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wn = wave % C::WN;
  const int wm = wave / C::WN;
  const int frow = lane & 15;
  const int fg = lane >> 4;
  // fragment byte offsets inside a tile: row frow (+16 per sub-tile), chunks 2g, 2g+1
  // (sub-tiles start at multiples of 16 rows, so swz_key(row) = swz_key(frow))
  const int f0 = swz(frow, 2 * fg);
  const int f1 = swz(frow, 2 * fg + 1);

  // ---- DMA plan: wave w moves row octets w, w + kWaves, ...  In an octet,
  //      lane L lands at row 8o + (L >> 3), physical chunk (L & 7), which holds
  //      logical chunk (L & 7) ^ swz_key(row) of the swizzled layout.  The
  //      per-lane byte offsets clamp rows past the tile's valid range.
  const int lrow = lane >> 3;
  // (kGather: rs[i] is the source row of octet i's activation row; the offsets
  // are then relative to qa itself rather than to the tile's first row)
  auto dma_offsets = [&](uint32_t (&g)[C::kLoadsPerWave], int n_valid, int m_valid,
                         const int32_t (&rs)[C::kLoadsPerWave]) {
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) {
      const int o = wave + i * C::kWaves;               // wave-uniform
      const bool w = o < C::BN / 8;
      const int r = (w ? o : o - C::BN / 8) * 8 + lrow;
      const int lchunk = (lane & 7) ^ swz_key(r);
      const int arow = kGather ? rs[i] : min(r, m_valid - 1);
      g[i] = w ? (uint32_t)(min(r, n_valid - 1) * ldw + lchunk * 16)
               : (uint32_t)(arow * lda + lchunk * 16);
    }
  };
  // kGather: issue the loads of a tile's source rows (octet rows and this
  // lane's scale row); they are consumed a tile later
  auto load_rows = [&](const TileJob& j, int32_t (&rs)[C::kLoadsPerWave], int32_t& srow) {
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) {
      const int o = wave + i * C::kWaves;
      rs[i] = 0;
      if (o >= C::BN / 8) rs[i] = gidx[j.row_lo + min((o - C::BN / 8) * 8 + lrow, j.m_valid - 1)];
    }
    srow = gidx[j.row_lo + min(wave * 64 + lane, j.m_valid - 1)];
  };
  auto clamp_rows = [&](int32_t (&rs)[C::kLoadsPerWave], int32_t& srow) {
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) rs[i] = min(max(rs[i], 0), src_rows - 1);
    srow = min(max(srow, 0), src_rows - 1);
  };
  // scales: wave w < kScaleLoads DMAs tokens 64w .. 64w+63 of the tile (clamped
  // to the last valid row); this wave's 128-row weight scale block is read with
  // scalar loads (a wave past N reads the last block and stores nothing)
  const bool sdma = wave < C::kScaleLoads;
  auto n_valid_of = [&](const TileJob& j) { return min(C::BN, N - j.n0); };
  auto sa_lane_of = [&](const TileJob& j) { return sa + j.row_lo + min(wave * 64 + lane, j.m_valid - 1); };

  TileJob cur;
  if (!jobs.next(cur)) return;
  TileJob nxt = cur;
  bool has_nxt = false;
  uint32_t goff[C::kLoadsPerWave], goff_n[C::kLoadsPerWave];
  int32_t rs_c[C::kLoadsPerWave] = {}, rs_n[C::kLoadsPerWave] = {};
  int32_t srow_c = 0, srow_n = 0;
  if constexpr (kGather) {
    load_rows(cur, rs_c, srow_c);
    clamp_rows(rs_c, srow_c);
  }
  dma_offsets(goff, n_valid_of(cur), cur.m_valid, rs_c);
  if constexpr (kCross) {
    has_nxt = jobs.next(nxt);
    if constexpr (kGather) {
      if (has_nxt) load_rows(nxt, rs_n, srow_n);
    } else {
      if (has_nxt) dma_offsets(goff_n, n_valid_of(nxt), nxt.m_valid, rs_n);
    }
  }
  // this lane's activation-scale row of a tile (the scale DMA of waves < kScaleLoads)
  auto sa_lane_cur = [&]() { return kGather ? sa + srow_c : sa_lane_of(cur); };

  // prologue: the first tile's first S-1 K blocks into slots 0 .. S-2
#pragma unroll
  for (int p = 0; p < S - 1; ++p) {
    if (p > 0 && p >= KB) break;
    const uint8_t* wb = qw + cur.qw_off + (int64_t)cur.n0 * ldw + p * 128;
    const uint8_t* ab = (kGather ? qa : qa + (int64_t)cur.row_lo * lda) + p * 128;
    uint8_t* ps = lds + p * C::kStageBytes;
#pragma unroll
    for (int i = 0; i < C::kLoadsPerWave; ++i) {
      const int o = wave + i * C::kWaves;
      lds_dma16((o < C::BN / 8 ? wb : ab) + goff[i], ps + o * 1024);
    }
    if (sdma) lds_dma4(sa_lane_cur() + (int64_t)p * ld_sa, ps + C::kWBytes + C::kABytes + wave * 256);
  }

  int slot = 0;
  for (;;) {
    const int n_valid = n_valid_of(cur);
    const uint8_t* wbase = qw + cur.qw_off + (int64_t)cur.n0 * ldw;
    const uint8_t* abase = kGather ? qa : qa + (int64_t)cur.row_lo * lda;
    const float* sa_lane = sa_lane_cur();
    const float* swrow = sw + cur.sw_off + (int64_t)(min(cur.n0 + wn * C::WTN, N - 1) >> 7) * sw_ld;

    v4f32 acc[C::TN][C::TM];
#pragma unroll
    for (int i = 0; i < C::TN; ++i)
#pragma unroll
      for (int j = 0; j < C::TM; ++j) acc[i][j] = (v4f32){0.f, 0.f, 0.f, 0.f};

    for (int kb = 0; kb < KB; ++kb) {
      // this step's DMA (with S = 2 also a previous tile's output stores)
      const int later = min(S - 2, KB - 1 - kb);
      if (sdma) wait_dma_step<S, C::kLoadsPerWave + 1>(later);
      else wait_dma_step<S, C::kLoadsPerWave>(later);
      lds_barrier();

      // refill the slot of step s-1 with step s+S-1: a later K block of this
      // tile or, with kCross after its last, the first K block of the next tile
      // (if any).  With 8
      // sub-tile rows per wave the DMA instructions are spread over the first
      // half of the sub-tile loop below (issued all at once they stall the wave
      // on a full address queue, issued later they arrive after the next
      // barrier); with fewer, all are issued with the first one (measured
      // fastest for the 128x128 tiles).
      const bool last = kb + 1 == KB;
      const bool refill = kb + S - 1 < KB || (last && has_nxt);
      uint8_t* dslot = lds + (slot == 0 ? S - 1 : slot - 1) * C::kStageBytes;
      const uint8_t* dwb = wbase;
      const uint8_t* dab = abase;
      uint32_t dsoff = (kb + S - 1) * 128;
      const float* dsa = sa_lane + (int64_t)(kb + S - 1) * ld_sa;
      if constexpr (kCross) {
        if (last) {
          dwb = qw + nxt.qw_off + (int64_t)nxt.n0 * ldw;
          dab = kGather ? qa : qa + (int64_t)nxt.row_lo * lda;
          dsoff = 0;
          if constexpr (kGather) {
            // the next tile's source rows, loaded a tile ago (retired by this
            // step's vmcnt(0)): its DMA offsets and scale row
            if (has_nxt) {
              clamp_rows(rs_n, srow_n);
              dma_offsets(goff_n, n_valid_of(nxt), nxt.m_valid, rs_n);
            }
            dsa = sa + srow_n;
          } else {
            dsa = sa_lane_of(nxt);
          }
        }
      }
      const __amdgpu_buffer_rsrc_t rw = buffer_rsrc(dwb), ra = buffer_rsrc(dab);

      constexpr int kDmaSpread = C::TN >= 8 ? C::TN / 2 : 1;   // sub-tile rows that carry DMA issue
      const uint8_t* st = lds + slot * C::kStageBytes;
      const float* sts = reinterpret_cast<const float*>(st + C::kWBytes + C::kABytes) + wm * C::WTM + (lane & 15);
      float sc[C::TM];
      int se[C::TM];
      int sw_e8 = 0;
      if constexpr (kMx) {
        // power-of-two scales: their UE8M0 bytes (the fp32 exponent fields) go
        // to the MX-scaled MFMA, which applies them to the products itself
        sw_e8 = (int)(__float_as_uint(swrow[kb]) >> 23);
#pragma unroll
        for (int tm = 0; tm < C::TM; ++tm) se[tm] = (int)(__float_as_uint(sts[tm * 16]) >> 23);
      } else {
        const float swv = swrow[kb];
#pragma unroll
        for (int tm = 0; tm < C::TM; ++tm) sc[tm] = sts[tm * 16] * swv;
      }

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
            uint32_t off = goff[i];
            if constexpr (kCross) off = last ? goff_n[i] : goff[i];
            lds_dma16(o < C::BN / 8 ? rw : ra, off, dsoff, dslot + o * 1024);
          }
        }
        if (tn == 0 && sdma && refill) lds_dma4(dsa, dslot + C::kWBytes + C::kABytes + wave * 256);
        v8i32 af_next = af;
        if (tn + 1 < C::TN) af_next = lds_frag2(stw + (tn + 1) * 16 * 128, f0, f1);
        if constexpr (kMx) {
          // lane L supplies the scale of its own operand rows: weight row L % 16
          // (one 128-row block per wave: the uniform sw_e8) and token L % 16 of
          // the sub-tile (se), for all four 32-wide K slices of the block
#pragma unroll
          for (int tm = 0; tm < C::TM; ++tm)
            acc[tn][tm] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(af, bf[tm], acc[tn][tm], 0, 0, 0, sw_e8,
                                                                           0, se[tm]);
        } else {
          // all MFMAs of the sub-tile row first (independent results in flight),
          // then their scale FMAs
          v4f32 p[C::TM];
#pragma unroll
          for (int tm = 0; tm < C::TM; ++tm) p[tm] = mfma_fp8_16x16x128(af, bf[tm]);
#pragma unroll
          for (int tm = 0; tm < C::TM; ++tm)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[tn][tm][r] = __builtin_fmaf(p[tm][r], sc[tm], acc[tn][tm][r]);
        }
        af = af_next;
      }
      slot = slot + 1 == S ? 0 : slot + 1;
    }

    // ---- tile end.  The slot of the last K step (slot ^ 1 now; kCross, so
    //      S = 2) is free once every wave is past the barrier below; with kCross
    //      the other holds the next tile's first K block (in flight).  Without
    //      kCross no DMA is in flight and the whole ring is free.
    if constexpr (kPartial) {
      // split-K partial: the fp32 sums, four consecutive n per lane (16 bytes)
#pragma unroll
      for (int tn = 0; tn < C::TN; ++tn) {
        const int nl = wn * C::WTN + tn * 16 + 4 * fg;
#pragma unroll
        for (int tm = 0; tm < C::TM; ++tm) {
          const int ml = wm * C::WTM + tm * 16 + frow;
          if (ml < cur.m_valid && nl < n_valid)
            *reinterpret_cast<v4f32*>(part + (int64_t)(cur.row_lo + ml) * N + cur.n0 + nl) = acc[tn][tm];
        }
      }
    } else {
      // fp32 -> bf16 (RNE), staged in LDS, then full 16-byte chunks of whole
      // output rows with streaming stores.  Direct 8-byte stores from the MFMA
      // layout wrote partial cache lines (1.6x the output bytes reached HBM)
      // and let the output displace the operands in the memory-side cache.
      // Staging layout: rows of BN bf16; 16-byte chunk c of row r (counted
      // within the row group) sits at c ^ (r & 15) (r & 7 for 64-wide tiles), so the 16 rows of one
      // fragment store, and the rows of one read-back wave instruction, spread
      // evenly over the 64 banks.  Row groups of kRows rows fit one slot (or,
      // without kCross, the whole ring).
      constexpr int kRowBytes = C::BN * 2;
      constexpr int kChunks = kRowBytes / 16;
      constexpr int kSpace = kCross ? C::kStageBytes : C::kLdsBytes;
      constexpr int kRowsFit = kSpace / kRowBytes;
      constexpr int kRows = kRowsFit >= C::BM ? C::BM : (kRowsFit / C::WTM) * C::WTM;
      static_assert(kChunks % 8 == 0 && kRows >= C::WTM && C::BM % kRows == 0, "bf16 staging must fit");
      // (64-wide tiles: 8 chunks per row, key r & 7, which keeps the XOR inside the row)
      constexpr int kSwz = kChunks % 16 == 0 ? 15 : 7;
      uint8_t* stage = kCross ? lds + (slot ^ 1) * C::kStageBytes : lds;
#pragma unroll
      for (int g0 = 0; g0 < C::BM; g0 += kRows) {
        lds_barrier();                       // the staging space is free (last K step / previous group)
        if (wm * C::WTM >= g0 && wm * C::WTM < g0 + kRows) {
#pragma unroll
          for (int tn = 0; tn < C::TN; ++tn) {
            const int nl = wn * C::WTN + tn * 16 + 4 * fg;
#pragma unroll
            for (int tm = 0; tm < C::TM; ++tm) {
              const int ml = wm * C::WTM + tm * 16 + frow - g0;
              uint2 o;
              o.x = f32_to_bf16_rne(acc[tn][tm][0]) | (f32_to_bf16_rne(acc[tn][tm][1]) << 16);
              o.y = f32_to_bf16_rne(acc[tn][tm][2]) | (f32_to_bf16_rne(acc[tn][tm][3]) << 16);
              *reinterpret_cast<uint2*>(stage + ml * kRowBytes + (((nl >> 3) ^ (ml & kSwz)) << 4) + ((nl >> 2) & 1) * 8) = o;
            }
          }
        }
        lds_barrier();
        const int c = t % kChunks;             // this thread's chunk of every row it writes
#pragma unroll 4
        for (int r = t / kChunks; r < kRows; r += C::kThreads / kChunks) {
          if (g0 + r < cur.m_valid && c * 8 < n_valid) {
            const uint4 v = *reinterpret_cast<const uint4*>(stage + r * kRowBytes + ((c ^ (r & kSwz)) << 4));
            store_stream16(y + (int64_t)(cur.row_lo + g0 + r) * ldy + cur.n0 + c * 8, v);
          }
        }
      }
    }

    if constexpr (!kCross) {
      break;                                   // one tile per workgroup
    } else {
      // (the next step's top barrier orders the staging reads before the slot is refilled)
      if (!has_nxt) break;
      cur = nxt;
#pragma unroll
      for (int i = 0; i < C::kLoadsPerWave; ++i) goff[i] = goff_n[i];
      has_nxt = jobs.next(nxt);
      if constexpr (kGather) {
        srow_c = srow_n;
        if (has_nxt) load_rows(nxt, rs_n, srow_n);
      } else {
        if (has_nxt) dma_offsets(goff_n, n_valid_of(nxt), nxt.m_valid, rs_n);
      }
    }
  }
  // (the last step of the last tile issued no DMA: nothing is in flight here)
}

}  // namespace fp8rl
