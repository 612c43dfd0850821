// Internal launchers behind the C ABI (include/fp8rl.h).  Arguments are
// validated by the API layer before any of these is called; each launcher only
// picks a grid and enqueues its kernel(s) on `stream`.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fp8rl {

// pow2_scale: power-of-two (UE8M0) block scales instead of fl32(amax / 448)
hipError_t launch_quant_weight_block128(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                                        uint8_t* q, int64_t ldq, float* scale, hipStream_t stream,
                                        bool pow2_scale);

// Several weight matrices in one launch (at most kWeightBatchJobs, each already
// validated like a single call; jobs with no blocks are skipped).  The total
// block count must stay below 2^31.
constexpr int kWeightBatchJobs = 64;
struct WeightJob {
  const uint16_t* w;
  int64_t n, k, ldw;
  uint8_t* q;
  int64_t ldq;
  float* scale;
};
hipError_t launch_quant_weight_block128_batched(const WeightJob* jobs, int count, hipStream_t stream);

hipError_t launch_quant_act_token_group128(const uint16_t* a, int64_t m, int64_t k, int64_t lda,
                                           uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                           hipStream_t stream, bool pow2_scale);

hipError_t launch_silu_mul_quant_group128(const uint16_t* gu, int64_t m, int64_t inter, int64_t ld_gu,
                                          uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                          uint16_t* h, int64_t ldh, hipStream_t stream);

hipError_t launch_gather_rows_fp8(const uint8_t* q_src, int64_t ldq_src, const float* s_src, int64_t ld_s_src,
                                  const int32_t* index, int64_t src_rows, int64_t rows, int64_t k,
                                  uint8_t* q_dst, int64_t ldq_dst, float* s_dst, int64_t ld_s_dst,
                                  hipStream_t stream);

// pow2_scales: every scale is a power of two 2^-127 .. 2^127 (only the fp32
// exponent fields are read; the MX-scaled MFMA applies them)
hipError_t launch_gemm_w8a8_block(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                  const uint8_t* qw, int64_t ldw, const float* sw,
                                  uint16_t* y, int64_t ldy, int64_t m, int64_t n, int64_t k,
                                  hipStream_t stream, bool pow2_scales);

// Split-K factor the dense GEMM uses for this shape (1: no split); the
// workspace it needs is splits * m * n fp32 values.
int splitk_factor(int64_t m, int64_t n, int64_t k);

hipError_t launch_gemm_w8a8_block_splitk(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                         const uint8_t* qw, int64_t ldw, const float* sw, uint16_t* y,
                                         int64_t ldy, int64_t m, int64_t n, int64_t k, float* part, int splits,
                                         hipStream_t stream);

// Device address, on the current device, of the library's static split-K
// scratch (kSplitKScratchBytes); fetched once per device, no allocation.  The
// split rule keeps splits * m * n <= 256 * 128 * 128 floats, so every split
// shape fits.
constexpr int64_t kSplitKScratchBytes = int64_t(16) << 20;
hipError_t splitk_scratch(float** out);

hipError_t launch_grouped_gemm_w8a8_block(const uint8_t* qa, const float* sa, int64_t ld_sa,
                                          const uint8_t* qw, const float* sw,
                                          const int32_t* group_offsets, int64_t num_groups,
                                          int64_t total_rows, uint16_t* y, int64_t n, int64_t k,
                                          hipStream_t stream, bool pow2_scales);

// The grouped GEMM over gathered rows: output row r uses activation row
// row_index[r] of qa [src_rows][lda] and of sa [K/128][ld_sa] (indices clamped
// into range); src_rows * lda < 2^32.
hipError_t launch_grouped_gemm_w8a8_block_gathered(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                                   int64_t src_rows, const int32_t* row_index, const uint8_t* qw,
                                                   const float* sw, const int32_t* group_offsets, int64_t num_groups,
                                                   int64_t total_rows, uint16_t* y, int64_t n, int64_t k,
                                                   hipStream_t stream);

// Token-level TIS weights and mismatch-KL sums: workgroups of the first pass
// (each leaves 4 doubles of partial sums in `partial`), then one that adds them.
int tis_blocks(int64_t n);

hipError_t launch_tis_weights_kl(const float* logp_train, const float* logp_rollout, const uint8_t* mask, int64_t n,
                                 float clip_c, float* w_tis, double* stats, double* partial, hipStream_t stream);

// FP8 KV cache: per-tensor scale calibration (workgroup maxima in `partial`,
// kv_amax_blocks(n) words), quantised writes into the paged cache, and decode
// attention over it (fp8_cache false: the same kernel over a bf16 cache).
int kv_amax_blocks(int64_t n);

hipError_t launch_kv_calibrate_scale(const uint16_t* x, int64_t n, float* scale, uint32_t* partial,
                                     hipStream_t stream);

hipError_t launch_kv_cache_write(const uint16_t* k, const uint16_t* v, int64_t tokens, int kv_heads,
                                 const int64_t* slots, int64_t num_blocks, const float* k_scale, const float* v_scale,
                                 uint8_t* k_cache, uint8_t* v_cache, hipStream_t stream);

struct AttnSplit {
  int split_tokens;      // tokens per wave (a multiple of 16)
  int max_splits;        // splits of the longest sequence
  int partial_floats;    // floats per (sequence, kv head, split) record
};
AttnSplit attn_decode_split(int64_t batch, int64_t kv_heads, int64_t group, int64_t max_seq_len);

hipError_t launch_attention_decode(const uint16_t* q, const void* k_cache, const void* v_cache, bool fp8_cache,
                                   int64_t num_blocks, const int32_t* block_table, int64_t max_blocks,
                                   const int32_t* seq_lens, int64_t batch, int64_t q_heads, int64_t kv_heads,
                                   int64_t max_seq_len, const float* k_scale, const float* v_scale, float sm_scale,
                                   uint16_t* out, float* partial, hipStream_t stream);

}  // namespace fp8rl
