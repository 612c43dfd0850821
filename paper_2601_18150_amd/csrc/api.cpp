// C ABI of libfp8rl (declared in include/fp8rl.h): argument validation, then
// launches on the caller's stream.  No allocation, no synchronisation, no
// state kept between calls.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8rl.h"
#include "launch.hpp"

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 31;   // per-dimension limit (32-bit tile indices)
constexpr int64_t kMaxLd = int64_t(1) << 24;     // GEMM operand row pitch limit (32-bit in-tile DMA offsets)

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int hip_status(hipError_t e) { return e == hipSuccess ? FP8RL_OK : FP8RL_ERR_HIP; }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// Validation shared by the dense GEMM entry points: an FP8RL_* error, FP8RL_OK for
// a valid call with nothing to do, or kLaunch.
constexpr int kLaunch = -1;

int check_dense(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa, const uint8_t* qw, int64_t ldw,
                const float* sw, const uint16_t* y, int64_t ldy, int64_t m, int64_t n, int64_t k) {
  if (m < 0 || n < 0 || k < 0) return FP8RL_ERR_INVALID_ARG;
  if (n % 128 || k % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (m >= kMaxDim || n >= kMaxDim || k >= kMaxDim) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (((m + 127) / 128) * (n / 128) >= (int64_t(1) << 30)) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (m == 0 || n == 0) return FP8RL_OK;
  if (!qa || !sa || !qw || !sw || !y) return FP8RL_ERR_INVALID_ARG;
  if (k == 0) return FP8RL_ERR_UNSUPPORTED_SHAPE;   // an empty reduction is not a blockwise GEMM
  if (lda < k || ldw < k || ldy < n || ld_sa < m) return FP8RL_ERR_INVALID_ARG;
  if (lda >= kMaxLd || ldw >= kMaxLd) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (!aligned(qa, 16) || !aligned(qw, 16) || !aligned(y, 16) || !aligned(sa, 4) || !aligned(sw, 4) ||
      lda % 16 || ldw % 16 || ldy % 8)
    return FP8RL_ERR_MISALIGNED;
  return kLaunch;
}

}  // namespace

extern "C" {

const char* fp8rl_status_string(int status) {
  switch (status) {
    case FP8RL_OK: return "FP8RL_OK";
    case FP8RL_ERR_INVALID_ARG: return "FP8RL_ERR_INVALID_ARG";
    case FP8RL_ERR_UNSUPPORTED_SHAPE: return "FP8RL_ERR_UNSUPPORTED_SHAPE";
    case FP8RL_ERR_MISALIGNED: return "FP8RL_ERR_MISALIGNED";
    case FP8RL_ERR_HIP: return "FP8RL_ERR_HIP";
    case FP8RL_ERR_SCRATCH_LIMIT: return "FP8RL_ERR_SCRATCH_LIMIT";
    default: return "FP8RL_ERR_UNKNOWN";
  }
}

int fp8rl_version(void) { return 100; }   // 0.1.0

// Validation of one weight matrix: an FP8RL_* error, FP8RL_OK (nothing to do) or kLaunch.
static int check_weight(const uint16_t* w, int64_t n, int64_t k, int64_t ldw, const uint8_t* q, int64_t ldq,
                        const float* scale) {
  if (n < 0 || k < 0) return FP8RL_ERR_INVALID_ARG;
  if (n % 128 || k % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (n >= kMaxDim || k >= kMaxDim || (n / 128) * (k / 128) >= (int64_t(1) << 24))
    return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (n == 0 || k == 0) return FP8RL_OK;
  if (!w || !q || !scale) return FP8RL_ERR_INVALID_ARG;
  if (ldw < k || ldq < k) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(w, 16) || !aligned(q, 16) || !aligned(scale, 4) || ldw % 8 || ldq % 16)
    return FP8RL_ERR_MISALIGNED;
  return kLaunch;
}

static int quant_weight(const uint16_t* w, int64_t n, int64_t k, int64_t ldw, uint8_t* q, int64_t ldq,
                        float* scale, void* stream, bool pow2) {
  const int st = check_weight(w, n, k, ldw, q, ldq, scale);
  if (st != kLaunch) return st;
  return hip_status(fp8rl::launch_quant_weight_block128(w, n, k, ldw, q, ldq, scale, as_stream(stream), pow2));
}

int fp8rl_quant_weight_block128_batched(const fp8rl_weight_job* jobs, int64_t count, void* stream) {
  if (count < 0 || (count > 0 && !jobs)) return FP8RL_ERR_INVALID_ARG;
  for (int64_t i = 0; i < count; ++i) {
    const fp8rl_weight_job& j = jobs[i];
    const int st = check_weight(j.w, j.n, j.k, j.ldw, j.q, j.ldq, j.scale);
    if (st != kLaunch && st != FP8RL_OK) return st;
  }
  fp8rl::WeightJob chunk[fp8rl::kWeightBatchJobs];
  for (int64_t i0 = 0; i0 < count; i0 += fp8rl::kWeightBatchJobs) {
    const int c = (int)(count - i0 < fp8rl::kWeightBatchJobs ? count - i0 : fp8rl::kWeightBatchJobs);
    for (int i = 0; i < c; ++i) {
      const fp8rl_weight_job& j = jobs[i0 + i];
      chunk[i] = fp8rl::WeightJob{j.w, j.n, j.k, j.ldw, j.q, j.ldq, j.scale};
    }
    const int st = hip_status(fp8rl::launch_quant_weight_block128_batched(chunk, c, as_stream(stream)));
    if (st != FP8RL_OK) return st;
  }
  return FP8RL_OK;
}

int fp8rl_quant_weight_block128(const uint16_t* w, int64_t n, int64_t k, int64_t ldw, uint8_t* q,
                                int64_t ldq, float* scale, void* stream) {
  return quant_weight(w, n, k, ldw, q, ldq, scale, stream, false);
}

int fp8rl_quant_weight_block128_ue8m0(const uint16_t* w, int64_t n, int64_t k, int64_t ldw, uint8_t* q,
                                      int64_t ldq, float* scale, void* stream) {
  return quant_weight(w, n, k, ldw, q, ldq, scale, stream, true);
}

static int quant_act(const uint16_t* a, int64_t m, int64_t k, int64_t lda, uint8_t* q, int64_t ldq, float* scale,
                     int64_t ld_scale, void* stream, bool pow2) {
  if (m < 0 || k < 0) return FP8RL_ERR_INVALID_ARG;
  if (k % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (m >= kMaxDim || k >= kMaxDim || m * (k / 128) >= (int64_t(1) << 28)) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (m == 0 || k == 0) return FP8RL_OK;
  if (!a || !q || !scale) return FP8RL_ERR_INVALID_ARG;
  if (lda < k || ldq < k || ld_scale < m) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(a, 16) || !aligned(q, 16) || !aligned(scale, 4) || lda % 8 || ldq % 16)
    return FP8RL_ERR_MISALIGNED;
  return hip_status(
      fp8rl::launch_quant_act_token_group128(a, m, k, lda, q, ldq, scale, ld_scale, as_stream(stream), pow2));
}

int fp8rl_quant_act_token_group128(const uint16_t* a, int64_t m, int64_t k, int64_t lda, uint8_t* q,
                                   int64_t ldq, float* scale, int64_t ld_scale, void* stream) {
  return quant_act(a, m, k, lda, q, ldq, scale, ld_scale, stream, false);
}

int fp8rl_quant_act_token_group128_ue8m0(const uint16_t* a, int64_t m, int64_t k, int64_t lda, uint8_t* q,
                                         int64_t ldq, float* scale, int64_t ld_scale, void* stream) {
  return quant_act(a, m, k, lda, q, ldq, scale, ld_scale, stream, true);
}

int fp8rl_silu_mul_quant_group128(const uint16_t* gu, int64_t m, int64_t inter, int64_t ld_gu, uint8_t* q,
                                  int64_t ldq, float* scale, int64_t ld_scale, uint16_t* h, int64_t ldh,
                                  void* stream) {
  if (m < 0 || inter < 0) return FP8RL_ERR_INVALID_ARG;
  if (inter % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (m >= kMaxDim || 2 * inter >= kMaxDim || m * (inter / 128) >= (int64_t(1) << 28))
    return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (m == 0 || inter == 0) return FP8RL_OK;
  if (!gu || !q || !scale) return FP8RL_ERR_INVALID_ARG;
  if (ld_gu < 2 * inter || ldq < inter || ld_scale < m || (h && ldh < inter)) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(gu, 16) || !aligned(q, 16) || !aligned(scale, 4) || ld_gu % 8 || ldq % 16) return FP8RL_ERR_MISALIGNED;
  if (h && (!aligned(h, 16) || ldh % 8)) return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_silu_mul_quant_group128(gu, m, inter, ld_gu, q, ldq, scale, ld_scale, h,
                                                          h ? ldh : 0, as_stream(stream)));
}

int fp8rl_gather_rows_fp8(const uint8_t* q_src, int64_t ldq_src, const float* s_src, int64_t ld_s_src,
                          int64_t src_rows, const int32_t* index, int64_t rows, int64_t k, uint8_t* q_dst,
                          int64_t ldq_dst, float* s_dst, int64_t ld_s_dst, void* stream) {
  if (rows < 0 || k < 0 || src_rows < 0) return FP8RL_ERR_INVALID_ARG;
  if (k % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (rows >= kMaxDim || src_rows >= kMaxDim || k >= kMaxDim || rows * (k / 16) >= (int64_t(1) << 31))
    return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (rows == 0 || k == 0) return FP8RL_OK;
  if (src_rows == 0 || !q_src || !s_src || !index || !q_dst || !s_dst) return FP8RL_ERR_INVALID_ARG;
  if (ldq_src < k || ldq_dst < k || ld_s_src < src_rows || ld_s_dst < rows) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(q_src, 16) || !aligned(q_dst, 16) || ldq_src % 16 || ldq_dst % 16 || !aligned(s_src, 4) ||
      !aligned(s_dst, 4) || !aligned(index, 4))
    return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_gather_rows_fp8(q_src, ldq_src, s_src, ld_s_src, index, src_rows, rows, k, q_dst,
                                                  ldq_dst, s_dst, ld_s_dst, as_stream(stream)));
}

int fp8rl_gemm_w8a8_block(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa, const uint8_t* qw,
                          int64_t ldw, const float* sw, uint16_t* y, int64_t ldy, int64_t m, int64_t n,
                          int64_t k, void* stream) {
  const int st = check_dense(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k);
  if (st != kLaunch) return st;
  return hip_status(
      fp8rl::launch_gemm_w8a8_block(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, as_stream(stream), false));
}

int fp8rl_gemm_w8a8_block_ue8m0(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                const uint8_t* qw, int64_t ldw, const float* sw, uint16_t* y, int64_t ldy,
                                int64_t m, int64_t n, int64_t k, void* stream) {
  const int st = check_dense(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k);
  if (st != kLaunch) return st;
  return hip_status(
      fp8rl::launch_gemm_w8a8_block(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, as_stream(stream), true));
}

int64_t fp8rl_gemm_w8a8_block_workspace_size(int64_t m, int64_t n, int64_t k) {
  if (m <= 0 || n <= 0 || k <= 0 || n % 128 || k % 128 || m >= kMaxDim || n >= kMaxDim || k >= kMaxDim) return 0;
  const int splits = fp8rl::splitk_factor(m, n, k);
  return splits > 1 ? int64_t(splits) * m * n * 4 : 0;
}

int fp8rl_gemm_w8a8_block_ws(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa, const uint8_t* qw,
                             int64_t ldw, const float* sw, uint16_t* y, int64_t ldy, int64_t m, int64_t n,
                             int64_t k, void* workspace, int64_t workspace_bytes, void* stream) {
  const int st = check_dense(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k);
  if (st != kLaunch) return st;
  if (workspace_bytes < 0 || (workspace_bytes > 0 && !workspace)) return FP8RL_ERR_INVALID_ARG;
  if (workspace_bytes > 0 && !aligned(workspace, 16)) return FP8RL_ERR_MISALIGNED;
  const int splits = fp8rl::splitk_factor(m, n, k);
  if (splits > 1 && workspace_bytes >= int64_t(splits) * m * n * 4)
    return hip_status(fp8rl::launch_gemm_w8a8_block_splitk(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k,
                                                           static_cast<float*>(workspace), splits,
                                                           as_stream(stream)));
  return hip_status(
      fp8rl::launch_gemm_w8a8_block(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, as_stream(stream), false));
}

static_assert(FP8RL_SPLITK_SCRATCH_BYTES == fp8rl::kSplitKScratchBytes, "header and library scratch sizes differ");

int fp8rl_gemm_w8a8_block_noalloc(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa, const uint8_t* qw,
                                  int64_t ldw, const float* sw, uint16_t* y, int64_t ldy, int64_t m, int64_t n,
                                  int64_t k, void* stream) {
  const int st = check_dense(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k);
  if (st != kLaunch) return st;
  const int splits = fp8rl::splitk_factor(m, n, k);
  if (splits > 1) {
    if (int64_t(splits) * m * n * 4 > fp8rl::kSplitKScratchBytes) return FP8RL_ERR_SCRATCH_LIMIT;
    float* part = nullptr;
    if (fp8rl::splitk_scratch(&part) != hipSuccess) return FP8RL_ERR_HIP;
    return hip_status(fp8rl::launch_gemm_w8a8_block_splitk(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, part,
                                                           splits, as_stream(stream)));
  }
  return hip_status(
      fp8rl::launch_gemm_w8a8_block(qa, lda, sa, ld_sa, qw, ldw, sw, y, ldy, m, n, k, as_stream(stream), false));
}

static int grouped(const uint8_t* qa, const float* sa, int64_t ld_sa, const uint8_t* qw, const float* sw,
                   const int32_t* group_offsets, int64_t num_groups, int64_t total_rows, uint16_t* y, int64_t n,
                   int64_t k, void* stream, bool pow2);

int fp8rl_grouped_gemm_w8a8_block(const uint8_t* qa, const float* sa, int64_t ld_sa, const uint8_t* qw,
                                  const float* sw, const int32_t* group_offsets, int64_t num_groups,
                                  int64_t total_rows, uint16_t* y, int64_t n, int64_t k, void* stream) {
  return grouped(qa, sa, ld_sa, qw, sw, group_offsets, num_groups, total_rows, y, n, k, stream, false);
}

int fp8rl_grouped_gemm_w8a8_block_ue8m0(const uint8_t* qa, const float* sa, int64_t ld_sa, const uint8_t* qw,
                                        const float* sw, const int32_t* group_offsets, int64_t num_groups,
                                        int64_t total_rows, uint16_t* y, int64_t n, int64_t k, void* stream) {
  return grouped(qa, sa, ld_sa, qw, sw, group_offsets, num_groups, total_rows, y, n, k, stream, true);
}

int fp8rl_grouped_gemm_w8a8_block_gathered(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                           int64_t src_rows, const int32_t* row_index, const uint8_t* qw,
                                           const float* sw, const int32_t* group_offsets, int64_t num_groups,
                                           int64_t total_rows, uint16_t* y, int64_t n, int64_t k, void* stream) {
  if (total_rows < 0 || n < 0 || k < 0 || src_rows < 0) return FP8RL_ERR_INVALID_ARG;
  if (num_groups < 1) return FP8RL_ERR_INVALID_ARG;
  if (n % 128 || k % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (total_rows >= kMaxDim || n >= kMaxDim || k >= kMaxLd || num_groups > 1024 || src_rows >= kMaxDim ||
      (total_rows / 128 + num_groups) * (n / 128) >= (int64_t(1) << 31))
    return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (total_rows == 0 || n == 0) return FP8RL_OK;
  if (!qa || !sa || !qw || !sw || !group_offsets || !y || !row_index || src_rows == 0) return FP8RL_ERR_INVALID_ARG;
  if (k == 0) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (lda < k || ld_sa < src_rows) return FP8RL_ERR_INVALID_ARG;
  if (src_rows * lda >= (int64_t(1) << 32)) return FP8RL_ERR_UNSUPPORTED_SHAPE;   // 32-bit DMA offsets
  if (!aligned(qa, 16) || !aligned(qw, 16) || !aligned(y, 16) || !aligned(sa, 4) || !aligned(sw, 4) ||
      !aligned(group_offsets, 4) || !aligned(row_index, 4) || lda % 16)
    return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_grouped_gemm_w8a8_block_gathered(qa, lda, sa, ld_sa, src_rows, row_index, qw, sw,
                                                                   group_offsets, num_groups, total_rows, y, n, k,
                                                                   as_stream(stream)));
}

static int grouped(const uint8_t* qa, const float* sa, int64_t ld_sa, const uint8_t* qw, const float* sw,
                   const int32_t* group_offsets, int64_t num_groups, int64_t total_rows, uint16_t* y, int64_t n,
                   int64_t k, void* stream, bool pow2) {
  if (total_rows < 0 || n < 0 || k < 0) return FP8RL_ERR_INVALID_ARG;
  if (num_groups < 1) return FP8RL_ERR_INVALID_ARG;
  if (n % 128 || k % 128) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (total_rows >= kMaxDim || n >= kMaxDim || k >= kMaxLd || num_groups > 1024 ||
      (total_rows / 128 + num_groups) * (n / 128) >= (int64_t(1) << 31))
    return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (total_rows == 0 || n == 0) return FP8RL_OK;
  if (!qa || !sa || !qw || !sw || !group_offsets || !y) return FP8RL_ERR_INVALID_ARG;
  if (k == 0) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (ld_sa < total_rows) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(qa, 16) || !aligned(qw, 16) || !aligned(y, 16) || !aligned(sa, 4) || !aligned(sw, 4) ||
      !aligned(group_offsets, 4))
    return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_grouped_gemm_w8a8_block(qa, sa, ld_sa, qw, sw, group_offsets, num_groups,
                                                          total_rows, y, n, k, as_stream(stream), pow2));
}

int64_t fp8rl_tis_workspace_size(int64_t n) {
  if (n < 0) return 0;
  return int64_t(fp8rl::tis_blocks(n)) * 4 * int64_t(sizeof(double));
}

int fp8rl_tis_weights_kl(const float* logp_train, const float* logp_rollout, const uint8_t* mask, int64_t n,
                         float clip_c, float* w_tis, double* stats, void* workspace, int64_t workspace_bytes,
                         void* stream) {
  if (n < 0 || !(clip_c > 0.0f) || !(clip_c <= 3.4028234663852886e38f)) return FP8RL_ERR_INVALID_ARG;
  if (n >= (int64_t(1) << 48)) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (!stats || !workspace) return FP8RL_ERR_INVALID_ARG;
  if (n > 0 && (!logp_train || !logp_rollout || !w_tis)) return FP8RL_ERR_INVALID_ARG;
  if (workspace_bytes < fp8rl_tis_workspace_size(n)) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(logp_train, 16) || !aligned(logp_rollout, 16) || !aligned(w_tis, 16) || !aligned(mask, 4) ||
      !aligned(stats, 8) || !aligned(workspace, 8))
    return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_tis_weights_kl(logp_train, logp_rollout, mask, n, clip_c, w_tis, stats,
                                                 static_cast<double*>(workspace), as_stream(stream)));
}

int64_t fp8rl_kv_calibrate_workspace_size(int64_t n) {
  return n < 0 ? 0 : int64_t(fp8rl::kv_amax_blocks(n)) * 4;
}

int fp8rl_kv_calibrate_scale(const uint16_t* x, int64_t n, float* scale, void* workspace, int64_t workspace_bytes,
                             void* stream) {
  if (n < 0 || !scale || !workspace || (n > 0 && !x)) return FP8RL_ERR_INVALID_ARG;
  if (n >= (int64_t(1) << 46)) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (workspace_bytes < fp8rl_kv_calibrate_workspace_size(n)) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(scale, 4) || !aligned(workspace, 4)) return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_kv_calibrate_scale(x, n, scale, static_cast<uint32_t*>(workspace),
                                                     as_stream(stream)));
}

int fp8rl_kv_cache_write_fp8(const uint16_t* k, const uint16_t* v, int64_t tokens, int64_t kv_heads,
                             int64_t head_dim, const int64_t* slot_mapping, int64_t num_blocks, const float* k_scale,
                             const float* v_scale, uint8_t* k_cache, uint8_t* v_cache, void* stream) {
  if (tokens < 0 || kv_heads < 1 || num_blocks < 0) return FP8RL_ERR_INVALID_ARG;
  if (head_dim != 128 || kv_heads > 1024 || tokens >= (int64_t(1) << 31) ||
      (tokens + 3) / 4 * kv_heads * 16 >= (int64_t(1) << 31))
    return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (tokens == 0) return FP8RL_OK;
  if (!k || !v || !slot_mapping || !k_scale || !v_scale || !k_cache || !v_cache) return FP8RL_ERR_INVALID_ARG;
  if (!aligned(k, 16) || !aligned(v, 16) || !aligned(k_cache, 8) || !aligned(v_cache, 8) || !aligned(slot_mapping, 8) ||
      !aligned(k_scale, 4) || !aligned(v_scale, 4))
    return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_kv_cache_write(k, v, tokens, (int)kv_heads, slot_mapping, num_blocks, k_scale,
                                                 v_scale, k_cache, v_cache, as_stream(stream)));
}

int64_t fp8rl_attention_decode_workspace_size(int64_t batch, int64_t q_heads, int64_t kv_heads,
                                              int64_t max_seq_len) {
  if (batch < 0 || kv_heads < 1 || q_heads < kv_heads || q_heads % kv_heads || max_seq_len < 0) return 0;
  const fp8rl::AttnSplit sp = fp8rl::attn_decode_split(batch, kv_heads, q_heads / kv_heads, max_seq_len);
  return batch * kv_heads * int64_t(sp.max_splits) * sp.partial_floats * 4;
}

static int attention_decode(const uint16_t* q, const void* k_cache, const void* v_cache, bool fp8, int64_t num_blocks,
                            const int32_t* block_table, int64_t max_blocks, const int32_t* seq_lens, int64_t batch,
                            int64_t q_heads, int64_t kv_heads, int64_t head_dim, int64_t max_seq_len,
                            const float* k_scale, const float* v_scale, float sm_scale, uint16_t* out,
                            void* workspace, int64_t workspace_bytes, void* stream) {
  if (batch < 0 || kv_heads < 1 || q_heads < 1 || max_seq_len < 0 || max_blocks < 0 || num_blocks < 0)
    return FP8RL_ERR_INVALID_ARG;
  if (!(sm_scale > 0.0f) || !(sm_scale <= 3.4028234663852886e38f)) return FP8RL_ERR_INVALID_ARG;
  if (head_dim != 128 || q_heads % kv_heads) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  const int64_t group = q_heads / kv_heads;
  if (group != 1 && group != 2 && group != 4 && group != 8) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (batch > 65535 || kv_heads > 65535 || max_seq_len >= (int64_t(1) << 30)) return FP8RL_ERR_UNSUPPORTED_SHAPE;
  if (batch == 0) return FP8RL_OK;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !out || !workspace) return FP8RL_ERR_INVALID_ARG;
  if (fp8 && (!k_scale || !v_scale)) return FP8RL_ERR_INVALID_ARG;
  if (num_blocks < 1 || max_blocks < 1 || max_blocks * 16 < max_seq_len) return FP8RL_ERR_INVALID_ARG;
  if (workspace_bytes < fp8rl_attention_decode_workspace_size(batch, q_heads, kv_heads, max_seq_len))
    return FP8RL_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(block_table, 4) ||
      !aligned(seq_lens, 4) || !aligned(out, 4) || !aligned(workspace, 16) || !aligned(k_scale, 4) ||
      !aligned(v_scale, 4))
    return FP8RL_ERR_MISALIGNED;
  return hip_status(fp8rl::launch_attention_decode(q, k_cache, v_cache, fp8, num_blocks, block_table, max_blocks,
                                                   seq_lens, batch, q_heads, kv_heads, max_seq_len, k_scale, v_scale,
                                                   sm_scale, out, static_cast<float*>(workspace), as_stream(stream)));
}

int fp8rl_attention_decode_fp8kv(const uint16_t* q, const uint8_t* k_cache, const uint8_t* v_cache, int64_t num_blocks,
                                 const int32_t* block_table, int64_t max_blocks, const int32_t* seq_lens,
                                 int64_t batch, int64_t q_heads, int64_t kv_heads, int64_t head_dim,
                                 int64_t max_seq_len, const float* k_scale, const float* v_scale, float sm_scale,
                                 uint16_t* out, void* workspace, int64_t workspace_bytes, void* stream) {
  return attention_decode(q, k_cache, v_cache, true, num_blocks, block_table, max_blocks, seq_lens, batch, q_heads,
                          kv_heads, head_dim, max_seq_len, k_scale, v_scale, sm_scale, out, workspace,
                          workspace_bytes, stream);
}

int fp8rl_attention_decode_bf16kv(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                  int64_t num_blocks, const int32_t* block_table, int64_t max_blocks,
                                  const int32_t* seq_lens, int64_t batch, int64_t q_heads, int64_t kv_heads,
                                  int64_t head_dim, int64_t max_seq_len, float sm_scale, uint16_t* out,
                                  void* workspace, int64_t workspace_bytes, void* stream) {
  return attention_decode(q, k_cache, v_cache, false, num_blocks, block_table, max_blocks, seq_lens, batch, q_heads,
                          kv_heads, head_dim, max_seq_len, nullptr, nullptr, sm_scale, out, workspace,
                          workspace_bytes, stream);
}

}  // extern "C"
