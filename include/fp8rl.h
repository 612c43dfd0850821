/*
 * fp8rl -- blockwise FP8 (OCP E4M3) W8A8 linear layer for AMD MI355X (gfx950).
 *
 * The operations follow the FP8 rollout method of "FP8-RL" (arXiv 2601.18150):
 *   - weights are quantised to E4M3 with one fp32 scale per 128x128 block,
 *     re-run after every RL step when the trainer's bf16 weights are synced
 *     into the rollout engine (section 2.1.1, Eq. (1); section 2.1.2);
 *   - activations are quantised dynamically at every forward pass with one
 *     fp32 scale per token and 128-wide group along K (section 2.1.1 "Static vs
 *     dynamic quantization"; section 3.1 "1x128 tiles for activations");
 *   - the linear layer is an FP8 GEMM consuming both, accumulating in fp32 and
 *     writing bf16, dense or grouped per MoE expert (section 2.1.1
 *     "Quantization scope", section 2.1.4).
 *
 * Conventions shared by every entry point
 *   - All data pointers are DEVICE pointers (memory of the current HIP device)
 *     owned by the caller.  The library allocates no memory, never
 *     synchronises, keeps no state between calls, and only enqueues kernels on
 *     `stream` (a hipStream_t; NULL = the default stream).  Calls are
 *     asynchronous: a device fault surfaces at the caller's next sync.
 *   - bf16 values are passed as their uint16_t bit patterns, E4M3 values as
 *     uint8_t codes (OCP E4M3 "fn": bias 7, max 448, 0x7F/0xFF NaN, no inf).
 *   - Matrices are row-major; ld* is the distance in ELEMENTS between rows.
 *   - Outputs must not alias inputs.
 *   - Return value: FP8RL_OK or an error code.  On any error nothing is
 *     launched and no output is touched.
 *   - Size 0 along M (or total_rows) is a valid no-op returning FP8RL_OK.
 *   - Inputs must be finite (no NaN/inf); for non-finite inputs the outputs are
 *     unspecified (not checked: it would need a device read).
 *
 * Quantisation rule (identical for weight blocks and activation groups):
 *   amax  = max |x| over the block/group (bf16 widened exactly to fp32)
 *   scale = amax / 448 as an IEEE fp32 division (round to nearest even,
 *           subnormals kept); scale = 1.0 when amax == 0
 *   code  = E4M3(fl32(x / scale)) -- one IEEE fp32 division, then one
 *           round-to-nearest-even onto the E4M3 grid, saturating at +-448,
 *           keeping the sign of x (so -0 gives 0x80).
 *   Every block/group's largest element therefore maps to +-448 exactly.
 *   Codes and scales are bit-for-bit deterministic.
 */
#ifndef FP8RL_H
#define FP8RL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FP8RL_OK = 0,
  FP8RL_ERR_INVALID_ARG = 1,       /* null pointer with nonzero size, negative size, ld too small, num_groups < 1 */
  FP8RL_ERR_UNSUPPORTED_SHAPE = 2, /* K or N not a multiple of 128, or a size beyond 2^31 elements per row/col */
  FP8RL_ERR_MISALIGNED = 3,        /* a pointer or leading dimension breaks the alignment rules stated below */
  FP8RL_ERR_HIP = 4,               /* the HIP runtime reported an error at launch */
  FP8RL_ERR_SCRATCH_LIMIT = 5      /* the call needs more than the library's static scratch (no-allocation entry point) */
} fp8rl_status;

/*
 * Weight quantisation, one fp32 scale per 128x128 block (section 2.1.1, Eq. (1)).
 *
 * w      [n][ldw]  bf16 weight, nn.Linear layout: n output rows, k input columns
 * q      [n][ldq]  E4M3 codes out
 * scale  [n/128][k/128] fp32 out, contiguous; scale[i*(k/128)+j] belongs to
 *        rows 128i..128i+127, columns 128j..128j+127
 * n, k   multiples of 128 (else FP8RL_ERR_UNSUPPORTED_SHAPE); n == 0 is a no-op
 * Alignment: w, q 16-byte aligned; ldw % 8 == 0; ldq % 16 == 0; scale 4-byte aligned.
 * ldw >= k, ldq >= k (else FP8RL_ERR_INVALID_ARG).
 */
int fp8rl_quant_weight_block128(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                                uint8_t* q, int64_t ldq, float* scale, void* stream);

/*
 * Weight re-quantisation of many matrices in one pass.  After every RL step the
 * trainer's updated bf16 weights are synced into the rollout engine and every
 * quantised linear layer is re-quantised (section 2.1.2; section 2.1.1 Eq. (1)).
 * For each jobs[i] this computes exactly what
 *   fp8rl_quant_weight_block128(w, n, k, ldw, q, ldq, scale, stream)
 * computes (same layouts, alignment and size rules, bit-identical codes and
 * scales), with up to 64 matrices per kernel launch, so the memory pipeline stays
 * full across matrices instead of ramping up and draining once per matrix.
 *
 * jobs   HOST array of `count` job descriptors, read during the call only; the
 *        pointers inside are device pointers.  Jobs with n == 0 or k == 0 are
 *        skipped.  No job's outputs may overlap another job's inputs or outputs.
 * count  >= 0 (0 is a no-op); jobs may be NULL only when count == 0.
 * Errors: every job is validated before anything is launched; the first invalid
 * job's error code is returned (FP8RL_ERR_INVALID_ARG also for count < 0 or a
 * NULL jobs array).  FP8RL_ERR_HIP after a launch failure: launches of earlier
 * 64-job chunks may then have run.
 */
typedef struct fp8rl_weight_job {
  const uint16_t* w;     /* [n][ldw] bf16 weight */
  int64_t n, k, ldw;
  uint8_t* q;            /* [n][ldq] E4M3 codes out */
  int64_t ldq;
  float* scale;          /* [n/128][k/128] fp32 block scales out */
} fp8rl_weight_job;

int fp8rl_quant_weight_block128_batched(const fp8rl_weight_job* jobs, int64_t count, void* stream);

/*
 * Dynamic activation quantisation, one fp32 scale per token per 128-wide K group
 * (section 2.1.1 "Static vs dynamic quantization"; section 3.1 1x128 tiles).
 *
 * a      [m][lda]  bf16 activations (m tokens, k features)
 * q      [m][ldq]  E4M3 codes out
 * scale  [k/128][ld_scale] fp32 out, token index contiguous:
 *        scale[g*ld_scale + t] belongs to token t, columns 128g..128g+127.
 *        Entries t >= m are not written.
 * k      multiple of 128; m >= 0 arbitrary (m == 0 is a no-op)
 * Alignment: a, q 16-byte aligned; lda % 8 == 0; ldq % 16 == 0; scale 4-byte aligned.
 * lda >= k, ldq >= k, ld_scale >= m.
 */
int fp8rl_quant_act_token_group128(const uint16_t* a, int64_t m, int64_t k, int64_t lda,
                                   uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                   void* stream);

/*
 * Dense blockwise-scaled FP8 GEMM:  y = bf16( qa . qw^T ) with the block scales
 * (section 2.1.1 Eq. (1) scales on both operands; section 2.1.4 FP8 GEMM):
 *
 *   y[i][j] = bf16_rne( sum_kb  sa[kb*ld_sa + i] * sw[(j/128)*(k/128) + kb]
 *                               * sum_{c in kb} dec(qa[i][c]) * dec(qw[j][c]) )
 *
 * qa  [m][lda] E4M3 activation codes; sa [k/128][ld_sa] their scales (as written
 *     by fp8rl_quant_act_token_group128)
 * qw  [n][ldw] E4M3 weight codes;     sw [n/128][k/128] their block scales (as
 *     written by fp8rl_quant_weight_block128)
 * y   [m][ldy] bf16 out
 * fp32 accumulation inside each 128-wide K block, fp32 scale application per K
 * block, fp32 -> bf16 round-to-nearest-even at the end; no bias.
 * n, k multiples of 128; m >= 0 arbitrary (m == 0 is a no-op); at most 2^30
 * output tiles of 128 x 128 (ceil(m/128) * n/128), else FP8RL_ERR_UNSUPPORTED_SHAPE.
 * Alignment: qa, qw, y 16-byte aligned; lda % 16 == 0; ldw % 16 == 0; ldy % 8 == 0;
 * sa, sw 4-byte aligned.  lda >= k, ldw >= k, ldy >= n, ld_sa >= m;
 * lda, ldw < 2^24 (else FP8RL_ERR_UNSUPPORTED_SHAPE).
 */
int fp8rl_gemm_w8a8_block(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                          const uint8_t* qw, int64_t ldw, const float* sw,
                          uint16_t* y, int64_t ldy, int64_t m, int64_t n, int64_t k,
                          void* stream);

/*
 * The same dense product (same operation and arguments as fp8rl_gemm_w8a8_block,
 * section 2.1.1 Eq. (1) and section 2.1.4), for callers that can lend a
 * workspace: shapes whose output tiles are too few to fill the GPU (decode,
 * m of up to a few hundred tokens; for 128 < m <= 256 only when k > 4096, as
 * shorter K ranges run unsplit on 64 x 64 tiles) split the K range over several
 * workgroups, which write fp32 partial sums to the workspace; a second kernel
 * adds them in a fixed order and rounds to bf16 once.
 *
 * fp8rl_gemm_w8a8_block_workspace_size: bytes of workspace the split needs for
 * this shape (splits * m * n * 4), 0 when the shape is not split (then
 * fp8rl_gemm_w8a8_block_ws runs exactly fp8rl_gemm_w8a8_block) or is invalid.
 * A pure function of (m, n, k); no device call.
 *
 * fp8rl_gemm_w8a8_block_ws: workspace is a DEVICE buffer of workspace_bytes,
 * 16-byte aligned, owned by the caller, no initial contents required; it is
 * overwritten, and two calls that overlap in time must not share it.  With
 * workspace_bytes below the size above the call runs unsplit.  Errors: those
 * of fp8rl_gemm_w8a8_block, then FP8RL_ERR_INVALID_ARG for workspace_bytes < 0
 * or a NULL workspace with workspace_bytes > 0, FP8RL_ERR_MISALIGNED for a
 * workspace not 16-byte aligned.  The split result is deterministic and meets
 * the same tolerance; it is not bit-identical to the unsplit path (the K
 * blocks are summed in a different fp32 order).
 */
int64_t fp8rl_gemm_w8a8_block_workspace_size(int64_t m, int64_t n, int64_t k);

int fp8rl_gemm_w8a8_block_ws(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                             const uint8_t* qw, int64_t ldw, const float* sw,
                             uint16_t* y, int64_t ldy, int64_t m, int64_t n, int64_t k,
                             void* workspace, int64_t workspace_bytes, void* stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, serving loops
 * that forbid allocation): the dense product of fp8rl_gemm_w8a8_block_ws without
 * a workspace argument.  The split-K partial sums go to a static device array of
 * FP8RL_SPLITK_SCRATCH_BYTES (16 MiB) inside the library, one per GPU, held
 * until the process ends; its address on the current device is looked up once
 * (hipGetSymbolAddress) and the call itself allocates nothing.  Same arguments,
 * validation and result as fp8rl_gemm_w8a8_block_ws given a workspace of
 * fp8rl_gemm_w8a8_block_workspace_size(m, n, k) bytes (bit-identical output).
 * FP8RL_ERR_SCRATCH_LIMIT (nothing launched) when that size exceeds the static
 * array; with the current split rule no valid shape needs more than 16 MiB.
 * The array keeps the last call's contents and needs no clearing (every partial
 * sum read is written first by the same call).  Calls that overlap in time on
 * one GPU (concurrent streams or threads) share the array and race: serialise
 * them.
 */
#define FP8RL_SPLITK_SCRATCH_BYTES (16ll << 20)

int fp8rl_gemm_w8a8_block_noalloc(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                  const uint8_t* qw, int64_t ldw, const float* sw,
                                  uint16_t* y, int64_t ldy, int64_t m, int64_t n, int64_t k,
                                  void* stream);

/*
 * Grouped (MoE expert) blockwise-scaled FP8 GEMM (section 2.1.1: MoE expert
 * layers fc1/fc2 are quantised like every other linear layer).
 *
 * Rows are stored grouped by expert: rows group_offsets[e] .. group_offsets[e+1]-1
 * of qa / y belong to expert e and use weight e.  For each expert with rows:
 *   y[rows of e] = the dense product above with qw[e], sw[e].
 * Experts without rows cost nothing and write nothing.
 *
 * qa            [total_rows][k] E4M3 codes, contiguous
 * sa            [k/128][ld_sa] fp32, indexed by global row; ld_sa >= total_rows
 * qw            [num_groups][n][k] E4M3 codes, contiguous
 * sw            [num_groups][n/128][k/128] fp32, contiguous
 * group_offsets DEVICE int32 [num_groups+1]: offsets[0] == 0, non-decreasing,
 *               offsets[num_groups] == total_rows (precondition, not checked:
 *               checking would need a device read)
 * y             [total_rows][n] bf16 out, contiguous
 * n, k multiples of 128, k < 2^24; 1 <= num_groups <= 1024 (else
 * FP8RL_ERR_UNSUPPORTED_SHAPE); total_rows >= 0 (0 is a no-op).
 * Alignment: qa, qw, y 16-byte aligned; k % 16 == 0 follows from k % 128 == 0.
 */
int fp8rl_grouped_gemm_w8a8_block(const uint8_t* qa, const float* sa, int64_t ld_sa,
                                  const uint8_t* qw, const float* sw,
                                  const int32_t* group_offsets, int64_t num_groups,
                                  int64_t total_rows, uint16_t* y, int64_t n, int64_t k,
                                  void* stream);

/*
 * The grouped GEMM over gathered rows: MoE dispatch and expert product in one
 * pass.  Per-token quantisation commutes with copying rows (section 2.1.1:
 * one scale per token and 128-wide group), so tokens are quantised once and
 * each expert reads its tokens' codes and scales directly:
 *   y[r] = (grouped product above)[r] with activation row row_index[r],
 * i.e. exactly fp8rl_gather_rows_fp8(row_index) followed by
 * fp8rl_grouped_gemm_w8a8_block, without the gathered copy (bit-identical
 * results: the same sums in the same order).
 *
 * qa         [src_rows][lda] E4M3 codes of the tokens; lda >= k, lda % 16 == 0
 * sa         [k/128][ld_sa] fp32 token scales; ld_sa >= src_rows
 * src_rows   >= 1 when total_rows > 0; src_rows * lda < 2^32 (else
 *            FP8RL_ERR_UNSUPPORTED_SHAPE)
 * row_index  DEVICE int32 [total_rows]: the token of each expert-ordered row
 *            (precondition 0 <= row_index[r] < src_rows; an index outside is
 *            clamped into range, reading a wrong row, never out of bounds)
 * qw, sw, group_offsets, num_groups, total_rows, y, n, k: as above.
 * Alignment: qa, qw, y 16-byte aligned; sa, sw, group_offsets, row_index
 * 4-byte aligned.
 */
int fp8rl_grouped_gemm_w8a8_block_gathered(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                           int64_t src_rows, const int32_t* row_index,
                                           const uint8_t* qw, const float* sw,
                                           const int32_t* group_offsets, int64_t num_groups,
                                           int64_t total_rows, uint16_t* y, int64_t n, int64_t k,
                                           void* stream);

/*
 * Power-of-two (UE8M0) scale variant (section 2.4.3, "Scaling Factor: FP32 vs
 * Power-of-2": the same 128x128 / 1x128 blocks with scales restricted to 2^k).
 * Same arguments, layouts, error codes and alignment rules as the fp32-scale
 * entry points above; the scales are written as fp32 values 2^k:
 *   k = the smallest integer with amax <= 448 * 2^k, clamped below at -127
 *       (the smallest UE8M0 value); 1.0 for an all-zero block or group;
 *   code = E4M3(x * 2^-k) (an exact scaling, then round to nearest even).
 * The UE8M0 byte of a scale is k + 127, the fp32 value's exponent field.
 */
int fp8rl_quant_weight_block128_ue8m0(const uint16_t* w, int64_t n, int64_t k, int64_t ldw,
                                      uint8_t* q, int64_t ldq, float* scale, void* stream);

int fp8rl_quant_act_token_group128_ue8m0(const uint16_t* a, int64_t m, int64_t k, int64_t lda,
                                         uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                         void* stream);

/*
 * The dense and grouped GEMMs for power-of-two scales: the same products as
 * fp8rl_gemm_w8a8_block / fp8rl_grouped_gemm_w8a8_block, with the scales
 * applied by gfx950's MX-scaled MFMA (no per-K-block scale arithmetic in the
 * kernel).  Same arguments, layouts, error codes and alignment rules.
 * Precondition (not checked, it would need a device read): every sa and sw
 * entry is a power of two 2^-127 .. 2^127, as the _ue8m0 quantisers write
 * them; only the exponent field of each scale is read.
 */
int fp8rl_gemm_w8a8_block_ue8m0(const uint8_t* qa, int64_t lda, const float* sa, int64_t ld_sa,
                                const uint8_t* qw, int64_t ldw, const float* sw,
                                uint16_t* y, int64_t ldy, int64_t m, int64_t n, int64_t k, void* stream);

int fp8rl_grouped_gemm_w8a8_block_ue8m0(const uint8_t* qa, const float* sa, int64_t ld_sa,
                                        const uint8_t* qw, const float* sw,
                                        const int32_t* group_offsets, int64_t num_groups,
                                        int64_t total_rows, uint16_t* y, int64_t n, int64_t k,
                                        void* stream);

/*
 * Down-projection input of the gated MLP, quantised (section 2.1.1: down_proj /
 * MoE fc2 are quantised like every linear layer, their activations dynamically
 * with 1x128 groups; section 3.1).  From the fused gate_up output:
 *
 *   h[t][c] = bf16_rne( SiLU(gu[t][c]) * gu[t][inter + c] ),  SiLU(g) = g / (1 + e^-g)
 *
 * evaluated in fp32 and rounded once, then quantised exactly as
 * fp8rl_quant_act_token_group128 quantises a bf16 input (the codes and scales
 * are bit-identical to running that entry point on h).
 *
 * gu     [m][ld_gu] bf16: columns 0..inter-1 gate, inter..2*inter-1 up
 * q      [m][ldq]  E4M3 codes of h out
 * scale  [inter/128][ld_scale] fp32 out, token index contiguous (as above)
 * h      [m][ldh]  bf16 h out, or NULL to skip writing it (ldh then ignored)
 * inter  multiple of 128 (else FP8RL_ERR_UNSUPPORTED_SHAPE); m == 0 is a no-op
 * Alignment: gu, q, h 16-byte aligned; ld_gu % 8 == 0; ldh % 8 == 0; ldq % 16 == 0;
 * scale 4-byte aligned.  ld_gu >= 2*inter, ldq >= inter, ldh >= inter, ld_scale >= m.
 */
int fp8rl_silu_mul_quant_group128(const uint16_t* gu, int64_t m, int64_t inter, int64_t ld_gu,
                                  uint8_t* q, int64_t ldq, float* scale, int64_t ld_scale,
                                  uint16_t* h, int64_t ldh, void* stream);

/*
 * Row gather of quantised activations (MoE dispatch: each token's row goes to the
 * rows of its experts).  Per-token 1x128 quantisation commutes with copying rows
 * (section 2.1.1, dynamic per-token activation scales), so tokens are quantised
 * once and gathered:
 *
 *   q_dst[r][:] = q_src[index[r]][:],   s_dst[g*ld_s_dst + r] = s_src[g*ld_s_src + index[r]]
 *
 * q_src  [src_rows][ldq_src] E4M3; s_src [k/128][ld_s_src] fp32 (token index contiguous)
 * index  DEVICE int32 [rows], each in [0, src_rows) (precondition, not checked:
 *        an index outside is clamped into range, so it reads a wrong row but
 *        never outside the source)
 * q_dst  [rows][ldq_dst] out; s_dst [k/128][ld_s_dst] out
 * k multiple of 128; rows == 0 is a no-op; src_rows >= 1 when rows > 0.
 * Destination and source must not overlap.
 * Alignment: q_src, q_dst 16-byte aligned; ldq_src % 16 == 0; ldq_dst % 16 == 0;
 * s_src, s_dst 4-byte aligned.  ldq_* >= k, ld_s_src >= src_rows, ld_s_dst >= rows.
 */
int fp8rl_gather_rows_fp8(const uint8_t* q_src, int64_t ldq_src, const float* s_src, int64_t ld_s_src,
                          int64_t src_rows, const int32_t* index, int64_t rows, int64_t k,
                          uint8_t* q_dst, int64_t ldq_dst, float* s_dst, int64_t ld_s_dst, void* stream);

/*
 * Token-level truncated importance sampling and the mismatch KL (section 2.1.3,
 * Eq. (2)-(3): w = pi_theta / pi_theta^FP8 per sampled token, truncated at C;
 * section 2.2: D_KL(pi^FP8 || pi_theta) over the rollout tokens).  For each token i:
 *
 *   d = logp_train[i] - logp_rollout[i]  (fp64, exact),   w = e^d
 *   w_tis[i] = fp32(min(w, clip_c)) for tokens in the mask, 0 for the others
 *
 * and over the tokens in the mask (fp64, deterministic order):
 *   stats[0] = sum of -d            (KL estimate: stats[0] / stats[2])
 *   stats[1] = sum of expm1(d) - d  (non-negative KL estimate: stats[1] / stats[2])
 *   stats[2] = number of tokens in the mask
 *   stats[3] = number of tokens with w > clip_c
 *
 * logp_train    DEVICE fp32 [n]: log-probabilities of the sampled tokens under the
 *               bf16 training policy; logp_rollout likewise under the FP8 rollout policy
 * mask          DEVICE uint8 [n], nonzero = token counts; NULL = every token counts
 * clip_c        C > 0, finite (the paper uses 2)
 * w_tis         DEVICE fp32 [n] out;  stats: DEVICE double [4] out (written also for n == 0)
 * workspace     caller-lent device memory of at least fp8rl_tis_workspace_size(n)
 *               bytes, 8-byte aligned, no initial contents, not shared by calls that
 *               may overlap (else FP8RL_ERR_INVALID_ARG when missing or short)
 * Inputs are finite (precondition).  Alignment: the fp32 arrays 16-byte, mask
 * 4-byte, stats and workspace 8-byte aligned.
 */
int64_t fp8rl_tis_workspace_size(int64_t n);

int fp8rl_tis_weights_kl(const float* logp_train, const float* logp_rollout, const uint8_t* mask, int64_t n,
                         float clip_c, float* w_tis, double* stats, void* workspace, int64_t workspace_bytes,
                         void* stream);

/*
 * FP8 KV cache (section 2.3): long-context rollouts are memory-bound, so keys and
 * values are cached in E4M3 with one fp32 scale per layer and tensor, recalibrated
 * at every RL step because the policy weights change (section 2.3.1).
 *
 * Calibration: scale = fl32(amax / 448) over x (bf16 [n], e.g. one layer's keys
 * of the step's calibration pass); 1.0 when every value is zero.  Writes the
 * DEVICE fp32 *scale (no host synchronisation).  workspace: caller-lent device
 * memory of fp8rl_kv_calibrate_workspace_size(n) bytes, 4-byte aligned, not
 * shared by overlapping calls.  x 16-byte aligned.  Inputs finite (precondition).
 */
int64_t fp8rl_kv_calibrate_workspace_size(int64_t n);

int fp8rl_kv_calibrate_scale(const uint16_t* x, int64_t n, float* scale, void* workspace, int64_t workspace_bytes,
                             void* stream);

/*
 * Cache write: new tokens' keys and values (bf16 [tokens][kv_heads][head_dim],
 * contiguous) into the paged caches (one kv head's 16-token block is contiguous
 * in both):
 *   k_cache [num_blocks][kv_heads][16][head_dim]       token o of a block at [o][d]
 *   v_cache [num_blocks][kv_heads][4][head_dim][4]     token o at [o / 4][d][o % 4]
 * (the value layout puts four tokens of one dim in one dword, the operand order
 * of the attention kernel's value product), with
 *   code = E4M3(fl32(x / s)) rounded to nearest even, saturated at +-448,
 * s = *k_scale / *v_scale (DEVICE fp32).  slot_mapping: DEVICE int64 [tokens],
 * slot = block * 16 + offset; slots outside [0, num_blocks * 16) are skipped
 * (negative: padding tokens); two tokens with one slot: which one's codes land
 * is unspecified.  head_dim must be 128; ceil(tokens / 4) * kv_heads * 16 < 2^31
 * (else FP8RL_ERR_UNSUPPORTED_SHAPE).  Alignment: k, v 16-byte; caches and
 * slot_mapping 8-byte.
 */
int fp8rl_kv_cache_write_fp8(const uint16_t* k, const uint16_t* v, int64_t tokens, int64_t kv_heads,
                             int64_t head_dim, const int64_t* slot_mapping, int64_t num_blocks, const float* k_scale,
                             const float* v_scale, uint8_t* k_cache, uint8_t* v_cache, void* stream);

/*
 * Decode attention over the paged FP8 cache, one new query token per sequence,
 * grouped query heads (query head h reads kv head h / (q_heads / kv_heads)):
 *   out[b][h] = softmax_t(sm_scale * q[b][h] . K_t) . V_t,
 *   K_t = dec(k code) * (*k_scale), V_t = dec(v code) * (*v_scale),
 * over the seq_lens[b] tokens of sequence b, whose 16-token blocks are
 * block_table[b][0 ..].  The arithmetic is bf16 x bf16 -> fp32 for the scores
 * (every E4M3 code is exact in bf16) and fp32 for the softmax and the values
 * ("KV cache FP8 only": the cache, not the attention math, is FP8).
 *
 * k_cache, v_cache  the layouts written by fp8rl_kv_cache_write_fp8
 * q            DEVICE bf16 [batch][q_heads][128];  out: DEVICE bf16 [batch][q_heads][128]
 * block_table  DEVICE int32 [batch][max_blocks]; seq_lens DEVICE int32 [batch]
 * max_seq_len  an upper bound of every seq_lens[b] (precondition: tokens past it are
 *              ignored), max_blocks * 16 >= max_seq_len; a block id outside
 *              [0, num_blocks) is clamped into range (reads a wrong block, never
 *              outside the cache); an empty sequence gives 0
 * q_heads / kv_heads in {1, 2, 4, 8}; head_dim 128; batch, kv_heads <= 65535
 * workspace    caller-lent device memory of
 *              fp8rl_attention_decode_workspace_size(batch, q_heads, kv_heads, max_seq_len)
 *              bytes, 16-byte aligned, not shared by overlapping calls
 * Alignment: q and the caches 16-byte, the rest 4-byte.
 * The _bf16kv variant reads bf16 caches of the same layout (no scales), for
 * comparison with the FP8 cache.
 */
int64_t fp8rl_attention_decode_workspace_size(int64_t batch, int64_t q_heads, int64_t kv_heads,
                                              int64_t max_seq_len);

int fp8rl_attention_decode_fp8kv(const uint16_t* q, const uint8_t* k_cache, const uint8_t* v_cache, int64_t num_blocks,
                                 const int32_t* block_table, int64_t max_blocks, const int32_t* seq_lens,
                                 int64_t batch, int64_t q_heads, int64_t kv_heads, int64_t head_dim,
                                 int64_t max_seq_len, const float* k_scale, const float* v_scale, float sm_scale,
                                 uint16_t* out, void* workspace, int64_t workspace_bytes, void* stream);

int fp8rl_attention_decode_bf16kv(const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                                  int64_t num_blocks, const int32_t* block_table, int64_t max_blocks,
                                  const int32_t* seq_lens, int64_t batch, int64_t q_heads, int64_t kv_heads,
                                  int64_t head_dim, int64_t max_seq_len, float sm_scale, uint16_t* out,
                                  void* workspace, int64_t workspace_bytes, void* stream);

/* Human-readable name of a status code (static string, never NULL). */
const char* fp8rl_status_string(int status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int fp8rl_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FP8RL_H */
