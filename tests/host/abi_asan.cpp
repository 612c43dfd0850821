// Host-only build of the C ABI's argument validation (csrc/api.cpp) with
// AddressSanitizer and UndefinedBehaviorSanitizer.  The kernel launchers are
// replaced by stubs that only count calls, so every entry point runs its whole
// validation path on the CPU; fake device pointers are never dereferenced.
// Each invalid call must return its documented status without launching, each
// valid one must reach exactly one launcher.  Built and run by tests/test_abi.py.
#include <cstdio>
#include <cstdlib>
#include <string>

#include "../../paper_2601_18150_amd/csrc/api.cpp"

namespace {
int g_launches = 0;
hipError_t stub() { ++g_launches; return hipSuccess; }
}  // namespace

namespace fp8rl {
hipError_t launch_quant_weight_block128(const uint16_t*, int64_t, int64_t, int64_t, uint8_t*, int64_t, float*,
                                        hipStream_t, bool) { return stub(); }
hipError_t launch_quant_weight_block128_batched(const WeightJob*, int, hipStream_t) { return stub(); }
hipError_t launch_quant_act_token_group128(const uint16_t*, int64_t, int64_t, int64_t, uint8_t*, int64_t, float*,
                                           int64_t, hipStream_t, bool) { return stub(); }
hipError_t launch_silu_mul_quant_group128(const uint16_t*, int64_t, int64_t, int64_t, uint8_t*, int64_t, float*,
                                          int64_t, uint16_t*, int64_t, hipStream_t) { return stub(); }
hipError_t launch_gather_rows_fp8(const uint8_t*, int64_t, const float*, int64_t, const int32_t*, int64_t, int64_t,
                                  int64_t, uint8_t*, int64_t, float*, int64_t, hipStream_t) { return stub(); }
hipError_t launch_gemm_w8a8_block(const uint8_t*, int64_t, const float*, int64_t, const uint8_t*, int64_t,
                                  const float*, uint16_t*, int64_t, int64_t, int64_t, int64_t, hipStream_t, bool) {
  return stub();
}
// a stand-in split rule (the real one lives with the kernels): split small-M shapes in 4
int splitk_factor(int64_t m, int64_t, int64_t k) { return (m <= 256 && k >= 2048) ? 4 : 1; }
hipError_t launch_gemm_w8a8_block_splitk(const uint8_t*, int64_t, const float*, int64_t, const uint8_t*, int64_t,
                                         const float*, uint16_t*, int64_t, int64_t, int64_t, int64_t, float*, int,
                                         hipStream_t) { return stub(); }
hipError_t splitk_scratch(float** out) { *out = reinterpret_cast<float*>(uintptr_t(1) << 24); return hipSuccess; }
hipError_t launch_grouped_gemm_w8a8_block(const uint8_t*, const float*, int64_t, const uint8_t*, const float*,
                                          const int32_t*, int64_t, int64_t, uint16_t*, int64_t, int64_t, hipStream_t,
                                          bool) { return stub(); }
hipError_t launch_grouped_gemm_w8a8_block_gathered(const uint8_t*, int64_t, const float*, int64_t, int64_t,
                                                   const int32_t*, const uint8_t*, const float*, const int32_t*,
                                                   int64_t, int64_t, uint16_t*, int64_t, int64_t, hipStream_t) {
  return stub();
}
int tis_blocks(int64_t n) { return n > 0 ? 16 : 1; }
hipError_t launch_tis_weights_kl(const float*, const float*, const uint8_t*, int64_t, float, float*, double*, double*,
                                 hipStream_t) { return stub(); }
int kv_amax_blocks(int64_t n) { return n > 0 ? 8 : 1; }
hipError_t launch_kv_calibrate_scale(const uint16_t*, int64_t, float*, uint32_t*, hipStream_t) { return stub(); }
hipError_t launch_kv_cache_write(const uint16_t*, const uint16_t*, int64_t, int, const int64_t*, int64_t, const float*,
                                 const float*, uint8_t*, uint8_t*, hipStream_t) { return stub(); }
AttnSplit attn_decode_split(int64_t, int64_t, int64_t, int64_t) { return AttnSplit{256, 4, 132}; }
hipError_t launch_attention_decode(const uint16_t*, const void*, const void*, bool, int64_t, const int32_t*, int64_t,
                                   const int32_t*, int64_t, int64_t, int64_t, int64_t, const float*, const float*,
                                   float, uint16_t*, float*, hipStream_t) { return stub(); }
}  // namespace fp8rl

namespace {
int g_fail = 0;

template <class T>
T* fake(uintptr_t off = 0) { return reinterpret_cast<T*>((uintptr_t(1) << 20) + off); }

void expect(const char* what, int got, int want) {
  if (got != want) {
    std::printf("FAIL %s: status %d, want %d\n", what, got, want);
    ++g_fail;
  }
}

// Run one call: status and number of launches it made.
#define CHECK(what, call, want_status, want_launches)                                                 \
  do {                                                                                                \
    const int l0 = g_launches;                                                                        \
    const int st = (call);                                                                            \
    expect(what, st, want_status);                                                                    \
    if (g_launches - l0 != (want_launches)) {                                                         \
      std::printf("FAIL %s: %d launches, want %d\n", what, g_launches - l0, (want_launches));         \
      ++g_fail;                                                                                       \
    }                                                                                                 \
  } while (0)
}  // namespace

int main() {
  const int OK = FP8RL_OK, INV = FP8RL_ERR_INVALID_ARG, SHP = FP8RL_ERR_UNSUPPORTED_SHAPE,
            MIS = FP8RL_ERR_MISALIGNED;
  auto* w = fake<uint16_t>();
  auto* q = fake<uint8_t>(1 << 16);
  auto* s = fake<float>(1 << 17);
  auto* y = fake<uint16_t>(1 << 18);
  auto* i32 = fake<int32_t>(1 << 19);
  auto* i64 = fake<int64_t>(1 << 19);
  void* ws = fake<void>(1 << 21);

  // weight quantisation
  CHECK("wq ok", fp8rl_quant_weight_block128(w, 256, 128, 128, q, 128, s, nullptr), OK, 1);
  CHECK("wq n%128", fp8rl_quant_weight_block128(w, 200, 128, 128, q, 128, s, nullptr), SHP, 0);
  CHECK("wq neg", fp8rl_quant_weight_block128(w, -128, 128, 128, q, 128, s, nullptr), INV, 0);
  CHECK("wq null", fp8rl_quant_weight_block128(nullptr, 128, 128, 128, q, 128, s, nullptr), INV, 0);
  CHECK("wq ld", fp8rl_quant_weight_block128(w, 128, 256, 128, q, 256, s, nullptr), INV, 0);
  CHECK("wq align", fp8rl_quant_weight_block128(fake<uint16_t>(2), 128, 128, 128, q, 128, s, nullptr), MIS, 0);
  CHECK("wq empty", fp8rl_quant_weight_block128(nullptr, 0, 128, 128, nullptr, 128, nullptr, nullptr), OK, 0);
  CHECK("wq ue8m0 ok", fp8rl_quant_weight_block128_ue8m0(w, 128, 128, 128, q, 128, s, nullptr), OK, 1);

  // batched weight quantisation
  fp8rl_weight_job jobs[3] = {{w, 128, 128, 128, q, 128, s}, {w, 256, 256, 256, q, 256, s},
                              {w, 0, 128, 128, nullptr, 128, nullptr}};
  CHECK("wqb ok", fp8rl_quant_weight_block128_batched(jobs, 3, nullptr), OK, 1);
  CHECK("wqb null jobs", fp8rl_quant_weight_block128_batched(nullptr, 2, nullptr), INV, 0);
  CHECK("wqb negative count", fp8rl_quant_weight_block128_batched(jobs, -1, nullptr), INV, 0);
  fp8rl_weight_job bad[2] = {{w, 128, 128, 128, q, 128, s}, {w, 100, 128, 128, q, 128, s}};
  CHECK("wqb bad job", fp8rl_quant_weight_block128_batched(bad, 2, nullptr), SHP, 0);

  // activation quantisation
  CHECK("aq ok", fp8rl_quant_act_token_group128(w, 37, 256, 256, q, 256, s, 40, nullptr), OK, 1);
  CHECK("aq ld_scale", fp8rl_quant_act_token_group128(w, 37, 256, 256, q, 256, s, 36, nullptr), INV, 0);
  CHECK("aq k%128", fp8rl_quant_act_token_group128(w, 37, 200, 256, q, 256, s, 40, nullptr), SHP, 0);
  CHECK("aq ue8m0 ok", fp8rl_quant_act_token_group128_ue8m0(w, 1, 128, 128, q, 128, s, 1, nullptr), OK, 1);

  // fused SiLU*mul + quantisation, row gather
  CHECK("silu ok", fp8rl_silu_mul_quant_group128(w, 3, 128, 256, q, 128, s, 3, y, 128, nullptr), OK, 1);
  CHECK("silu ld", fp8rl_silu_mul_quant_group128(w, 3, 128, 128, q, 128, s, 3, y, 128, nullptr), INV, 0);
  CHECK("gather ok", fp8rl_gather_rows_fp8(q, 128, s, 10, 10, i32, 20, 128, q, 128, s, 20, nullptr), OK, 1);
  CHECK("gather null idx", fp8rl_gather_rows_fp8(q, 128, s, 10, 10, nullptr, 20, 128, q, 128, s, 20, nullptr), INV, 0);

  // dense GEMM and its split-K / no-allocation forms
  CHECK("gemm ok", fp8rl_gemm_w8a8_block(q, 128, s, 8, q, 128, s, y, 128, 8, 128, 128, nullptr), OK, 1);
  CHECK("gemm n%128", fp8rl_gemm_w8a8_block(q, 128, s, 8, q, 128, s, y, 200, 8, 200, 128, nullptr), SHP, 0);
  CHECK("gemm lda<k", fp8rl_gemm_w8a8_block(q, 112, s, 8, q, 128, s, y, 128, 8, 128, 128, nullptr), INV, 0);
  CHECK("gemm pitch", fp8rl_gemm_w8a8_block(q, 1 << 24, s, 8, q, 128, s, y, 128, 8, 128, 128, nullptr), SHP, 0);
  CHECK("gemm align", fp8rl_gemm_w8a8_block(fake<uint8_t>(8), 128, s, 8, q, 128, s, y, 128, 8, 128, 128, nullptr),
        MIS, 0);
  CHECK("gemm ue8m0 ok", fp8rl_gemm_w8a8_block_ue8m0(q, 128, s, 8, q, 128, s, y, 128, 8, 128, 128, nullptr), OK, 1);
  const int64_t need = fp8rl_gemm_w8a8_block_workspace_size(100, 256, 2048);
  if (need != 4 * 100 * 256 * 4) { std::printf("FAIL workspace size %lld\n", (long long)need); ++g_fail; }
  CHECK("ws split", fp8rl_gemm_w8a8_block_ws(q, 2048, s, 100, q, 2048, s, y, 256, 100, 256, 2048, ws, need, nullptr),
        OK, 1);
  CHECK("ws short", fp8rl_gemm_w8a8_block_ws(q, 2048, s, 100, q, 2048, s, y, 256, 100, 256, 2048, ws, 64, nullptr),
        OK, 1);
  CHECK("ws negative", fp8rl_gemm_w8a8_block_ws(q, 2048, s, 100, q, 2048, s, y, 256, 100, 256, 2048, ws, -1, nullptr),
        INV, 0);
  CHECK("ws misaligned",
        fp8rl_gemm_w8a8_block_ws(q, 2048, s, 100, q, 2048, s, y, 256, 100, 256, 2048, fake<void>(4), need, nullptr),
        MIS, 0);
  CHECK("noalloc split", fp8rl_gemm_w8a8_block_noalloc(q, 2048, s, 100, q, 2048, s, y, 256, 100, 256, 2048, nullptr),
        OK, 1);
  CHECK("noalloc limit",
        fp8rl_gemm_w8a8_block_noalloc(q, 4096, s, 256, q, 4096, s, y, 8192, 256, 8192, 4096, nullptr),
        FP8RL_ERR_SCRATCH_LIMIT, 0);

  // grouped GEMMs
  CHECK("grouped ok", fp8rl_grouped_gemm_w8a8_block(q, s, 64, q, s, i32, 4, 64, y, 128, 128, nullptr), OK, 1);
  CHECK("grouped groups", fp8rl_grouped_gemm_w8a8_block(q, s, 64, q, s, i32, 0, 64, y, 128, 128, nullptr), INV, 0);
  CHECK("grouped too many", fp8rl_grouped_gemm_w8a8_block(q, s, 64, q, s, i32, 1025, 64, y, 128, 128, nullptr), SHP,
        0);
  CHECK("grouped ue8m0 ok", fp8rl_grouped_gemm_w8a8_block_ue8m0(q, s, 64, q, s, i32, 4, 64, y, 128, 128, nullptr), OK,
        1);
  CHECK("gathered ok",
        fp8rl_grouped_gemm_w8a8_block_gathered(q, 128, s, 16, 16, i32, q, s, i32, 4, 64, y, 128, 128, nullptr), OK, 1);
  CHECK("gathered null index",
        fp8rl_grouped_gemm_w8a8_block_gathered(q, 128, s, 16, 16, nullptr, q, s, i32, 4, 64, y, 128, 128, nullptr),
        INV, 0);

  // TIS, KV cache
  const int64_t tws = fp8rl_tis_workspace_size(1000);
  CHECK("tis ok", fp8rl_tis_weights_kl(s, s, q, 1000, 2.0f, s, fake<double>(1 << 22), ws, tws, nullptr), OK, 1);
  CHECK("tis clip", fp8rl_tis_weights_kl(s, s, q, 1000, 0.0f, s, fake<double>(1 << 22), ws, tws, nullptr), INV, 0);
  CHECK("tis short ws", fp8rl_tis_weights_kl(s, s, q, 1000, 2.0f, s, fake<double>(1 << 22), ws, 8, nullptr), INV, 0);
  const int64_t kws = fp8rl_kv_calibrate_workspace_size(4096);
  CHECK("kv cal ok", fp8rl_kv_calibrate_scale(w, 4096, s, ws, kws, nullptr), OK, 1);
  CHECK("kv cal null", fp8rl_kv_calibrate_scale(w, 4096, nullptr, ws, kws, nullptr), INV, 0);
  CHECK("kv write ok", fp8rl_kv_cache_write_fp8(w, w, 4, 8, 128, i64, 2, s, s, q, q, nullptr), OK, 1);
  CHECK("kv write head", fp8rl_kv_cache_write_fp8(w, w, 4, 8, 64, i64, 2, s, s, q, q, nullptr), SHP, 0);
  const int64_t aws = fp8rl_attention_decode_workspace_size(2, 32, 8, 4096);
  CHECK("attn ok", fp8rl_attention_decode_fp8kv(w, q, q, 16, i32, 256, i32, 2, 32, 8, 128, 4096, s, s, 0.08f, y, ws,
                                                aws, nullptr), OK, 1);
  CHECK("attn group", fp8rl_attention_decode_fp8kv(w, q, q, 16, i32, 256, i32, 2, 48, 3, 128, 4096, s, s, 0.08f, y,
                                                   ws, aws, nullptr), SHP, 0);
  CHECK("attn sm_scale", fp8rl_attention_decode_bf16kv(w, w, w, 16, i32, 256, i32, 2, 32, 8, 128, 4096, -1.0f, y, ws,
                                                       aws, nullptr), INV, 0);

  if (std::string(fp8rl_status_string(FP8RL_ERR_SCRATCH_LIMIT)) != "FP8RL_ERR_SCRATCH_LIMIT") ++g_fail;
  if (g_fail) {
    std::printf("%d failures\n", g_fail);
    return 1;
  }
  std::printf("ok: %d launches\n", g_launches);
  return 0;
}
