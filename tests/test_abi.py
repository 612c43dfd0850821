"""CPU-side checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects bad arguments with the documented status codes
before launching anything.  Every call here fails validation (or is an empty
no-op), so none of them reaches the GPU, even on a machine that has one: the
fake pointers are never dereferenced."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fp8rl.h")

OK, INVALID, SHAPE, MISALIGNED = 0, 1, 2, 3
A16 = 1 << 20          # a fake, 16-byte-aligned device address (never dereferenced)
A4 = A16 + 4           # 4-byte aligned only


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fp8rl_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2601_18150_amd as fp8rl
    return fp8rl.load()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for f in ("fp8rl_quant_weight_block128", "fp8rl_quant_act_token_group128",
              "fp8rl_gemm_w8a8_block", "fp8rl_grouped_gemm_w8a8_block",
              "fp8rl_silu_mul_quant_group128", "fp8rl_gather_rows_fp8", "fp8rl_tis_weights_kl"):
        assert f in names


def test_library_exports_every_declared_symbol(lib):
    import paper_2601_18150_amd as fp8rl
    out = subprocess.run(["nm", "-D", "--defined-only", fp8rl.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (fp8rl_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_status_strings_and_version(lib):
    import paper_2601_18150_amd as fp8rl
    assert fp8rl.fp8rl_status_string(0) == "FP8RL_OK"
    assert fp8rl.fp8rl_status_string(3) == "FP8RL_ERR_MISALIGNED"
    assert fp8rl.fp8rl_status_string(5) == "FP8RL_ERR_SCRATCH_LIMIT"
    assert fp8rl.fp8rl_status_string(99) == "FP8RL_ERR_UNKNOWN"
    assert fp8rl.fp8rl_version() >= 100


def test_quant_weight_argument_errors(lib):
    f = lib.fp8rl_quant_weight_block128
    assert f(A16, -128, 128, 128, A16, 128, A16, None) == INVALID
    assert f(A16, 128, 200, 200, A16, 208, A16, None) == SHAPE
    assert f(A16, 100, 128, 128, A16, 128, A16, None) == SHAPE
    assert f(None, 128, 128, 128, A16, 128, A16, None) == INVALID
    assert f(A16, 128, 128, 120, A16, 128, A16, None) == INVALID      # ldw < k
    assert f(A16, 128, 128, 128, A16, 127, A16, None) == INVALID      # ldq < k
    assert f(A4, 128, 128, 128, A16, 128, A16, None) == MISALIGNED
    assert f(A16, 128, 128, 132, A16, 128, A16, None) == MISALIGNED   # ldw % 8
    assert f(A16, 128, 128, 128, A16, 136, A16, None) == MISALIGNED   # ldq % 16
    assert f(A16, 0, 128, 128, A16, 128, A16, None) == OK             # empty: no-op
    assert f(None, 0, 0, 0, None, 0, None, None) == OK


def test_quant_weight_batched_argument_errors(lib):
    """Every job is validated before anything is launched: one bad job among good
    ones returns its code (none of these calls reaches the GPU)."""
    import paper_2601_18150_amd as fp8rl
    f = lib.fp8rl_quant_weight_block128_batched

    def jobs(*specs):
        arr = (fp8rl.WeightJob * len(specs))()
        for i, (w, n, k, ldw, q, ldq, sc) in enumerate(specs):
            arr[i] = fp8rl.WeightJob(w, n, k, ldw, q, ldq, sc)
        return ctypes.addressof(arr), arr

    good = (A16, 128, 256, 256, A16, 256, A16)
    assert f(None, -1, None) == INVALID
    assert f(None, 3, None) == INVALID                                   # NULL array, count > 0
    assert f(None, 0, None) == OK                                        # empty batch: no-op
    for bad, code in [((A16, -128, 128, 128, A16, 128, A16), INVALID),
                      ((A16, 128, 200, 200, A16, 208, A16), SHAPE),
                      ((None, 128, 128, 128, A16, 128, A16), INVALID),
                      ((A16, 128, 128, 120, A16, 128, A16), INVALID),     # ldw < k
                      ((A4, 128, 128, 128, A16, 128, A16), MISALIGNED),
                      ((A16, 128, 128, 128, A16, 136, A16), MISALIGNED)]:  # ldq % 16
        for specs in ((bad,), (good, bad), (good, good, bad)):
            p, keep = jobs(*specs)
            assert f(p, len(specs), None) == code, (specs, code)
    p, keep = jobs((A16, 0, 128, 128, A16, 128, A16), (None, 0, 0, 0, None, 0, None))
    assert f(p, 2, None) == OK                                           # only empty jobs: no-op
    # a bad job in the second 64-job chunk: rejected before the first chunk launches
    p, keep = jobs(*([good] * 69 + [(A16, 128, 128, 128, A16, 136, A16)]))
    assert f(p, 70, None) == MISALIGNED


def test_quant_act_argument_errors(lib):
    f = lib.fp8rl_quant_act_token_group128
    assert f(A16, -1, 128, 128, A16, 128, A16, 1, None) == INVALID
    assert f(A16, 4, 100, 128, A16, 128, A16, 4, None) == SHAPE
    assert f(A16, 4, 128, 128, A16, 128, A16, 3, None) == INVALID     # ld_scale < m
    assert f(A16, 4, 128, 128, None, 128, A16, 4, None) == INVALID
    assert f(A16, 4, 128, 128, A16 + 8, 128, A16, 4, None) == MISALIGNED
    assert f(A16, 4, 128, 128, A16, 128, A16 + 2, 4, None) == MISALIGNED
    assert f(None, 0, 128, 128, None, 128, None, 0, None) == OK


def test_gemm_argument_errors(lib):
    f = lib.fp8rl_gemm_w8a8_block
    #      qa  lda  sa  ld_sa qw  ldw  sw  y   ldy  m  n    k
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 128, -8, 128, 128, None) == INVALID
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 200, 8, 200, 128, None) == SHAPE
    assert f(A16, 256, A16, 8, A16, 256, A16, A16, 128, 8, 128, 192, None) == SHAPE
    big = 1 << 30                                                     # 2^46 output tiles
    assert f(A16, 128, A16, big, A16, 128, A16, A16, big, big, big, 128, None) == SHAPE
    assert f(A16, 128, A16, 7, A16, 128, A16, A16, 128, 8, 128, 128, None) == INVALID  # ld_sa < m
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 120, 8, 128, 128, None) == INVALID  # ldy < n
    assert f(A16, 128, A16, 8, None, 128, A16, A16, 128, 8, 128, 128, None) == INVALID
    assert f(A16 + 8, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == MISALIGNED
    assert f(A16, 136, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == MISALIGNED
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 132, 8, 128, 128, None) == MISALIGNED
    assert f(A16, 1 << 24, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == SHAPE   # row pitch limit
    assert f(A16, 128, A16, 8, A16, 1 << 24, A16, A16, 128, 8, 128, 128, None) == SHAPE
    assert f(None, 128, None, 0, None, 128, None, None, 128, 0, 128, 128, None) == OK


def test_grouped_gathered_argument_errors(lib):
    f = lib.fp8rl_grouped_gemm_w8a8_block_gathered
    #       qa  lda  sa  ld_sa src idx  qw   sw   off  g  rows y    n    k
    assert f(A16, 128, A16, 8, 8, A16, A16, A16, A16, 2, -1, A16, 128, 128, None) == INVALID
    assert f(A16, 128, A16, 8, 8, A16, A16, A16, A16, 0, 8, A16, 128, 128, None) == INVALID     # no groups
    assert f(A16, 128, A16, 8, 8, A16, A16, A16, A16, 2, 8, A16, 200, 128, None) == SHAPE      # n % 128
    assert f(A16, 128, A16, 8, 0, A16, A16, A16, A16, 2, 8, A16, 128, 128, None) == INVALID    # no tokens
    assert f(A16, 128, A16, 8, 8, None, A16, A16, A16, 2, 8, A16, 128, 128, None) == INVALID   # no index
    assert f(A16, 112, A16, 8, 8, A16, A16, A16, A16, 2, 8, A16, 128, 128, None) == INVALID    # lda < k
    assert f(A16, 128, A16, 7, 8, A16, A16, A16, A16, 2, 8, A16, 128, 128, None) == INVALID    # ld_sa < src_rows
    assert f(A16, 1 << 16, A16, 1 << 16, 1 << 16, A16, A16, A16, A16, 2, 8, A16, 128, 128, None) == SHAPE  # 2^32
    assert f(A16, 136, A16, 8, 8, A16, A16, A16, A16, 2, 8, A16, 128, 128, None) == MISALIGNED  # lda % 16
    assert f(A16, 128, A16, 8, 8, A16 + 2, A16, A16, A16, 2, 8, A16, 128, 128, None) == MISALIGNED
    assert f(None, 128, None, 8, 8, None, None, None, None, 2, 0, None, 128, 128, None) == OK  # no rows: no-op


def test_gemm_workspace_size(lib):
    """The split-K workspace is a pure function of the shape: splits x M x N fp32."""
    f = lib.fp8rl_gemm_w8a8_block_workspace_size
    assert f(256, 4096, 12288) == 4 * 256 * 4096 * 4      # decode down: 64 tiles -> 4 splits of 24 K blocks
    assert f(256, 6144, 4096) == 0                        # decode qkv: 384 unsplit 64x64 tiles
    assert f(256, 4096, 4096) == 0                        # decode o_proj: 256 unsplit 64x64 tiles
    assert f(256, 24576, 4096) == 0                       # 384 tiles of 128x128 fill the GPU
    assert f(128, 4096, 4096) == 8 * 128 * 4096 * 4       # M <= 128: 32 tiles of 128x128 -> 8 splits of 4 K blocks
    assert f(300, 6144, 4096) == 0                        # M > 256: 144 tiles of 128x128, over half the CUs
    assert f(8192, 24576, 4096) == 0                      # 256x256 tiles, never split
    assert f(64, 512, 512) == 0                           # 4 K blocks: no split shorter than 4
    assert f(37, 384, 13 * 128) == 3 * 37 * 384 * 4       # uneven split of 13 K blocks
    for bad in [(0, 128, 128), (8, 200, 128), (8, 128, 192), (-1, 128, 128), (8, 128, 0)]:
        assert f(*bad) == 0


def test_gemm_ws_argument_errors(lib):
    f = lib.fp8rl_gemm_w8a8_block_ws
    #      qa  lda  sa  ld_sa qw  ldw  sw  y   ldy  m  n    k    ws   ws_bytes
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 200, 8, 200, 128, A16, 1 << 20, None) == SHAPE
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, A16, -1, None) == INVALID
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None, 64, None) == INVALID
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, A16 + 4, 64, None) == MISALIGNED
    assert f(A16 + 8, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, A16, 64, None) == MISALIGNED
    assert f(None, 128, None, 0, None, 128, None, None, 128, 0, 128, 128, None, 0, None) == OK


def test_gemm_noalloc_argument_errors(lib):
    """The no-allocation entry point validates exactly like the dense GEMM, before any device call."""
    f = lib.fp8rl_gemm_w8a8_block_noalloc
    #      qa  lda  sa  ld_sa qw  ldw  sw  y   ldy  m  n    k
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 200, 8, 200, 128, None) == SHAPE
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 192, None) == SHAPE
    assert f(A16, 128, A16, 8, A16, 128, A16, A16, 128, -1, 128, 128, None) == INVALID
    assert f(A16, 100, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == INVALID
    assert f(A16, 128, A16, 4, A16, 128, A16, A16, 128, 8, 128, 128, None) == INVALID
    assert f(None, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == INVALID
    assert f(A16 + 8, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == MISALIGNED
    assert f(A16, 128, A16, 8, A16, 1 << 24, A16, A16, 128, 8, 128, 128, None) == SHAPE
    assert f(None, 128, None, 0, None, 128, None, None, 128, 0, 128, 128, None) == OK


def test_split_k_partials_fit_the_static_scratch(lib):
    """Every shape the split rule splits needs at most FP8RL_SPLITK_SCRATCH_BYTES (16 MiB) of partial
    sums (splits x tiles <= 256 tiles of 128 x 128), so the no-allocation entry point never
    returns FP8RL_ERR_SCRATCH_LIMIT for a valid shape; the worst case is reached exactly."""
    f = lib.fp8rl_gemm_w8a8_block_workspace_size
    text = open(HEADER).read()
    limit = int(re.search(r"#define FP8RL_SPLITK_SCRATCH_BYTES \((\d+)ll << (\d+)\)", text).group(1)) << 20
    assert limit == 16 << 20
    worst = 0
    for m in list(range(1, 300, 7)) + [128, 256, 384, 511, 512, 1024, 2047, 4096]:
        for n in (128, 256, 384, 640, 1024, 2048, 4096, 8192, 16384, 32768):
            for k in (512, 1024, 4096, 12288, 65536):
                worst = max(worst, f(m, n, k))
    assert 0 < worst <= limit
    assert f(256, 4096, 12288) == limit          # the Qwen3-8B decode down projection fills it


def test_grouped_gemm_argument_errors(lib):
    f = lib.fp8rl_grouped_gemm_w8a8_block
    #        qa  sa  ld_sa qw  sw  off  G  R   y   n    k
    assert f(A16, A16, 8, A16, A16, A16, 0, 8, A16, 128, 128, None) == INVALID    # no groups
    assert f(A16, A16, 8, A16, A16, A16, 2, -1, A16, 128, 128, None) == INVALID
    assert f(A16, A16, 8, A16, A16, A16, 2, 8, A16, 192, 128, None) == SHAPE
    assert f(A16, A16, 8, A16, A16, A16, 1025, 8, A16, 128, 128, None) == SHAPE   # over 1024 experts
    assert f(A16, A16, 8, A16, A16, A16, 2, 8, A16, 128, 1 << 24, None) == SHAPE  # k at the row pitch limit
    assert f(A16, A16, 7, A16, A16, A16, 2, 8, A16, 128, 128, None) == INVALID    # ld_sa < R
    assert f(A16, A16, 8, A16, A16, None, 2, 8, A16, 128, 128, None) == INVALID
    assert f(A16, A16, 8, A16, A16, A16 + 2, 2, 8, A16, 128, 128, None) == MISALIGNED
    assert f(A16, A16, 8, A4, A16, A16, 2, 8, A16, 128, 128, None) == MISALIGNED
    assert f(None, None, 0, None, None, None, 2, 0, None, 128, 128, None) == OK


def test_silu_mul_quant_argument_errors(lib):
    f = lib.fp8rl_silu_mul_quant_group128
    #        gu   m  I    ld_gu q   ldq  s   ld_s h  ldh
    assert f(A16, -1, 128, 256, A16, 128, A16, 1, None, 0, None) == INVALID
    assert f(A16, 4, 100, 256, A16, 128, A16, 4, None, 0, None) == SHAPE
    assert f(A16, 4, 128, 255, A16, 128, A16, 4, None, 0, None) == INVALID       # ld_gu < 2I
    assert f(A16, 4, 128, 256, A16, 120, A16, 4, None, 0, None) == INVALID       # ldq < I
    assert f(A16, 4, 128, 256, A16, 128, A16, 3, None, 0, None) == INVALID       # ld_scale < m
    assert f(A16, 4, 128, 256, A16, 128, A16, 4, A16, 64, None) == INVALID       # ldh < I
    assert f(None, 4, 128, 256, A16, 128, A16, 4, None, 0, None) == INVALID
    assert f(A16 + 8, 4, 128, 256, A16, 128, A16, 4, None, 0, None) == MISALIGNED
    assert f(A16, 4, 128, 260, A16, 128, A16, 4, None, 0, None) == MISALIGNED    # ld_gu % 8
    assert f(A16, 4, 128, 256, A16, 136, A16, 4, None, 0, None) == MISALIGNED    # ldq % 16
    assert f(A16, 4, 128, 256, A16, 128, A16, 4, A16 + 8, 128, None) == MISALIGNED
    assert f(A16, 4, 128, 256, A16, 128, A16, 4, A16, 132, None) == MISALIGNED   # ldh % 8
    assert f(None, 0, 128, 256, None, 128, None, 0, None, 0, None) == OK


def test_gather_rows_argument_errors(lib):
    f = lib.fp8rl_gather_rows_fp8
    #        qs  ldq  ss  ld_ss S  idx  R  k    qd  ldqd sd  ld_sd
    assert f(A16, 128, A16, 8, 8, A16, -1, 128, A16, 128, A16, 8, None) == INVALID
    assert f(A16, 128, A16, 8, 8, A16, 4, 100, A16, 128, A16, 8, None) == SHAPE
    assert f(A16, 128, A16, 8, 0, A16, 4, 128, A16, 128, A16, 8, None) == INVALID   # rows from nothing
    assert f(A16, 128, A16, 7, 8, A16, 4, 128, A16, 128, A16, 8, None) == INVALID   # ld_s_src < S
    assert f(A16, 128, A16, 8, 8, A16, 4, 128, A16, 128, A16, 3, None) == INVALID   # ld_s_dst < R
    assert f(A16, 120, A16, 8, 8, A16, 4, 128, A16, 128, A16, 8, None) == INVALID   # ldq_src < k
    assert f(A16, 128, A16, 8, 8, None, 4, 128, A16, 128, A16, 8, None) == INVALID
    assert f(A16 + 8, 128, A16, 8, 8, A16, 4, 128, A16, 128, A16, 8, None) == MISALIGNED
    assert f(A16, 136, A16, 8, 8, A16, 4, 128, A16, 128, A16, 8, None) == MISALIGNED
    assert f(A16, 128, A16, 8, 8, A16 + 2, 4, 128, A16, 128, A16, 8, None) == MISALIGNED
    assert f(A16, 128, A16 + 2, 8, 8, A16, 4, 128, A16, 128, A16, 8, None) == MISALIGNED
    assert f(None, 128, None, 0, 0, None, 0, 128, None, 128, None, 0, None) == OK


def test_ue8m0_entry_points_validate_like_the_fp32_ones(lib):
    """The power-of-two variants share the argument checks of their fp32 counterparts."""
    wq = lib.fp8rl_quant_weight_block128_ue8m0
    assert wq(A16, 128, 200, 200, A16, 208, A16, None) == SHAPE
    assert wq(A4, 128, 128, 128, A16, 128, A16, None) == MISALIGNED
    assert wq(None, 128, 128, 128, A16, 128, A16, None) == INVALID
    assert wq(None, 0, 0, 0, None, 0, None, None) == OK
    aq = lib.fp8rl_quant_act_token_group128_ue8m0
    assert aq(A16, 4, 128, 128, A16, 128, A16, 3, None) == INVALID
    assert aq(A16, 4, 100, 128, A16, 128, A16, 4, None) == SHAPE
    assert aq(A16, 4, 128, 128, A16 + 8, 128, A16, 4, None) == MISALIGNED
    g = lib.fp8rl_gemm_w8a8_block_ue8m0
    assert g(A16, 128, A16, 8, A16, 128, A16, A16, 128, 8, 192, 128, None) == SHAPE
    assert g(A16, 128, A16, 7, A16, 128, A16, A16, 128, 8, 128, 128, None) == INVALID
    assert g(A16 + 8, 128, A16, 8, A16, 128, A16, A16, 128, 8, 128, 128, None) == MISALIGNED
    assert g(None, 128, None, 0, None, 128, None, None, 128, 0, 128, 128, None) == OK
    gg = lib.fp8rl_grouped_gemm_w8a8_block_ue8m0
    assert gg(A16, A16, 8, A16, A16, A16, 0, 8, A16, 128, 128, None) == INVALID
    assert gg(A16, A16, 8, A16, A16, A16, 1025, 8, A16, 128, 128, None) == SHAPE
    assert gg(A16, A16, 8, A4, A16, A16, 2, 8, A16, 128, 128, None) == MISALIGNED
    assert gg(None, None, 0, None, None, None, 2, 0, None, 128, 128, None) == OK


def test_tis_argument_errors(lib):
    f = lib.fp8rl_tis_weights_kl
    size = lib.fp8rl_tis_workspace_size
    size.restype = ctypes.c_int64
    size.argtypes = [ctypes.c_int64]
    f.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int64, ctypes.c_float] + [ctypes.c_void_p] * 3 + \
        [ctypes.c_int64, ctypes.c_void_p]
    assert size(0) == 32 and size(-1) == 0 and size(1000) == 32 and size(1 << 30) == 2048 * 32
    ws = size(1000)
    #        lt   lr  mask   n    C    w    stats ws   bytes
    assert f(A16, A16, None, -1, 2.0, A16, A16, A16, ws, None) == INVALID
    assert f(A16, A16, None, 1000, 0.0, A16, A16, A16, ws, None) == INVALID          # C must be > 0
    assert f(A16, A16, None, 1000, float("inf"), A16, A16, A16, ws, None) == INVALID
    assert f(A16, A16, None, 1000, float("nan"), A16, A16, A16, ws, None) == INVALID
    assert f(None, A16, None, 1000, 2.0, A16, A16, A16, ws, None) == INVALID
    assert f(A16, A16, None, 1000, 2.0, A16, None, A16, ws, None) == INVALID          # no stats
    assert f(A16, A16, None, 1000, 2.0, A16, A16, None, ws, None) == INVALID          # no workspace
    assert f(A16, A16, None, 1000, 2.0, A16, A16, A16, ws - 8, None) == INVALID       # short workspace
    assert f(A16 + 2, A16, None, 1000, 2.0, A16, A16, A16, ws, None) == MISALIGNED
    assert f(A16, A16 + 4, None, 1000, 2.0, A16, A16, A16, ws, None) == MISALIGNED   # 16-byte loads
    assert f(A16, A16, A16 + 2, 1000, 2.0, A16, A16, A16, ws, None) == MISALIGNED    # mask 4-byte
    assert f(A16, A16, None, 1000, 2.0, A16, A16 + 4, A16, ws, None) == MISALIGNED    # stats 8-byte
    assert f(A16, A16, None, 1000, 2.0, A16, A16, A16 + 4, ws, None) == MISALIGNED


def test_kv_calibrate_argument_errors(lib):
    size = lib.fp8rl_kv_calibrate_workspace_size
    f = lib.fp8rl_kv_calibrate_scale
    assert size(-1) == 0 and size(0) == 4 and size(100000) == 49 * 4 and size(1 << 40) == 1024 * 4
    ws = size(100000)
    #        x    n       scale ws   bytes
    assert f(A16, -1, A16, A16, ws, None) == INVALID
    assert f(None, 100000, A16, A16, ws, None) == INVALID
    assert f(A16, 100000, None, A16, ws, None) == INVALID
    assert f(A16, 100000, A16, None, ws, None) == INVALID
    assert f(A16, 100000, A16, A16, ws - 4, None) == INVALID                  # short workspace
    assert f(A16, 1 << 46, A16, A16, 1 << 20, None) == SHAPE
    assert f(A16 + 8, 100000, A16, A16, ws, None) == MISALIGNED               # 16-byte loads
    assert f(A16, 100000, A16 + 2, A16, ws, None) == MISALIGNED
    assert f(A16, 100000, A16, A16 + 2, ws, None) == MISALIGNED


def test_kv_cache_write_argument_errors(lib):
    f = lib.fp8rl_kv_cache_write_fp8
    #        k    v    T   kvh hd   slots nb  ks   vs   kc   vc
    assert f(A16, A16, -1, 8, 128, A16, 40, A16, A16, A16, A16, None) == INVALID
    assert f(A16, A16, 300, 0, 128, A16, 40, A16, A16, A16, A16, None) == INVALID
    assert f(A16, A16, 300, 8, 128, A16, -1, A16, A16, A16, A16, None) == INVALID
    assert f(A16, A16, 300, 8, 64, A16, 40, A16, A16, A16, A16, None) == SHAPE        # head_dim 128 only
    assert f(A16, A16, 300, 1025, 128, A16, 40, A16, A16, A16, A16, None) == SHAPE
    assert f(A16, A16, 1 << 31, 8, 128, A16, 40, A16, A16, A16, A16, None) == SHAPE
    assert f(A16, A16, 1 << 27, 1024, 128, A16, 40, A16, A16, A16, A16, None) == SHAPE  # grid of 2^31 threads
    assert f(A16, A16, 300, 8, 128, None, 40, A16, A16, A16, A16, None) == INVALID
    assert f(A16, A16, 300, 8, 128, A16, 40, A16, None, A16, A16, None) == INVALID
    assert f(A16 + 8, A16, 300, 8, 128, A16, 40, A16, A16, A16, A16, None) == MISALIGNED
    assert f(A16, A16, 300, 8, 128, A16 + 4, 40, A16, A16, A16, A16, None) == MISALIGNED
    assert f(A16, A16, 300, 8, 128, A16, 40, A16, A16, A16, A16 + 4, None) == MISALIGNED
    assert f(None, None, 0, 8, 128, None, 40, None, None, None, None, None) == OK      # no tokens: no-op


def test_attention_decode_argument_errors(lib):
    size = lib.fp8rl_attention_decode_workspace_size
    assert size(2, 8, 2, 100) > 0
    assert size(-1, 8, 2, 100) == 0 and size(2, 8, 3, 100) == 0 and size(2, 1, 2, 100) == 0 and size(2, 8, 2, -1) == 0
    ws = size(2, 8, 2, 100)
    f = lib.fp8rl_attention_decode_fp8kv
    g = lib.fp8rl_attention_decode_bf16kv

    def call(batch=2, qh=8, kvh=2, hd=128, nb=10, max_blocks=8, max_seq=100, ks=A16, sm=0.088, q=A16, wsb=ws,
             table=A16, out=A16):
        #        q  kc   vc   nb  table max_blocks seq_lens batch qh kvh hd max_seq ks vs sm out ws bytes
        return f(q, A16, A16, nb, table, max_blocks, A16, batch, qh, kvh, hd, max_seq, ks, A16, sm, out, A16, wsb,
                 None)

    assert call(batch=-1) == INVALID
    assert call(sm=0.0) == INVALID and call(sm=float("nan")) == INVALID and call(sm=float("inf")) == INVALID
    assert call(hd=64) == SHAPE
    assert call(qh=12, kvh=4) == SHAPE                    # group of 3
    assert call(qh=32, kvh=2) == SHAPE                    # group of 16
    assert call(qh=6, kvh=4) == SHAPE                     # not a multiple
    assert call(batch=65536) == SHAPE
    assert call(max_seq=1 << 30) == SHAPE
    assert call(ks=None) == INVALID                       # FP8 cache needs its scales
    assert call(table=None) == INVALID and call(out=None) == INVALID
    assert call(nb=0) == INVALID
    assert call(max_blocks=6) == INVALID                  # 6 * 16 < 100
    assert call(wsb=ws - 16) == INVALID
    assert call(q=A16 + 8) == MISALIGNED
    assert call(out=A16 + 2) == MISALIGNED
    assert call(batch=0, q=None, table=None, out=None) == OK
    #        q    kc   vc   nb  table max_b seq  batch qh kvh hd   max_seq sm   out  ws   bytes
    assert g(A16, A16, A16, 10, A16, 8, A16, 2, 8, 2, 64, 100, 0.088, A16, A16, ws, None) == SHAPE
    assert g(A16, A16, A16, 10, A16, 8, A16, 2, 8, 2, 128, 100, 0.088, A16, None, ws, None) == INVALID


def test_dma_probe_rejects_regions_outside_the_buffer():
    """The operand-stream probe checks on the host that every workgroup's region
    lies inside the source buffer (and its other sizes) before launching."""
    import paper_2601_18150_amd as fp8rl
    probe = ctypes.CDLL(os.path.join(os.path.dirname(fp8rl.LIB_PATH), "libfp8rl_probe.so"))
    fn = probe.fp8rl_probe_dma_rate
    fn.argtypes = [ctypes.c_void_p, ctypes.c_longlong, ctypes.c_longlong, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                   ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    good = dict(src=A16, src_bytes=1 << 30, region=1 << 20, blocks=256, waves=8, inflight=8, to_lds=1, iters=4,
                sink=A16, clk=A16)
    bad = [dict(src_bytes=(1 << 28) - 1),        # 256 regions of 1 MiB need 256 MiB
           dict(region=1000), dict(region=512), dict(region=1 << 31), dict(blocks=0), dict(waves=0),
           dict(waves=17), dict(inflight=3), dict(inflight=16), dict(iters=0), dict(src=None), dict(sink=None),
           dict(clk=None), dict(src_bytes=-1)]
    for b in bad:
        a = dict(good, **b)
        assert fn(a["src"], a["src_bytes"], a["region"], a["blocks"], a["waves"], a["inflight"], a["to_lds"],
                  a["iters"], a["sink"], a["clk"], None) == 1, b


def test_inner_loop_probe_rejects_bad_arguments():
    import paper_2601_18150_amd as fp8rl
    probe = ctypes.CDLL(os.path.join(os.path.dirname(fp8rl.LIB_PATH), "libfp8rl_probe.so"))
    fn = probe.fp8rl_probe_mfma_loop
    fn.argtypes = [ctypes.c_int] * 5 + [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    good = [0, 1, 1, 256, 10, A16, A16, None]
    for i, bad in [(0, 2), (0, -1), (1, 2), (2, 2), (3, 0), (4, 0), (5, None), (6, None)]:
        a = list(good)
        a[i] = bad
        assert fn(*a) == 1, (i, bad)


def test_binding_rejects_cpu_tensors():
    import torch
    import paper_2601_18150_amd as fp8rl
    w = torch.zeros(128, 128, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        fp8rl.fp8rl_quant_weight_block128(w)


def test_argument_validation_under_address_and_ub_sanitizers(tmp_path):
    """The C ABI's validation paths built for the host with AddressSanitizer and
    UndefinedBehaviorSanitizer (tests/host/abi_asan.cpp: csrc/api.cpp with stub
    launchers): every invalid call returns its status without launching, every
    valid one launches once, and the sanitizers report nothing."""
    import shutil
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = tmp_path / "abi_asan"
    src = os.path.join(ROOT, "tests", "host", "abi_asan.cpp")
    build = subprocess.run([gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                            "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                            f"-I{os.path.join(ROOT, 'include')}", src, "-o", str(exe)],
                           capture_output=True, text=True)
    if build.returncode != 0 and "asan" in (build.stderr or "").lower():
        pytest.skip("sanitizer runtime not available: " + build.stderr[-200:])
    assert build.returncode == 0, build.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-2000:]
    assert run.stdout.startswith("ok"), run.stdout
