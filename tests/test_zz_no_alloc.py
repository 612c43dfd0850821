"""The no-allocation GEMM entry point (static split-K scratch) against the
workspace entry point and the fp64 oracle, through the C ABI.

Two calls in a row on one GPU share the library's static array: the second,
smaller call must not see the first call's partial sums."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import cref, gemm
from tests.gpu_util import announce, need_gpu, u16

pytestmark = pytest.mark.gpu


def operands(m, n, k, seed):
    rng = np.random.default_rng(seed)
    a = torch.from_numpy(rng.standard_normal((m, k)).astype(np.float32)).to(torch.bfloat16)
    w = torch.from_numpy((rng.standard_normal((n, k)) * 0.02).astype(np.float32)).to(torch.bfloat16)
    qa, sa = cref.quant_act_token_group128(u16(a))
    qw, sw = cref.quant_weight_block128(u16(w))
    return qa, sa, qw, sw


def test_noalloc_matches_workspace_entry_point_twice():
    need_gpu()
    import paper_2601_18150_amd as fp8rl
    lib = ctypes.CDLL(fp8rl.LIB_PATH)
    P, I = ctypes.c_void_p, ctypes.c_int64
    noalloc = lib.fp8rl_gemm_w8a8_block_noalloc
    noalloc.argtypes = [P, I, P, I, P, I, P, P, I, I, I, I, P]
    with_ws = lib.fp8rl_gemm_w8a8_block_ws
    with_ws.argtypes = [P, I, P, I, P, I, P, P, I, I, I, I, P, I, P]
    wsize = lib.fp8rl_gemm_w8a8_block_workspace_size
    wsize.argtypes = [I, I, I]
    wsize.restype = I
    stream = torch.cuda.current_stream().cuda_stream
    # the Qwen3-8B decode down projection (4 K ranges, the whole 16 MiB), then a smaller split shape
    for m, n, k, seed in [(256, 4096, 12288, 1), (100, 256, 2048, 2)]:
        announce(f"noalloc gemm m={m} n={n} k={k}")
        need = wsize(m, n, k)
        assert need > 0, "the case is meant to split K"
        qa, sa, qw, sw = operands(m, n, k, seed)
        d = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in (qa, sa, qw, sw)]
        y0 = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device="cuda")
        y1 = torch.full((m, n), float("nan"), dtype=torch.bfloat16, device="cuda")
        ws = torch.full((need // 4,), float("nan"), dtype=torch.float32, device="cuda")
        args = (d[0].data_ptr(), k, d[1].data_ptr(), m, d[2].data_ptr(), k, d[3].data_ptr())
        assert noalloc(*args, y0.data_ptr(), n, m, n, k, stream) == 0
        assert with_ws(*args, y1.data_ptr(), n, m, n, k, ws.data_ptr(), need, stream) == 0
        torch.cuda.synchronize()
        assert torch.equal(y0.view(torch.int16), y1.view(torch.int16)), "not the workspace entry point's bits"
        ok, worst, _ = gemm.tolerance_check(y0.float().cpu().numpy(), gemm.gemm_ref_fp64(qa, sa, qw, sw))
        assert ok, f"outside the tolerance (worst {worst:.3f})"
