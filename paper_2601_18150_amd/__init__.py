"""Python binding of libfp8rl -- blockwise FP8 (E4M3) W8A8 linear layer on MI355X.

Argument marshalling only: every function below checks tensor shapes, dtypes
and devices, allocates outputs with torch when they are not supplied, and
calls the C entry point of the same name (include/fp8rl.h) on the current
torch stream.  All arithmetic runs in the HIP kernels of libfp8rl.so; there is
no CPU fallback: the library is loaded on first use (or by ``load()``) and a
missing or unloadable library raises ImportError.

Paper: "FP8-RL", arXiv 2601.18150 -- section 2.1.1 (blockwise E4M3 weights with
128x128 fp32 block scales, Eq. (1); dynamic per-token 1x128 activation
scales), section 2.1.2 (weights re-quantised at every RL step), section 2.1.4
(FP8 GEMM for the W8A8 linear layers, dense and MoE experts).
"""
from __future__ import annotations

import ctypes
import os

import torch  # loads torch's HIP runtime first, so libfp8rl binds to that same runtime

__all__ = [
    "LIB_PATH", "Fp8rlError", "load",
    "fp8rl_quant_weight_block128", "fp8rl_quant_weight_block128_batched", "fp8rl_quant_act_token_group128",
    "fp8rl_gemm_w8a8_block", "fp8rl_grouped_gemm_w8a8_block", "fp8rl_grouped_gemm_w8a8_block_gathered",
    "fp8rl_gemm_w8a8_block_workspace_size", "fp8rl_gemm_w8a8_block_ws", "fp8rl_gemm_w8a8_block_noalloc",
    "fp8rl_quant_weight_block128_ue8m0", "fp8rl_quant_act_token_group128_ue8m0",
    "fp8rl_gemm_w8a8_block_ue8m0", "fp8rl_grouped_gemm_w8a8_block_ue8m0",
    "fp8rl_silu_mul_quant_group128", "fp8rl_gather_rows_fp8",
    "fp8rl_tis_workspace_size", "fp8rl_tis_weights_kl",
    "fp8rl_kv_calibrate_scale", "fp8rl_kv_cache_write_fp8", "fp8rl_attention_decode_workspace_size",
    "fp8rl_attention_decode_fp8kv", "fp8rl_attention_decode_bf16kv",
    "fp8rl_status_string", "fp8rl_version",
    "quant_weight_block128", "quant_act_token_group128", "gemm_w8a8_block",
    "grouped_gemm_w8a8_block", "silu_mul_quant_group128", "gather_rows_fp8", "linear_w8a8",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfp8rl.so")

_STATUS = {0: "FP8RL_OK", 1: "FP8RL_ERR_INVALID_ARG", 2: "FP8RL_ERR_UNSUPPORTED_SHAPE",
           3: "FP8RL_ERR_MISALIGNED", 4: "FP8RL_ERR_HIP", 5: "FP8RL_ERR_SCRATCH_LIMIT"}


class Fp8rlError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} returned {status} ({_STATUS.get(status, 'unknown')})")
        self.status = status


def _hip_runtimes_mapped():
    try:
        with open("/proc/self/maps") as f:
            paths = {ln.split()[-1] for ln in f if "libamdhip64" in ln}
        return sorted(p for p in paths if p.startswith("/"))
    except OSError:
        return []


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2601_18150_amd.build` "
                          "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    P, I = ctypes.c_void_p, ctypes.c_int64
    sig = {
        "fp8rl_quant_weight_block128": [P, I, I, I, P, I, P, P],
        "fp8rl_quant_act_token_group128": [P, I, I, I, P, I, P, I, P],
        "fp8rl_gemm_w8a8_block": [P, I, P, I, P, I, P, P, I, I, I, I, P],
        "fp8rl_grouped_gemm_w8a8_block": [P, P, I, P, P, P, I, I, P, I, I, P],
        "fp8rl_grouped_gemm_w8a8_block_gathered": [P, I, P, I, I, P, P, P, P, I, I, P, I, I, P],
        "fp8rl_gemm_w8a8_block_ws": [P, I, P, I, P, I, P, P, I, I, I, I, P, I, P],
        "fp8rl_gemm_w8a8_block_noalloc": [P, I, P, I, P, I, P, P, I, I, I, I, P],
        "fp8rl_quant_weight_block128_ue8m0": [P, I, I, I, P, I, P, P],
        "fp8rl_quant_act_token_group128_ue8m0": [P, I, I, I, P, I, P, I, P],
        "fp8rl_gemm_w8a8_block_ue8m0": [P, I, P, I, P, I, P, P, I, I, I, I, P],
        "fp8rl_grouped_gemm_w8a8_block_ue8m0": [P, P, I, P, P, P, I, I, P, I, I, P],
        "fp8rl_silu_mul_quant_group128": [P, I, I, I, P, I, P, I, P, I, P],
        "fp8rl_tis_weights_kl": [P, P, P, I, ctypes.c_float, P, P, P, I, P],
        "fp8rl_kv_calibrate_scale": [P, I, P, P, I, P],
        "fp8rl_kv_cache_write_fp8": [P, P, I, I, I, P, I, P, P, P, P, P],
        "fp8rl_attention_decode_fp8kv": [P, P, P, I, P, I, P, I, I, I, I, I, P, P, ctypes.c_float, P, P, I, P],
        "fp8rl_attention_decode_bf16kv": [P, P, P, I, P, I, P, I, I, I, I, I, ctypes.c_float, P, P, I, P],
        "fp8rl_gather_rows_fp8": [P, I, P, I, I, P, I, I, P, I, P, I, P],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.fp8rl_quant_weight_block128_batched.argtypes = [P, I, P]
    lib.fp8rl_quant_weight_block128_batched.restype = ctypes.c_int
    lib.fp8rl_tis_workspace_size.argtypes = [I]
    lib.fp8rl_tis_workspace_size.restype = ctypes.c_int64
    lib.fp8rl_kv_calibrate_workspace_size.argtypes = [I]
    lib.fp8rl_kv_calibrate_workspace_size.restype = ctypes.c_int64
    lib.fp8rl_attention_decode_workspace_size.argtypes = [I, I, I, I]
    lib.fp8rl_attention_decode_workspace_size.restype = ctypes.c_int64
    lib.fp8rl_gemm_w8a8_block_workspace_size.argtypes = [I, I, I]
    lib.fp8rl_gemm_w8a8_block_workspace_size.restype = ctypes.c_int64
    lib.fp8rl_status_string.argtypes = [ctypes.c_int]
    lib.fp8rl_status_string.restype = ctypes.c_char_p
    lib.fp8rl_version.argtypes = []
    lib.fp8rl_version.restype = ctypes.c_int
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes mapped in this process: {runtimes}")
    return lib


_lib = None


def load():
    """Load libfp8rl.so (once) and return the ctypes handle."""
    global _lib
    if _lib is None:
        _lib = _load()
    return _lib


def _check(name: str, status: int):
    if status != 0:
        raise Fp8rlError(name, status)


def _stream(stream=None) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dev(*ts):
    dev = None
    for t in ts:
        if not t.is_cuda:
            raise ValueError("fp8rl tensors must live on a HIP device")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("fp8rl tensors must share one device")
    return dev


def _ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-D row-major tensor with unit column stride")
    return t.stride(0) if t.size(0) > 1 else max(t.stride(0), t.size(1))


def _u8(t: torch.Tensor) -> torch.Tensor:
    if t.dtype == torch.uint8:
        return t
    if t.dtype == torch.float8_e4m3fn:
        return t.view(torch.uint8)
    raise TypeError(f"expected uint8 / float8_e4m3fn codes, got {t.dtype}")


# ---------------------------------------------------------------------------
# Entry points with the C names
# ---------------------------------------------------------------------------
def fp8rl_status_string(status: int) -> str:
    return load().fp8rl_status_string(int(status)).decode()


def fp8rl_version() -> int:
    return int(load().fp8rl_version())


def fp8rl_quant_weight_block128(w: torch.Tensor, q: torch.Tensor | None = None,
                                scale: torch.Tensor | None = None, stream=None):
    """bf16 weight [N][K] -> (E4M3 codes uint8 [N][K], fp32 scales [N/128][K/128])."""
    return _quant_weight("fp8rl_quant_weight_block128", w, q, scale, stream)


class WeightJob(ctypes.Structure):
    """fp8rl_weight_job of include/fp8rl.h (device pointers, sizes in elements)."""
    _fields_ = [("w", ctypes.c_void_p), ("n", ctypes.c_int64), ("k", ctypes.c_int64), ("ldw", ctypes.c_int64),
                ("q", ctypes.c_void_p), ("ldq", ctypes.c_int64), ("scale", ctypes.c_void_p)]


def fp8rl_quant_weight_block128_batched(ws, qs=None, scales=None, stream=None):
    """Many bf16 weights [N_i][K_i] -> [(codes, scales)] in one pass (up to 64 matrices per launch);
    each result is bit-identical to fp8rl_quant_weight_block128 of that matrix."""
    ws = list(ws)
    qs = list(qs) if qs is not None else [None] * len(ws)
    scales = list(scales) if scales is not None else [None] * len(ws)
    if len(qs) != len(ws) or len(scales) != len(ws):
        raise ValueError("ws, qs and scales must have the same length")
    jobs = (WeightJob * max(len(ws), 1))()
    out = []
    for i, (w, q, sc) in enumerate(zip(ws, qs, scales)):
        if w.dtype != torch.bfloat16 or w.dim() != 2:
            raise TypeError("every w must be a 2-D bfloat16 tensor")
        n, k = w.shape
        if q is None:
            q = torch.empty((n, k), dtype=torch.uint8, device=w.device)
        if sc is None:
            sc = torch.empty((n // 128, k // 128), dtype=torch.float32, device=w.device)
        q = _u8(q)
        _dev(w, q, sc)
        if sc.dtype != torch.float32 or not sc.is_contiguous() or sc.numel() < (n // 128) * (k // 128):
            raise ValueError("scale must be a contiguous fp32 tensor of [N/128][K/128] elements")
        jobs[i] = WeightJob(w.data_ptr(), n, k, _ld(w), q.data_ptr(), _ld(q), sc.data_ptr())
        out.append((q, sc))
    if ws:
        _dev(*ws)
    st = load().fp8rl_quant_weight_block128_batched(ctypes.addressof(jobs), len(ws), _stream(stream))
    _check("fp8rl_quant_weight_block128_batched", st)
    return out


def fp8rl_quant_weight_block128_ue8m0(w: torch.Tensor, q: torch.Tensor | None = None,
                                      scale: torch.Tensor | None = None, stream=None):
    """As fp8rl_quant_weight_block128 with power-of-two (UE8M0) scales 2^k, stored as fp32."""
    return _quant_weight("fp8rl_quant_weight_block128_ue8m0", w, q, scale, stream)


def _quant_weight(name, w, q, scale, stream):
    if w.dtype != torch.bfloat16 or w.dim() != 2:
        raise TypeError("w must be a 2-D bfloat16 tensor")
    n, k = w.shape
    if q is None:
        q = torch.empty((n, k), dtype=torch.uint8, device=w.device)
    if scale is None:
        scale = torch.empty((n // 128, k // 128), dtype=torch.float32, device=w.device)
    q = _u8(q)
    _dev(w, q, scale)
    if scale.dtype != torch.float32 or not scale.is_contiguous() or scale.numel() < (n // 128) * (k // 128):
        raise ValueError("scale must be a contiguous fp32 tensor of [N/128][K/128] elements")
    st = getattr(load(), name)(w.data_ptr(), n, k, _ld(w), q.data_ptr(), _ld(q), scale.data_ptr(), _stream(stream))
    _check(name, st)
    return q, scale


def fp8rl_quant_act_token_group128(a: torch.Tensor, q: torch.Tensor | None = None,
                                   scale: torch.Tensor | None = None, ld_scale: int | None = None,
                                   stream=None):
    """bf16 activations [M][K] -> (E4M3 codes uint8 [M][K], fp32 scales [K/128][ld_scale])."""
    return _quant_act("fp8rl_quant_act_token_group128", a, q, scale, ld_scale, stream)


def fp8rl_quant_act_token_group128_ue8m0(a: torch.Tensor, q: torch.Tensor | None = None,
                                         scale: torch.Tensor | None = None, ld_scale: int | None = None,
                                         stream=None):
    """As fp8rl_quant_act_token_group128 with power-of-two (UE8M0) scales 2^k, stored as fp32."""
    return _quant_act("fp8rl_quant_act_token_group128_ue8m0", a, q, scale, ld_scale, stream)


def _quant_act(name, a, q, scale, ld_scale, stream):
    if a.dtype != torch.bfloat16 or a.dim() != 2:
        raise TypeError("a must be a 2-D bfloat16 tensor")
    m, k = a.shape
    if scale is not None and ld_scale is None:
        ld_scale = scale.stride(0) if scale.dim() == 2 else m
    if ld_scale is None:
        ld_scale = m
    if q is None:
        q = torch.empty((m, k), dtype=torch.uint8, device=a.device)
    if scale is None:
        scale = torch.empty((k // 128, ld_scale), dtype=torch.float32, device=a.device)
    q = _u8(q)
    _dev(a, q, scale)
    if scale.dtype != torch.float32 or scale.numel() < (k // 128) * ld_scale and m > 0:
        raise ValueError("scale must be fp32 with at least [K/128][ld_scale] elements")
    st = getattr(load(), name)(a.data_ptr(), m, k, _ld(a) if m else k, q.data_ptr(), _ld(q) if m else k,
                               scale.data_ptr(), ld_scale, _stream(stream))
    _check(name, st)
    return q, scale


def _dense_args(qa, sa, qw, sw, y):
    qa, qw = _u8(qa), _u8(qw)
    m, k = qa.shape
    n, k2 = qw.shape
    if k != k2:
        raise ValueError("K mismatch")
    if sa.dtype != torch.float32 or sw.dtype != torch.float32:
        raise TypeError("scales must be fp32")
    if sa.dim() != 2 or sa.size(0) != k // 128 or sa.stride(1) != 1 or sa.size(1) < m:
        raise ValueError("sa must be [K/128][ld >= M] with unit stride")
    if not sw.is_contiguous() or sw.numel() != (n // 128) * (k // 128):
        raise ValueError("sw must be contiguous [N/128][K/128]")
    if y is None:
        y = torch.empty((m, n), dtype=torch.bfloat16, device=qa.device)
    if y.dtype != torch.bfloat16 or tuple(y.shape) != (m, n):
        raise ValueError("y must be bf16 [M][N]")
    _dev(qa, sa, qw, sw, y)
    return qa, qw, y, m, n, k


def fp8rl_gemm_w8a8_block(qa: torch.Tensor, sa: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor,
                          y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """y[M][N] bf16 = blockwise-scaled FP8 product of qa [M][K] (scales sa [K/128][>=M])
    and qw [N][K] (scales sw [N/128][K/128])."""
    return _gemm("fp8rl_gemm_w8a8_block", qa, sa, qw, sw, y, stream)


def fp8rl_gemm_w8a8_block_ue8m0(qa: torch.Tensor, sa: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor,
                                y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """As fp8rl_gemm_w8a8_block for power-of-two scales (from the _ue8m0 quantisers), which the
    MX-scaled MFMA applies in hardware."""
    return _gemm("fp8rl_gemm_w8a8_block_ue8m0", qa, sa, qw, sw, y, stream)


def _gemm(name, qa, sa, qw, sw, y, stream):
    qa, qw, y, m, n, k = _dense_args(qa, sa, qw, sw, y)
    if m == 0:
        return y
    st = getattr(load(), name)(qa.data_ptr(), _ld(qa), sa.data_ptr(), sa.stride(0), qw.data_ptr(), _ld(qw),
                               sw.data_ptr(), y.data_ptr(), _ld(y), m, n, k, _stream(stream))
    _check(name, st)
    return y


def fp8rl_gemm_w8a8_block_workspace_size(m: int, n: int, k: int) -> int:
    """Bytes of workspace fp8rl_gemm_w8a8_block_ws splits K with for this shape (0: no split)."""
    return int(load().fp8rl_gemm_w8a8_block_workspace_size(m, n, k))


def fp8rl_gemm_w8a8_block_ws(qa: torch.Tensor, sa: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor,
                             workspace: torch.Tensor, y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """fp8rl_gemm_w8a8_block with a caller-owned device workspace (any dtype, contiguous) that
    lets shapes with too few output tiles split K; see the C header for the contract."""
    qa, qw, y, m, n, k = _dense_args(qa, sa, qw, sw, y)
    if not workspace.is_contiguous():
        raise ValueError("workspace must be contiguous")
    _dev(qa, workspace)
    if m == 0:
        return y
    nbytes = workspace.numel() * workspace.element_size()
    st = load().fp8rl_gemm_w8a8_block_ws(qa.data_ptr(), _ld(qa), sa.data_ptr(), sa.stride(0), qw.data_ptr(),
                                      _ld(qw), sw.data_ptr(), y.data_ptr(), _ld(y), m, n, k,
                                      workspace.data_ptr(), nbytes, _stream(stream))
    _check("fp8rl_gemm_w8a8_block_ws", st)
    return y


def fp8rl_gemm_w8a8_block_noalloc(qa: torch.Tensor, sa: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor,
                                  y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """fp8rl_gemm_w8a8_block_ws with the split-K partial sums in the library's static
    device scratch instead of a workspace (the C call allocates nothing; pass y to
    keep the wrapper from allocating the output)."""
    qa, qw, y, m, n, k = _dense_args(qa, sa, qw, sw, y)
    if m == 0:
        return y
    st = load().fp8rl_gemm_w8a8_block_noalloc(qa.data_ptr(), _ld(qa), sa.data_ptr(), sa.stride(0), qw.data_ptr(),
                                              _ld(qw), sw.data_ptr(), y.data_ptr(), _ld(y), m, n, k, _stream(stream))
    _check("fp8rl_gemm_w8a8_block_noalloc", st)
    return y


def fp8rl_grouped_gemm_w8a8_block(qa: torch.Tensor, sa: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor,
                                  group_offsets: torch.Tensor, y: torch.Tensor | None = None,
                                  stream=None) -> torch.Tensor:
    """Per expert e: y[off_e:off_e+1] = blockwise FP8 product with qw[e], sw[e].

    qa [R][K] codes grouped by expert; sa [K/128][ld >= R]; qw [G][N][K];
    sw [G][N/128][K/128]; group_offsets int32 [G+1] on the device.
    """
    return _grouped("fp8rl_grouped_gemm_w8a8_block", qa, sa, qw, sw, group_offsets, y, stream)


def fp8rl_grouped_gemm_w8a8_block_ue8m0(qa: torch.Tensor, sa: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor,
                                        group_offsets: torch.Tensor, y: torch.Tensor | None = None,
                                        stream=None) -> torch.Tensor:
    """As fp8rl_grouped_gemm_w8a8_block for power-of-two scales (MX-scaled MFMA)."""
    return _grouped("fp8rl_grouped_gemm_w8a8_block_ue8m0", qa, sa, qw, sw, group_offsets, y, stream)


def _grouped(name, qa, sa, qw, sw, group_offsets, y, stream):
    qa, qw = _u8(qa), _u8(qw)
    r, k = qa.shape
    g, n, k2 = qw.shape
    if k != k2:
        raise ValueError("K mismatch")
    if not qa.is_contiguous() or not qw.is_contiguous() or not sw.is_contiguous():
        raise ValueError("qa, qw and sw must be contiguous")
    if sw.numel() != g * (n // 128) * (k // 128) or sw.dtype != torch.float32:
        raise ValueError("sw must be fp32 [G][N/128][K/128]")
    if sa.dtype != torch.float32 or sa.dim() != 2 or sa.size(0) != k // 128 or sa.stride(1) != 1 or sa.size(1) < r:
        raise ValueError("sa must be fp32 [K/128][ld >= R]")
    if group_offsets.dtype != torch.int32 or group_offsets.numel() != g + 1 or not group_offsets.is_contiguous():
        raise ValueError("group_offsets must be a contiguous int32 tensor of G+1 entries")
    if y is None:
        y = torch.empty((r, n), dtype=torch.bfloat16, device=qa.device)
    if y.dtype != torch.bfloat16 or tuple(y.shape) != (r, n) or not y.is_contiguous():
        raise ValueError("y must be contiguous bf16 [R][N]")
    _dev(qa, sa, qw, sw, group_offsets, y)
    if r == 0:
        return y
    st = getattr(load(), name)(qa.data_ptr(), sa.data_ptr(), sa.stride(0), qw.data_ptr(), sw.data_ptr(),
                               group_offsets.data_ptr(), g, r, y.data_ptr(), n, k, _stream(stream))
    _check(name, st)
    return y


def fp8rl_grouped_gemm_w8a8_block_gathered(qa: torch.Tensor, sa: torch.Tensor, row_index: torch.Tensor,
                                           qw: torch.Tensor, sw: torch.Tensor, group_offsets: torch.Tensor,
                                           y: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The grouped product over gathered rows: row r of y (expert-grouped order) uses
    token row_index[r] of qa [T][K] (row pitch allowed) and sa [K/128][ld >= T];
    equal bit for bit to fp8rl_gather_rows_fp8 followed by fp8rl_grouped_gemm_w8a8_block."""
    name = "fp8rl_grouped_gemm_w8a8_block_gathered"
    qa, qw = _u8(qa), _u8(qw)
    t, k = qa.shape
    g, n, k2 = qw.shape
    if k != k2:
        raise ValueError("K mismatch")
    if not qw.is_contiguous() or not sw.is_contiguous():
        raise ValueError("qw and sw must be contiguous")
    if sw.numel() != g * (n // 128) * (k // 128) or sw.dtype != torch.float32:
        raise ValueError("sw must be fp32 [G][N/128][K/128]")
    if sa.dtype != torch.float32 or sa.dim() != 2 or sa.size(0) != k // 128 or sa.stride(1) != 1 or sa.size(1) < t:
        raise ValueError("sa must be fp32 [K/128][ld >= T]")
    if row_index.dtype != torch.int32 or row_index.dim() != 1 or not row_index.is_contiguous():
        raise ValueError("row_index must be a contiguous 1-D int32 tensor")
    if group_offsets.dtype != torch.int32 or group_offsets.numel() != g + 1 or not group_offsets.is_contiguous():
        raise ValueError("group_offsets must be a contiguous int32 tensor of G+1 entries")
    r = row_index.numel()
    if y is None:
        y = torch.empty((r, n), dtype=torch.bfloat16, device=qa.device)
    if y.dtype != torch.bfloat16 or tuple(y.shape) != (r, n) or not y.is_contiguous():
        raise ValueError("y must be contiguous bf16 [R][N]")
    _dev(qa, sa, row_index, qw, sw, group_offsets, y)
    if r == 0:
        return y
    st = load().fp8rl_grouped_gemm_w8a8_block_gathered(qa.data_ptr(), _ld(qa), sa.data_ptr(), sa.stride(0), t,
                                                       row_index.data_ptr(), qw.data_ptr(), sw.data_ptr(),
                                                       group_offsets.data_ptr(), g, r, y.data_ptr(), n, k,
                                                       _stream(stream))
    _check(name, st)
    return y


def fp8rl_silu_mul_quant_group128(gu: torch.Tensor, q: torch.Tensor | None = None,
                                  scale: torch.Tensor | None = None, ld_scale: int | None = None,
                                  h: torch.Tensor | None = None, want_h: bool = False, stream=None):
    """bf16 gate_up [M][2I] ([gate | up]) -> (E4M3 codes of h [M][I], fp32 scales
    [I/128][ld_scale], h or None) with h = bf16(SiLU(gate) * up).  h is written only
    when a tensor is passed or want_h is set."""
    if gu.dtype != torch.bfloat16 or gu.dim() != 2:
        raise TypeError("gu must be a 2-D bfloat16 tensor")
    m, two_i = gu.shape
    if two_i % 2:
        raise ValueError("gate_up must have an even number of columns")
    inter = two_i // 2
    if scale is not None and ld_scale is None:
        ld_scale = scale.stride(0) if scale.dim() == 2 else m
    if ld_scale is None:
        ld_scale = m
    if q is None:
        q = torch.empty((m, inter), dtype=torch.uint8, device=gu.device)
    if scale is None:
        scale = torch.empty((inter // 128, ld_scale), dtype=torch.float32, device=gu.device)
    if h is None and want_h:
        h = torch.empty((m, inter), dtype=torch.bfloat16, device=gu.device)
    q = _u8(q)
    _dev(gu, q, scale, *([h] if h is not None else []))
    if scale.dtype != torch.float32 or scale.numel() < (inter // 128) * ld_scale and m > 0:
        raise ValueError("scale must be fp32 with at least [I/128][ld_scale] elements")
    if h is not None and (h.dtype != torch.bfloat16 or h.dim() != 2 or tuple(h.shape) != (m, inter)):
        raise ValueError("h must be bf16 [M][I]")
    hp, ldh = (h.data_ptr(), _ld(h) if m else inter) if h is not None else (None, 0)
    st = load().fp8rl_silu_mul_quant_group128(gu.data_ptr(), m, inter, _ld(gu) if m else two_i, q.data_ptr(),
                                           _ld(q) if m else inter, scale.data_ptr(), ld_scale, hp, ldh,
                                           _stream(stream))
    _check("fp8rl_silu_mul_quant_group128", st)
    return q, scale, h


def fp8rl_gather_rows_fp8(q_src: torch.Tensor, s_src: torch.Tensor, index: torch.Tensor,
                          q_dst: torch.Tensor | None = None, s_dst: torch.Tensor | None = None,
                          stream=None):
    """Rows index[r] of quantised activations: q_src [S][K] codes, s_src [K/128][ld >= S]
    scales -> (q_dst [R][K], s_dst [K/128][ld >= R]).  index: device int32 [R], each
    in [0, S)."""
    q_src = _u8(q_src)
    src_rows, k = q_src.shape
    if index.dtype != torch.int32 or index.dim() != 1 or not index.is_contiguous():
        raise ValueError("index must be a contiguous 1-D int32 tensor")
    rows = index.numel()
    if s_src.dtype != torch.float32 or s_src.dim() != 2 or s_src.stride(1) != 1 or s_src.size(0) != k // 128:
        raise ValueError("s_src must be fp32 [K/128][ld >= S]")
    if q_dst is None:
        q_dst = torch.empty((rows, k), dtype=torch.uint8, device=q_src.device)
    if s_dst is None:
        s_dst = torch.empty((k // 128, rows), dtype=torch.float32, device=q_src.device)
    q_dst = _u8(q_dst)
    if s_dst.dtype != torch.float32 or s_dst.dim() != 2 or s_dst.stride(1) != 1 or s_dst.size(0) != k // 128:
        raise ValueError("s_dst must be fp32 [K/128][ld >= R]")
    _dev(q_src, s_src, index, q_dst, s_dst)
    if rows == 0:
        return q_dst, s_dst
    ld_s_src = s_src.stride(0) if s_src.size(0) > 1 else s_src.size(1)
    ld_s_dst = s_dst.stride(0) if s_dst.size(0) > 1 else s_dst.size(1)
    st = load().fp8rl_gather_rows_fp8(q_src.data_ptr(), _ld(q_src), s_src.data_ptr(), ld_s_src, src_rows,
                                   index.data_ptr(), rows, k, q_dst.data_ptr(), _ld(q_dst), s_dst.data_ptr(),
                                   ld_s_dst, _stream(stream))
    _check("fp8rl_gather_rows_fp8", st)
    return q_dst, s_dst


def fp8rl_tis_workspace_size(n: int) -> int:
    return int(load().fp8rl_tis_workspace_size(int(n)))


def fp8rl_tis_weights_kl(logp_train: torch.Tensor, logp_rollout: torch.Tensor, mask: torch.Tensor | None = None,
                         clip_c: float = 2.0, w_tis: torch.Tensor | None = None, stats: torch.Tensor | None = None,
                         workspace: torch.Tensor | None = None, stream=None):
    """Token-level TIS weights min(e^d, C) (0 outside the mask) and the fp64 mismatch-KL sums
    (sum -d, sum expm1(d) - d, valid tokens, truncated tokens) of d = logp_train - logp_rollout.
    Returns (w_tis fp32 [n], stats fp64 [4]); the workspace is allocated when not supplied."""
    if logp_train.dtype != torch.float32 or logp_rollout.dtype != torch.float32:
        raise TypeError("log-probabilities must be fp32")
    if logp_train.dim() != 1 or logp_train.shape != logp_rollout.shape:
        raise ValueError("logp_train and logp_rollout must be 1-D of one length")
    if not logp_train.is_contiguous() or not logp_rollout.is_contiguous():
        raise ValueError("log-probabilities must be contiguous")
    n = logp_train.numel()
    dev = logp_train.device
    if mask is not None and (mask.dtype not in (torch.uint8, torch.bool) or mask.shape != logp_train.shape
                             or not mask.is_contiguous()):
        raise ValueError("mask must be a contiguous uint8/bool tensor of the same length")
    if w_tis is None:
        w_tis = torch.empty(n, dtype=torch.float32, device=dev)
    if stats is None:
        stats = torch.empty(4, dtype=torch.float64, device=dev)
    need = fp8rl_tis_workspace_size(n)
    if workspace is None:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=dev)
    _dev(logp_train, logp_rollout, w_tis, stats, workspace, *([mask] if mask is not None else []))
    mp = None if mask is None else mask.view(torch.uint8).data_ptr()
    st = load().fp8rl_tis_weights_kl(logp_train.data_ptr(), logp_rollout.data_ptr(), mp, n, float(clip_c),
                                     w_tis.data_ptr(), stats.data_ptr(), workspace.data_ptr(),
                                     workspace.numel() * workspace.element_size(), _stream(stream))
    _check("fp8rl_tis_weights_kl", st)
    return w_tis, stats


def fp8rl_kv_calibrate_scale(x: torch.Tensor, scale: torch.Tensor | None = None,
                             workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Per-tensor FP8 scale of a bf16 calibration tensor: fp32 [1] = amax / 448 (1.0 if zero), on the device."""
    if x.dtype != torch.bfloat16 or not x.is_contiguous():
        raise TypeError("x must be a contiguous bfloat16 tensor")
    n = x.numel()
    if scale is None:
        scale = torch.empty(1, dtype=torch.float32, device=x.device)
    need = int(load().fp8rl_kv_calibrate_workspace_size(n))
    if workspace is None:
        workspace = torch.empty(max(need, 4), dtype=torch.uint8, device=x.device)
    _dev(x, scale, workspace)
    st = load().fp8rl_kv_calibrate_scale(x.data_ptr(), n, scale.data_ptr(), workspace.data_ptr(),
                                         workspace.numel() * workspace.element_size(), _stream(stream))
    _check("fp8rl_kv_calibrate_scale", st)
    return scale


def fp8rl_kv_cache_write_fp8(k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor, k_scale: torch.Tensor,
                             v_scale: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, stream=None):
    """Quantise new tokens' k, v (bf16 [T][kv_heads][128]) into the paged caches
    (uint8 [num_blocks][kv_heads][16][128]) at slot_mapping (int64 [T])."""
    if k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16 or k.shape != v.shape or k.dim() != 3:
        raise TypeError("k and v must be bfloat16 [T][kv_heads][head_dim]")
    if not (k.is_contiguous() and v.is_contiguous() and k_cache.is_contiguous() and v_cache.is_contiguous()):
        raise ValueError("k, v and the caches must be contiguous")
    if slot_mapping.dtype != torch.int64 or slot_mapping.numel() != k.shape[0]:
        raise ValueError("slot_mapping must be int64 [T]")
    t, kvh, dim = k.shape
    k_cache, v_cache = _u8(k_cache), _u8(v_cache)
    _dev(k, v, slot_mapping, k_scale, v_scale, k_cache, v_cache)
    st = load().fp8rl_kv_cache_write_fp8(k.data_ptr(), v.data_ptr(), t, kvh, dim, slot_mapping.data_ptr(),
                                         k_cache.shape[0], k_scale.data_ptr(), v_scale.data_ptr(),
                                         k_cache.data_ptr(), v_cache.data_ptr(), _stream(stream))
    _check("fp8rl_kv_cache_write_fp8", st)


def fp8rl_attention_decode_workspace_size(batch: int, q_heads: int, kv_heads: int, max_seq_len: int) -> int:
    return int(load().fp8rl_attention_decode_workspace_size(batch, q_heads, kv_heads, max_seq_len))


def _attention(name, q, k_cache, v_cache, block_table, seq_lens, max_seq_len, sm_scale, scales, out, workspace,
               stream):
    if q.dtype != torch.bfloat16 or q.dim() != 3 or not q.is_contiguous():
        raise TypeError("q must be contiguous bfloat16 [batch][q_heads][head_dim]")
    batch, q_heads, dim = q.shape
    num_blocks, kv_heads = k_cache.shape[0], k_cache.shape[1]
    if block_table.dtype != torch.int32 or block_table.dim() != 2 or not block_table.is_contiguous():
        raise ValueError("block_table must be contiguous int32 [batch][max_blocks]")
    if seq_lens.dtype != torch.int32 or seq_lens.numel() != batch:
        raise ValueError("seq_lens must be int32 [batch]")
    if out is None:
        out = torch.empty_like(q)
    need = fp8rl_attention_decode_workspace_size(batch, q_heads, kv_heads, max_seq_len)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    _dev(q, k_cache, v_cache, block_table, seq_lens, out, workspace, *scales)
    args = [q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), num_blocks, block_table.data_ptr(),
            block_table.shape[1], seq_lens.data_ptr(), batch, q_heads, kv_heads, dim, int(max_seq_len)]
    args += [s.data_ptr() for s in scales]
    args += [float(sm_scale), out.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
             _stream(stream)]
    _check(name, getattr(load(), name)(*args))
    return out


def fp8rl_attention_decode_fp8kv(q, k_cache, v_cache, block_table, seq_lens, max_seq_len, k_scale, v_scale, sm_scale,
                                 out=None, workspace=None, stream=None):
    """Decode attention over the paged FP8 caches (uint8 [num_blocks][kv_heads][16][128]),
    scales fp32 [1] on the device; returns bf16 [batch][q_heads][128]."""
    return _attention("fp8rl_attention_decode_fp8kv", q, _u8(k_cache), _u8(v_cache), block_table, seq_lens,
                      max_seq_len, sm_scale, [k_scale, v_scale], out, workspace, stream)


def fp8rl_attention_decode_bf16kv(q, k_cache, v_cache, block_table, seq_lens, max_seq_len, sm_scale, out=None,
                                  workspace=None, stream=None):
    """The same decode attention over bf16 caches (bf16 [num_blocks][kv_heads][16][128])."""
    if k_cache.dtype != torch.bfloat16 or v_cache.dtype != torch.bfloat16:
        raise TypeError("bf16 caches expected")
    return _attention("fp8rl_attention_decode_bf16kv", q, k_cache, v_cache, block_table, seq_lens, max_seq_len,
                      sm_scale, [], out, workspace, stream)


# short aliases
quant_weight_block128 = fp8rl_quant_weight_block128
quant_act_token_group128 = fp8rl_quant_act_token_group128
gemm_w8a8_block = fp8rl_gemm_w8a8_block
grouped_gemm_w8a8_block = fp8rl_grouped_gemm_w8a8_block
silu_mul_quant_group128 = fp8rl_silu_mul_quant_group128
gather_rows_fp8 = fp8rl_gather_rows_fp8


def linear_w8a8(x: torch.Tensor, qw: torch.Tensor, sw: torch.Tensor, stream=None) -> torch.Tensor:
    """The W8A8 linear layer's forward: dynamic activation quantisation, then the
    blockwise FP8 GEMM, both on one stream with no host synchronisation."""
    qa, sa = fp8rl_quant_act_token_group128(x, stream=stream)
    return fp8rl_gemm_w8a8_block(qa, sa, qw, sw, stream=stream)
