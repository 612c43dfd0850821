"""Blockwise-scaled FP8 GEMM, dense and grouped -- oracle, test infrastructure only.

The paper runs its W8A8 linear layers on FP8 GEMMs with the block scales of
section 2.1.1 (weights: one fp32 scale per 128x128 block; activations: one per
1x128 group) and recommends an FP8 GEMM library for them (section 2.1.4).  In
exact arithmetic the layer output is

    Y[m, n] = sum_k  dec(qA[m, k]) * sA[k // 128, m]  *  dec(qW[n, k]) * sW[n // 128, k // 128]

i.e. dequantise both operands, then multiply.  This module evaluates exactly
that in fp64 (``numpy.matmul`` as the one library step).  Every product of two
E4M3 values is exact in fp64; only the fp64 summation and the scale products
round, far below the tolerance used against the GPU.

MoE expert layers (fc1/fc2, section 2.1.1 "Quantization scope") apply the same
product per expert to the rows routed to it.  Reading: rows are stored grouped
by expert, with int32 offsets[g + 1] (offsets[0] = 0, non-decreasing,
offsets[g] = total rows); rows offsets[e]..offsets[e+1]-1 use expert e's weight.
"""
import numpy as np

from . import e4m3

BLOCK = 128


def dequant_act(qa: np.ndarray, sa: np.ndarray) -> np.ndarray:
    """codes [M][K], scales [K/128][ld >= M] -> fp64 [M][K]."""
    m, k = qa.shape
    s = np.repeat(np.asarray(sa, np.float64)[:, :m].T, BLOCK, axis=1)   # [M][K]
    return e4m3.decode(qa) * s


def dequant_weight(qw: np.ndarray, sw: np.ndarray) -> np.ndarray:
    """codes [N][K], scales [N/128][K/128] -> fp64 [N][K]."""
    s = np.repeat(np.repeat(np.asarray(sw, np.float64), BLOCK, axis=0), BLOCK, axis=1)
    return e4m3.decode(qw) * s


def gemm_ref_fp64(qa, sa, qw, sw) -> np.ndarray:
    """Y = dequant(A) @ dequant(W)^T in fp64 -> [M][N]."""
    return dequant_act(qa, sa) @ dequant_weight(qw, sw).T


def grouped_gemm_ref_fp64(qa, sa, qw, sw, offsets) -> np.ndarray:
    """Per expert e: Y[off_e:off_e+1] = dense reference with W_e.  Empty experts write nothing.

    qa [R][K]; sa [K/128][ld >= R] (columns indexed by global row);
    qw [G][N][K]; sw [G][N/128][K/128]; offsets int [G+1].
    Rows not covered by any expert (none, for valid offsets) stay 0.
    """
    qa = np.asarray(qa)
    offsets = np.asarray(offsets, dtype=np.int64)
    g, n, k = qw.shape
    r = qa.shape[0]
    y = np.zeros((r, n), dtype=np.float64)
    for e in range(g):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi <= lo:
            continue
        a = dequant_act(qa[lo:hi], np.asarray(sa)[:, lo:hi])
        y[lo:hi] = a @ dequant_weight(qw[e], sw[e]).T
    return y


def grouped_gemm_gathered_ref_fp64(qa_src, sa_src, row_index, qw, sw, offsets) -> np.ndarray:
    """The grouped product over gathered rows: row r (expert-grouped order) uses
    activation row row_index[r] of qa_src [T][K] and its scales sa_src[:, row_index[r]].
    Per-token scales make quantising commute with copying rows, so this is the
    dispatch of already-quantised tokens followed by the per-expert product.
    """
    row_index = np.asarray(row_index, dtype=np.int64)
    offsets = np.asarray(offsets, dtype=np.int64)
    g, n, k = qw.shape
    y = np.zeros((row_index.size, n), dtype=np.float64)
    for e in range(g):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi <= lo:
            continue
        rows = row_index[lo:hi]
        a = dequant_act(np.asarray(qa_src)[rows], np.asarray(sa_src)[:, rows])
        y[lo:hi] = a @ dequant_weight(qw[e], sw[e]).T
    return y


def gemm_blockwise_bruteforce(qa, sa, qw, sw) -> np.ndarray:
    """The same product written as the blockwise sum, with explicit Python loops.

    Y[m, n] = sum_kb sA[kb, m] * sW[n//128, kb] * sum_{k in kb} dec(qA[m,k]) * dec(qW[n,k]).
    No BLAS; pure Python floats (fp64).  For tiny shapes only: it pins the
    dequantise-then-matmul form above.
    """
    m, k = qa.shape
    n = qw.shape[0]
    da = e4m3.decode(qa).tolist()
    dw = e4m3.decode(qw).tolist()
    sa = np.asarray(sa, np.float64).tolist()
    sw = np.asarray(sw, np.float64).tolist()
    y = np.zeros((m, n), dtype=np.float64)
    for i in range(m):
        for j in range(n):
            total = 0.0
            for kb in range(k // BLOCK):
                part = 0.0
                for kk in range(kb * BLOCK, (kb + 1) * BLOCK):
                    part += da[i][kk] * dw[j][kk]
                total += sa[kb][i] * sw[j // BLOCK][kb] * part
            y[i, j] = total
    return y


def tolerance_check(y_gpu: np.ndarray, y_ref: np.ndarray, rel=4e-3, rms_frac=1e-3):
    """Pass criterion per element: |gpu - ref| <= rel*|ref| + rms_frac*rms(ref).

    rms is taken over every element of the call's output.  Returns
    (ok, worst_ratio, rms) where worst_ratio = max |err| / bound (<= 1 passes).
    """
    y_gpu = np.asarray(y_gpu, np.float64)
    y_ref = np.asarray(y_ref, np.float64)
    if y_ref.size == 0:
        return True, 0.0, 0.0
    rms = float(np.sqrt(np.mean(y_ref * y_ref)))
    bound = rel * np.abs(y_ref) + rms_frac * rms
    err = np.abs(y_gpu - y_ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(bound > 0, err / bound, np.where(err > 0, np.inf, 0.0))
    worst = float(np.max(ratio))
    return bool(np.all(err <= bound)), worst, rms
