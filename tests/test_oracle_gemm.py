"""Pins for the oracle's blockwise-scaled GEMM (dense and grouped).

* brute force: explicit Python loops over the blockwise sum (no BLAS);
* closed forms: integer codes with unit scales give exact integers; identity
  weights return the dequantised activations; a single nonzero K block isolates
  one (sA, sW) pair; distinct power-of-two scales expose any indexing slip;
* grouped = per-expert dense on slices, empty experts write nothing.
"""
import numpy as np
import pytest

from oracle import e4m3, gemm

CODE_ONE = 0x38          # 1.0 in E4M3


def int_codes(vals):
    """Small integers -> their exact E4M3 codes."""
    return e4m3.encode(np.asarray(vals, np.float32))


def rand_codes(shape, rng):
    c = rng.integers(0, 256, size=shape, dtype=np.uint8)
    c[(c & 0x7F) == 0x7F] = 0x38                       # no NaN codes
    return c


def test_dense_matches_bruteforce_tiny():
    rng = np.random.default_rng(0)
    m, n, k = 3, 256, 256
    qa, qw = rand_codes((m, k), rng), rand_codes((n, k), rng)
    sa = rng.random((k // 128, m + 2)).astype(np.float32) + 0.1
    sw = rng.random((n // 128, k // 128)).astype(np.float32) + 0.1
    y = gemm.gemm_ref_fp64(qa, sa, qw, sw)
    yb = gemm.gemm_blockwise_bruteforce(qa, sa, qw, sw)
    assert np.allclose(y, yb, rtol=1e-12, atol=1e-12 * np.abs(yb).max())


def test_integer_closed_form():
    rng = np.random.default_rng(1)
    m, n, k = 5, 128, 256
    ia = rng.integers(-3, 4, size=(m, k))
    iw = rng.integers(-3, 4, size=(n, k))
    y = gemm.gemm_ref_fp64(int_codes(ia), np.ones((2, m), np.float32),
                           int_codes(iw), np.ones((1, 2), np.float32))
    assert np.array_equal(y, (ia @ iw.T).astype(np.float64))


def test_identity_weight_returns_dequantised_activations():
    rng = np.random.default_rng(2)
    m, k = 4, 256
    qa = rand_codes((m, k), rng)
    sa = (2.0 ** rng.integers(-5, 5, size=(2, m))).astype(np.float32)
    qw = np.zeros((k, k), np.uint8)
    qw[np.arange(k), np.arange(k)] = CODE_ONE
    c = np.float32(0.375)
    sw = np.full((2, 2), c, np.float32)
    y = gemm.gemm_ref_fp64(qa, sa, qw, sw)
    want = e4m3.decode(qa) * np.repeat(sa.T.astype(np.float64), 128, axis=1) * float(c)
    assert np.array_equal(y, want)


def test_single_k_block_isolates_scale_pair():
    m, n, k = 2, 256, 384
    qa = np.zeros((m, k), np.uint8)
    qw = np.zeros((n, k), np.uint8)
    qa[:, 128:256] = CODE_ONE                          # only K block 1 is nonzero
    qw[:, 128:256] = CODE_ONE
    sa = np.array([[1, 1], [2.0 ** 3, 2.0 ** 5], [7, 7]], np.float32)   # [K/128][M]
    sw = np.array([[11, 2.0 ** -2, 13], [17, 2.0 ** -4, 19]], np.float32)  # [N/128][K/128]
    y = gemm.gemm_ref_fp64(qa, sa, qw, sw)
    for i in range(m):
        for j in range(n):
            assert y[i, j] == 128 * sa[1, i] * sw[j // 128, 1]


def test_power_of_two_scales_expose_indexing():
    # each (m, kb) and (nb, kb) gets a distinct power of two; codes all 1.0:
    # Y[m, n] = 128 * sum_kb sA[kb, m] * sW[n//128, kb] -- exact in fp64
    m, n, k = 3, 384, 512
    kb = k // 128
    sa = (2.0 ** (np.arange(kb * m).reshape(kb, m) * 2)).astype(np.float32)
    sw = (2.0 ** (-np.arange((n // 128) * kb).reshape(n // 128, kb) * 3)).astype(np.float32)
    qa = np.full((m, k), CODE_ONE, np.uint8)
    qw = np.full((n, k), CODE_ONE, np.uint8)
    y = gemm.gemm_ref_fp64(qa, sa, qw, sw)
    for i in range(m):
        for j in range(n):
            want = sum(128.0 * float(sa[b, i]) * float(sw[j // 128, b]) for b in range(kb))
            assert y[i, j] == want


def test_grouped_equals_per_expert_bruteforce():
    rng = np.random.default_rng(4)
    g, n, k = 4, 128, 256
    counts = [3, 0, 5, 2]                              # one empty expert
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    qa = rand_codes((r, k), rng)
    sa = rng.random((k // 128, r)).astype(np.float32) + 0.5
    qw = rand_codes((g, n, k), rng)
    sw = rng.random((g, n // 128, k // 128)).astype(np.float32) + 0.5
    y = gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, offsets)
    for e in range(g):
        lo, hi = offsets[e], offsets[e + 1]
        if hi > lo:
            yb = gemm.gemm_blockwise_bruteforce(qa[lo:hi], sa[:, lo:hi], qw[e], sw[e])
            assert np.allclose(y[lo:hi], yb, rtol=1e-12, atol=1e-12 * np.abs(yb).max())


def test_grouped_single_group_equals_dense():
    rng = np.random.default_rng(5)
    r, n, k = 7, 256, 256
    qa, qw = rand_codes((r, k), rng), rand_codes((1, n, k), rng)
    sa = rng.random((2, r)).astype(np.float32)
    sw = rng.random((1, 2, 2)).astype(np.float32)
    y = gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, np.array([0, r], np.int32))
    assert np.array_equal(y, gemm.gemm_ref_fp64(qa, sa, qw[0], sw[0]))


def test_grouped_gathered_rows_bruteforce_and_composition():
    """Rows taken from a token table by index (repeats, unused tokens, an empty expert):
    each row equals the blockwise brute force on its token; the whole equals gathering
    the quantised rows first and then the grouped product; the identity index gives
    the grouped product itself."""
    from oracle import act
    rng = np.random.default_rng(6)
    g, n, k, t = 3, 128, 256, 5
    counts = [4, 0, 3]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    index = np.array([4, 0, 4, 2, 1, 1, 3], np.int32)[:r]
    qa = rand_codes((t, k), rng)
    sa = rng.random((k // 128, t + 2)).astype(np.float32) + 0.5     # ld_sa > t
    qw = rand_codes((g, n, k), rng)
    sw = rng.random((g, n // 128, k // 128)).astype(np.float32) + 0.5
    y = gemm.grouped_gemm_gathered_ref_fp64(qa, sa, index, qw, sw, offsets)
    for e in range(g):
        for row in range(offsets[e], offsets[e + 1]):
            tok = index[row]
            yb = gemm.gemm_blockwise_bruteforce(qa[tok:tok + 1], sa[:, tok:tok + 1], qw[e], sw[e])
            assert np.allclose(y[row:row + 1], yb, rtol=1e-12, atol=1e-12 * np.abs(yb).max())
    qg, sg = act.gather_rows_fp8(qa, sa[:, :t], index)
    assert np.array_equal(y, gemm.grouped_gemm_ref_fp64(qg, sg, qw, sw, offsets))
    ident = np.arange(t, dtype=np.int32)
    off1 = np.array([0, 2, 2, t], np.int32)
    assert np.array_equal(gemm.grouped_gemm_gathered_ref_fp64(qa, sa, ident, qw, sw, off1),
                          gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, off1))


def test_tolerance_check_semantics():
    ref = np.array([[1.0, -2.0], [0.0, 4.0]])
    rms = np.sqrt(np.mean(ref ** 2))
    ok, worst, r = gemm.tolerance_check(ref + 4e-3 * np.abs(ref) + 0.999e-3 * rms, ref)
    assert ok and worst <= 1.0 and r == pytest.approx(rms)
    ok, worst, _ = gemm.tolerance_check(ref + 0.01, ref)
    assert not ok and worst > 1.0
