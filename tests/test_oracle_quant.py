"""Pins for the oracle's blockwise / groupwise quantisation (section 2.1.1, Eq. (1)).

What fixes the answer independently of the oracle's own code:
* the hand-worked block in tests/golden/quant_worked_block.txt;
* the invariant that each block's largest magnitude lands exactly on +-448;
* per element, the code equals torch's float8_e4m3fn cast of fl32(x / s);
* the E4M3 half-spacing error bound on the dequantised values;
* layout cases where each block/group has a distinct constant magnitude.
"""
import os

import numpy as np
import pytest
import torch

from oracle import e4m3, quant

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bits_to_f32(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def randn_bf16(shape, std, seed):
    rng = np.random.default_rng(seed)
    return f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * std)


def torch_cast(v):
    return torch.from_numpy(np.ascontiguousarray(v, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_worked_block_from_golden():
    kv = {}
    codes_at = []
    with open(os.path.join(GOLDEN, "quant_worked_block.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            p = line.split()
            if p[0] == "code":
                codes_at.append((int(p[1]), int(p[2]), int(p[3], 16)))
            else:
                kv[p[0]] = int(p[1], 16)
    x = np.ones((128, 128), np.float32)
    x[5, 7] = 2.0
    x[9, 3] = -1.0
    q, s = quant.quant_weight_block128(f32_to_bf16_bits(x))
    assert s.shape == (1, 1)
    assert int(s.view(np.uint32)[0, 0]) == kv["scale_bits"]
    want = np.full((128, 128), kv["code_default"], np.uint8)
    for r, c, code in codes_at:
        want[r, c] = code
    assert np.array_equal(q, want)


def _check_block_invariants(xb, qb, s):
    """Invariants any correct block/group quantiser satisfies."""
    amax = float(np.max(np.abs(xb)))
    assert not np.any((qb & 0x7F) == 0x7F), "NaN code"
    if amax == 0.0:
        assert s == np.float32(1.0)
        assert np.array_equal(qb & 0x7F, np.zeros_like(qb))
        assert np.array_equal(qb >> 7, np.signbit(xb).astype(np.uint8))
        return
    assert s == np.float32(np.float32(amax) / np.float32(448.0))
    at = np.abs(xb) == amax
    assert np.all((qb[at] & 0x7F) == 0x7E), "block amax must map to +-448"
    # per element: torch's cast of the fp32 quotient (a library routine)
    quot = (xb / np.float32(s)).astype(np.float32)
    assert np.array_equal(qb, torch_cast(quot))
    # E4M3 rounding error bound: half a grid step, relative 2^-4 in the normal
    # range and absolute 2^-10 * s in the subnormal range
    deq = e4m3.decode(qb) * np.float64(s)
    err = np.abs(deq - xb.astype(np.float64))
    bound = np.maximum(np.abs(xb.astype(np.float64)) * 2.0 ** -4, 2.0 ** -10 * np.float64(s)) * (1 + 1e-6)
    assert np.all(err <= bound)


def test_weight_quant_invariants_random():
    w = randn_bf16((384, 256), 0.02, 1)
    q, s = quant.quant_weight_block128(w)
    x = bits_to_f32(w)
    assert q.shape == (384, 256) and s.shape == (3, 2) and s.dtype == np.float32
    for i in range(3):
        for j in range(2):
            sl = (slice(128 * i, 128 * i + 128), slice(128 * j, 128 * j + 128))
            _check_block_invariants(x[sl], q[sl], s[i, j])


def test_weight_quant_special_blocks():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((256, 512)) * 0.02).astype(np.float32)
    x[0:128, 0:128] = 0.0                                  # all zero, mixed signs
    x[0:128, 0:128][::3, ::5] = -0.0
    x[0:128, 128:256] = 0.0                                # single nonzero
    x[17, 128 + 40] = -3.0
    x[128:256, 0:128] *= 1e36                              # huge, bf16 max present
    x[200, 9] = 3.3895313892515355e38
    x[128:256, 128:256] *= 1e-38                           # tiny: subnormal scale
    x[128:256, 256:384] = 2.0 ** -133                      # smallest bf16 subnormal everywhere
    x[130, 300] = -(2.0 ** -133)
    w = f32_to_bf16_bits(x)
    xf = bits_to_f32(w)
    q, s = quant.quant_weight_block128(w)
    for i in range(2):
        for j in range(4):
            sl = (slice(128 * i, 128 * i + 128), slice(128 * j, 128 * j + 128))
            _check_block_invariants(xf[sl], q[sl], s[i, j])
    # the single-nonzero block: one 0xFE, every other code +0
    blk = q[0:128, 128:256]
    assert blk[17, 40] == 0xFE and np.count_nonzero(blk) == 1
    assert s[0, 0] == np.float32(1.0)
    assert s[1, 1] < np.float32(2.0 ** -126)               # subnormal scale really exercised


def test_weight_quant_layout_distinct_constants():
    # block (i, j) holds the constant c_ij; N != K catches a transposed layout
    nb_n, nb_k = 3, 5
    c = (2.0 ** np.arange(nb_n * nb_k).reshape(nb_n, nb_k) * 0.75).astype(np.float32)
    x = np.repeat(np.repeat(c, 128, axis=0), 128, axis=1)
    x[::2, ::2] *= -1
    q, s = quant.quant_weight_block128(f32_to_bf16_bits(x))
    assert np.array_equal(s, (c / np.float32(448.0)).astype(np.float32))
    assert np.all((q & 0x7F) == 0x7E)
    assert np.array_equal(q >> 7, (x < 0).astype(np.uint8))


def test_weight_quant_rejects_ragged_shapes():
    with pytest.raises(ValueError):
        quant.quant_weight_block128(np.zeros((128, 200), np.uint16))


def test_act_quant_invariants_and_layout():
    m, k, ld = 37, 384, 40
    rng = np.random.default_rng(5)
    x = rng.standard_normal((m, k)).astype(np.float32)
    # distinct group magnitudes: group g of row r scaled by 2^(r % 7 - g)
    gains = 2.0 ** (np.arange(m)[:, None] % 7 - np.arange(k // 128)[None, :])
    x = (x * np.repeat(gains, 128, axis=1)).astype(np.float32)
    x[3, 128:256] = 0.0
    x[3, 130] = -0.0
    a = f32_to_bf16_bits(x)
    xf = bits_to_f32(a)
    q, s = quant.quant_act_token_group128(a, ld_scale=ld)
    assert s.shape == (k // 128, ld) and np.all(s[:, m:] == 0)
    for r in range(m):
        for g in range(k // 128):
            sl = slice(128 * g, 128 * g + 128)
            _check_block_invariants(xf[r, sl], q[r, sl], s[g, r])
    assert s[1, 3] == np.float32(1.0)


def test_act_quant_equals_weight_quant_on_one_row_blocks():
    # a 1x128 group is the weight rule applied to a one-row block: checking the
    # two entry points against each other on rows repeated 128 times
    rng = np.random.default_rng(9)
    row = f32_to_bf16_bits(rng.standard_normal(256).astype(np.float32))
    qa, sa = quant.quant_act_token_group128(row[None, :])
    qw, sw = quant.quant_weight_block128(np.repeat(row[None, :], 128, axis=0))
    assert np.array_equal(qw[0], qa[0]) and np.array_equal(sw[0], sa[:, 0])


def test_act_quant_empty_m():
    q, s = quant.quant_act_token_group128(np.zeros((0, 256), np.uint16))
    assert q.shape == (0, 256) and s.shape == (2, 0)
