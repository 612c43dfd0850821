"""Pins the C restatement of the quantiser (oracle/quant_ref.c) to the numpy
oracle and to torch's float8_e4m3fn cast, so the fast C form can stand in for
the numpy one in full-size and exhaustive checks."""
import numpy as np
import pytest
import torch

from oracle import cref, quant


def f32_to_bf16_bits(x):
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def all_finite_bf16_magnitudes():
    b = np.arange(0x7F80, dtype=np.uint16)          # +0 .. largest finite
    return b


def test_c_weight_quant_equals_numpy_oracle():
    rng = np.random.default_rng(21)
    x = (rng.standard_normal((256, 384)) * 0.02).astype(np.float32)
    x[0:128, 0:128] = 0.0
    x[0:128, 0:128][::7, ::3] = -0.0
    x[128:256, 128:256] *= 1e36
    x[130, 131] = -3.3895313892515355e38
    x[0:128, 256:384] *= 1e-37
    w = f32_to_bf16_bits(x)
    qn, sn = quant.quant_weight_block128(w)
    qc, sc = cref.quant_weight_block128(w)
    assert np.array_equal(qn, qc)
    assert np.array_equal(sn.view(np.uint32), sc.view(np.uint32))


def test_c_act_quant_equals_numpy_oracle():
    rng = np.random.default_rng(22)
    x = rng.standard_normal((33, 512)).astype(np.float32)
    x[:, 5] *= 50
    x[4, 128:256] = 0.0
    a = f32_to_bf16_bits(x)
    qn, sn = quant.quant_act_token_group128(a, ld_scale=40)
    qc, sc = cref.quant_act_token_group128(a, ld_scale=40)
    assert np.array_equal(qn, qc)
    assert np.array_equal(sn.view(np.uint32), sc.view(np.uint32))


def test_c_element_map_equals_numpy_and_torch_for_sampled_amax():
    mags = all_finite_bf16_magnitudes()
    rng = np.random.default_rng(23)
    amaxes = np.concatenate([
        np.array([1, 2, 0x0080, 0x3F80, 0x43E0, 0x7F7F, 0x7F7E, 0x0001], np.uint16),
        rng.choice(mags[1:], size=40, replace=False).astype(np.uint16),
    ])
    for am in amaxes.tolist():
        xs = mags[mags <= am]
        xs = np.concatenate([xs, xs | np.uint16(0x8000)])
        amv = np.full(xs.shape, am, np.uint16)
        got = cref.e4m3_of_quotient(xs, amv)
        s = quant._scale_from_amax(quant.bf16_bits_to_f32(np.array([am], np.uint16)))[0]
        want = quant.quantize_with_scale(quant.bf16_bits_to_f32(xs), s)
        assert np.array_equal(got, want), hex(am)
        quot = (quant.bf16_bits_to_f32(xs) / s).astype(np.float32)
        tc = torch.from_numpy(quot).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        assert np.array_equal(got, tc), hex(am)


@pytest.mark.slow
def test_c_element_map_equals_numpy_exhaustive():
    """Every (x, amax) bf16 pair with |x| <= amax: C form == numpy form (minutes)."""
    mags = all_finite_bf16_magnitudes()
    for am in range(1, 0x7F80):
        xs = mags[mags <= am]
        xs = np.concatenate([xs, xs | np.uint16(0x8000)])
        got = cref.e4m3_of_quotient(xs, np.full(xs.shape, am, np.uint16))
        s = quant._scale_from_amax(quant.bf16_bits_to_f32(np.array([am], np.uint16)))[0]
        want = quant.quantize_with_scale(quant.bf16_bits_to_f32(xs), s)
        assert np.array_equal(got, want), hex(am)


def test_c_ue8m0_quant_equals_numpy_oracle():
    """The C power-of-two variant equals oracle/ue8m0.py on special blocks and on a
    group for every finite bf16 magnitude (every scale exponent and the clamp)."""
    from oracle import ue8m0
    rng = np.random.default_rng(24)
    x = (rng.standard_normal((256, 384)) * 0.02).astype(np.float32)
    x[0:128, 0:128] = 0.0
    x[0:128, 0:128][::7, ::3] = -0.0
    x[128:256, 128:256] *= 1e36
    x[130, 131] = -3.3895313892515355e38
    x[0:128, 256:384] *= 1e-37
    w = f32_to_bf16_bits(x)
    qn, sn = ue8m0.quant_weight_block128_ue8m0(w)
    qc, sc = cref.quant_weight_block128_ue8m0(w)
    assert np.array_equal(qn, qc)
    assert np.array_equal(sn.view(np.uint32), sc.view(np.uint32))
    mags = all_finite_bf16_magnitudes()
    a = np.zeros((mags.size, 128), np.uint16)
    a[:, 0] = mags
    a[:, 1] = mags | 0x8000
    a[:, 2:] = rng.integers(0, 0x7F80, (mags.size, 126)).astype(np.uint16) % (mags[:, None].astype(np.int64) + 1)
    qn, sn = ue8m0.quant_act_token_group128_ue8m0(a, ld_scale=mags.size + 3)
    qc, sc = cref.quant_act_token_group128_ue8m0(a, ld_scale=mags.size + 3)
    assert np.array_equal(qn, qc)
    assert np.array_equal(sn.view(np.uint32), sc.view(np.uint32))
