"""Pins of oracle/ue8m0.py (power-of-two scale variant, section 2.4.3) against what
the definition and independent routines fix."""
import numpy as np
import torch

from oracle import e4m3, quant, ue8m0


def bf16_values(bits):
    return quant.bf16_bits_to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def all_positive_finite_bf16():
    return np.arange(0x0001, 0x7F80, dtype=np.uint32).astype(np.uint16)


def test_exponent_is_the_smallest_that_fits_every_bf16_amax():
    """Brute force over every positive finite bf16 amax: k is the first candidate in
    -127 .. 130 with amax <= 448 * 2^k (exact comparisons in fp64), no logarithm."""
    amax = bf16_values(all_positive_finite_bf16())
    ks = np.arange(-127, 131)
    fits = amax[:, None] <= 448.0 * np.ldexp(1.0, ks)[None, :]
    want = ks[np.argmax(fits, axis=1)]
    assert fits.any(axis=1).all()
    assert np.array_equal(ue8m0.scale_exponent(amax), want)


def test_exponent_worked_values():
    vals = [448.0, 450.0, 1.0, 0.875, 0.0, 3.3895313892515355e38, 2.0 ** -133, 448.0 * 2.0 ** -127,
            448.0 * 2.0 ** -126, 0.02, 224.0]
    want = [0, 1, -8, -9, 0, 120, -127, -127, -126, -14, -1]
    assert ue8m0.scale_exponent(np.array(vals)).tolist() == want


def test_codes_are_the_library_cast_of_the_exactly_scaled_values():
    """codes == torch float8_e4m3fn cast of x * 2^-k (|x * 2^-k| <= 448, so the
    library's non-saturating cast is exact RNE there)."""
    rng = np.random.default_rng(1)
    w = torch.from_numpy((rng.standard_normal((256, 384)) * 0.02).astype(np.float32))
    w[rng.integers(0, 256, 40), rng.integers(0, 384, 40)] *= 50
    w[0:128, 128:256] *= 1e-36                      # tiny block (clamped exponent)
    w[128:256, 0:128] = 0.0
    bits = w.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    codes, scales = ue8m0.quant_weight_block128_ue8m0(bits)
    x = bf16_values(bits)
    k = np.repeat(np.repeat(np.log2(scales.astype(np.float64)), 128, 0), 128, 1)
    scaled = torch.from_numpy(np.ldexp(x, -k.astype(np.int64)).astype(np.float32))
    want = scaled.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, want)
    assert scales[1, 0] == 1.0 and np.all(codes[128:256, 0:128] & 0x7F == 0)


def test_scales_are_powers_of_two_and_maxima_land_in_the_top_binade():
    rng = np.random.default_rng(2)
    a = torch.from_numpy((rng.standard_normal((37, 512)) * np.exp(rng.uniform(-30, 30, (37, 1)))).astype(np.float32))
    bits = a.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    codes, scales = ue8m0.quant_act_token_group128_ue8m0(bits, ld_scale=40)
    assert scales.shape == (4, 40) and np.all(scales[:, 37:] == 0)
    s = scales[:, :37].astype(np.float64)
    m, e = np.frexp(s)
    assert np.all(m == 0.5)
    x = np.abs(bf16_values(bits)).reshape(37, 4, 128)
    amax = x.max(axis=2)
    r = amax / s.T
    assert np.all((r > 224.0) & (r <= 448.0))
    top = (codes.reshape(37, 4, 128) & 0x7F)[np.arange(37)[:, None], np.arange(4)[None, :], x.argmax(axis=2)]
    assert np.all((top >= 0x76) & (top <= 0x7E))
    assert np.array_equal(ue8m0.e8m0_byte(s), e - 1 + 127)


def test_power_of_two_multiples_of_448_agree_with_the_fp32_scale_path():
    """When a group's maximum is 448 * 2^j, amax / 448 is exactly 2^j: the fp32-scale
    quantiser (an independent formula: IEEE division) gives the same scale and codes."""
    rng = np.random.default_rng(3)
    x = rng.uniform(-1, 1, (64, 256)).astype(np.float32)
    j = rng.integers(-20, 20, (64, 2))
    for g in range(2):
        x[:, g * 128:(g + 1) * 128] *= np.ldexp(448.0, j[:, g])[:, None].astype(np.float32)
        x[np.arange(64), g * 128 + rng.integers(0, 128, 64)] = np.ldexp(448.0, j[:, g]) * rng.choice([-1, 1], 64)
    bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    c1, s1 = ue8m0.quant_act_token_group128_ue8m0(bits)
    c2, s2 = quant.quant_act_token_group128(bits)
    assert np.array_equal(s1, s2) and np.array_equal(c1, c2)


def test_zero_and_signed_zero():
    bits = np.zeros((2, 128), dtype=np.uint16)
    bits[1, ::2] = 0x8000
    codes, scales = ue8m0.quant_act_token_group128_ue8m0(bits)
    assert np.all(scales == 1.0)
    assert np.all(codes[0] == 0) and np.all(codes[1, ::2] == 0x80) and np.all(codes[1, 1::2] == 0)
