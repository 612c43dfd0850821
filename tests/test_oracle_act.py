"""Pins of oracle/act.py (the down projection's input and the quantised-row gather)
against what the mathematics and independent routines fix."""
import numpy as np
import torch

from oracle import act, e4m3, quant


def bf16_value(bits):
    return quant.bf16_bits_to_f32(np.asarray(bits, dtype=np.uint16)).astype(np.float64)


def test_bf16_rounding_is_nearest_with_ties_to_even():
    """Brute force: the chosen bf16 value is the nearest of its two neighbours on the bf16
    grid, and an exact tie goes to the even significand."""
    rng = np.random.default_rng(1)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-95, 85, 20000))
    # exact ties: midpoints between consecutive bf16 values
    base = rng.integers(0x0001, 0x7F7E, 2000).astype(np.uint16)
    mid = (bf16_value(base) + bf16_value(base + 1)) / 2.0
    x = np.concatenate([x, mid, -mid])
    got = act.f64_to_bf16_bits(x)
    v = bf16_value(got)
    mag = got & 0x7FFF
    lo = bf16_value(np.maximum(mag.astype(np.int32) - 1, 0).astype(np.uint16)) * np.sign(x)
    hi = bf16_value((mag + 1).astype(np.uint16)) * np.sign(x)
    err = np.abs(v - x)
    assert np.all(err <= np.abs(lo - x)) and np.all(err <= np.abs(hi - x))
    ties = (err == np.abs(lo - x)) | (err == np.abs(hi - x))
    assert np.all((got[ties] & 1) == 0)
    assert ties.sum() >= 4000


def test_bf16_rounding_matches_torch_for_fp32_inputs():
    """For values exactly representable in fp32, rounding straight from fp64 is the
    library's fp32 -> bf16 conversion (round to nearest even)."""
    rng = np.random.default_rng(2)
    x32 = (rng.standard_normal(100000) * np.exp(rng.uniform(-80, 80, 100000))).astype(np.float32)
    want = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(act.f64_to_bf16_bits(x32.astype(np.float64)), want)


def test_bf16_rounding_special_values():
    x = np.array([0.0, -0.0, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 3.3895313892515355e38, 3.4e38])
    assert [hex(b) for b in act.f64_to_bf16_bits(x)] == ["0x0", "0x8000", "0x1", "0x0", "0x1", "0x7f7f", "0x7f80"]


def gate_up_bits(g, u):
    g = np.asarray(g, dtype=np.float32)
    u = np.asarray(u, dtype=np.float32)
    t = torch.from_numpy(np.concatenate([g, u], axis=1)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_silu_known_values():
    """SiLU(1) = 1 / (1 + 1/e) = 0.7310585786..., SiLU(-1) = -0.2689414213...; the
    bf16 values nearest to them are 0x3F3B (0.73046875) and 0xBE8A (-0.26953125)."""
    h = act.silu_mul_bf16(gate_up_bits([[1.0, -1.0, 0.0]], [[1.0, 1.0, 3.0]]), 3)
    assert [hex(v) for v in h[0]] == ["0x3f3b", "0xbe8a", "0x0"]


def test_silu_odd_part_is_the_identity():
    """SiLU(g) - SiLU(-g) = g exactly; after rounding both sides the difference is
    within half an ulp of each."""
    rng = np.random.default_rng(3)
    g = torch.from_numpy(rng.uniform(-20, 20, (1, 4096)).astype(np.float32)).to(torch.bfloat16).float().numpy()
    ones = np.ones_like(g)
    hp = bf16_value(act.silu_mul_bf16(gate_up_bits(g, ones), 4096))
    hn = bf16_value(act.silu_mul_bf16(gate_up_bits(-g, ones), 4096))
    ulp = lambda v: 2.0 ** (np.floor(np.log2(np.maximum(np.abs(v), 2.0 ** -126))) - 7)
    assert np.all(np.abs(hp - hn - g.astype(np.float64)) <= (ulp(hp) + ulp(hn)) / 2)


def test_silu_limits():
    """Large positive g: SiLU(g) = g to far below bf16 precision; large negative g:
    |SiLU(g)| is below the smallest bf16 subnormal, so h is -0."""
    big = np.array([[40.0, 100.0, 1000.0, 3.0e38]])
    bits = gate_up_bits(big, np.ones_like(big))
    h = act.silu_mul_bf16(bits, 4)
    assert np.array_equal(h, bits[:, :4])
    neg = np.array([[-120.0, -1000.0, -3.0e38]])
    h = act.silu_mul_bf16(gate_up_bits(neg, np.ones_like(neg)), 3)
    assert np.all(h == 0x8000)


def test_silu_mul_close_to_torch_fp32():
    """The library's fp32 SiLU times up, rounded to bf16 (two roundings), agrees with the
    exactly evaluated value except for rare one-ulp differences."""
    rng = np.random.default_rng(4)
    g = rng.standard_normal((64, 1024)).astype(np.float32) * 3
    u = rng.standard_normal((64, 1024)).astype(np.float32)
    bits = gate_up_bits(g, u)
    got = act.silu_mul_bf16(bits, 1024)
    gu = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float()
    ref = (torch.nn.functional.silu(gu[:, :1024]) * gu[:, 1024:]).to(torch.bfloat16)
    ref = ref.view(torch.int16).numpy().view(np.uint16)
    diff = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 1
    assert (diff != 0).mean() < 0.01


def test_fused_quant_keeps_the_group_invariant():
    """The quantised h: every nonzero group holds a code of magnitude 448 (0x7E) at its
    largest element, and dequantised codes are within half an E4M3 step of h."""
    rng = np.random.default_rng(5)
    g = rng.standard_normal((9, 256)).astype(np.float32)
    u = rng.standard_normal((9, 256)).astype(np.float32)
    h, codes, scales = act.silu_mul_quant_group128(gate_up_bits(g, u), 256, ld_scale=12)
    assert scales.shape == (2, 12)
    hv = bf16_value(h)
    for grp in range(2):
        sl = slice(grp * 128, (grp + 1) * 128)
        assert np.all(((codes[:, sl] & 0x7F) == 0x7E).any(axis=1))
        deq = e4m3.decode(codes[:, sl]) * scales[grp, :9, None]
        assert np.all(np.abs(deq - hv[:, sl]) <= np.abs(hv[:, sl]) * 2.0 ** -4 + scales[grp, :9, None] * 2.0 ** -10)


def test_gather_commutes_with_row_quantisation():
    """Quantising the gathered rows equals gathering the quantised rows (per-row groups)."""
    rng = np.random.default_rng(6)
    x = torch.from_numpy(rng.standard_normal((50, 384)).astype(np.float32)).to(torch.bfloat16)
    bits = x.view(torch.int16).numpy().view(np.uint16)
    index = rng.integers(0, 50, 173)
    q, s = quant.quant_act_token_group128(bits)
    gq, gs = act.gather_rows_fp8(q, s, index)
    wq, ws = quant.quant_act_token_group128(bits[index])
    assert np.array_equal(gq, wq) and np.array_equal(gs.view(np.uint32), ws.view(np.uint32))


# ---------------------------------------------------------------------------
# correct rounding of SiLU(g) * u, checked against 150-digit decimal arithmetic
# (the decimal module's exp is correctly rounded) and by brute-force nearest
# ---------------------------------------------------------------------------
def _exact_silu_mul(g: float, u: float):
    import decimal
    ctx = decimal.Context(prec=150)
    gd, ud = decimal.Decimal(g), decimal.Decimal(u)
    return ctx.multiply(ctx.divide(gd, ctx.add(1, ctx.exp(-gd))), ud)


def _assert_nearest(bits: int, exact) -> None:
    """bits is the bf16 nearest to `exact` (strictly: the exact value is never a tie)."""
    import decimal
    mag = bits & 0x7FFF
    neg = bool(bits & 0x8000)
    val = lambda b: decimal.Decimal(float(bf16_value(np.array([b], dtype=np.uint16))[0]))
    with decimal.localcontext(decimal.Context(prec=200)):    # differences of dyadic values: exact
        x = -exact if neg else exact
        if exact == 0:
            assert mag == 0
            return
        assert x > 0, "sign"
        d = abs(x - val(mag))
        assert d < abs(x - val(mag + 1)), f"bits {hex(bits)}: the next magnitude is nearer to {exact}"
        if mag > 0:
            assert d < abs(x - val(mag - 1)), f"bits {hex(bits)}: the previous magnitude is nearer to {exact}"


def _pairs_from_bits(gb, ub):
    gb = np.asarray(gb, dtype=np.uint16)[None, :]
    ub = np.asarray(ub, dtype=np.uint16)[None, :]
    return np.concatenate([gb, ub], axis=1), gb.shape[1]


def test_silu_mul_correctly_rounded_random_pairs():
    """Random finite gate values over the whole useful range (both limits and the
    fp64-evaluated middle) and random up values: brute-force nearest bf16 of the
    150-digit value."""
    rng = np.random.default_rng(11)
    g = np.concatenate([
        rng.integers(0x0001, 0x4380, 600),              # positive, up to 256
        rng.integers(0x8001, 0xC300, 600),              # negative, down to -128
        rng.integers(0x3400, 0x4200, 300),              # 2^-23 .. 32 (both limits' edges)
    ]).astype(np.uint16)
    u = rng.integers(0x0001, 0x7F00, g.size).astype(np.uint16) | (rng.integers(0, 2, g.size) << 15).astype(np.uint16)
    bits, n = _pairs_from_bits(g, u)
    h = act.silu_mul_bf16(bits, n)[0]
    gv, uv = bf16_value(g), bf16_value(u)
    for i in range(n):
        _assert_nearest(int(h[i]), _exact_silu_mul(float(gv[i]), float(uv[i])))


def _tie_pairs(g_bits):
    """Pairs (g, u) whose product g u (or g u / 2) is exactly a bf16 rounding tie:
    u runs over all 128 significands in [1, 2); keep the products with 9 significant
    bits ending in 1."""
    gs, us = [], []
    ub = np.arange(0x3F80, 0x4000, dtype=np.uint16)
    for gb in g_bits:
        gv = float(bf16_value(np.array([gb], dtype=np.uint16))[0])
        for u16 in ub:
            uv = float(bf16_value(np.array([u16], dtype=np.uint16))[0])
            m, _ = np.frexp(abs(gv * uv))
            sig = int(round(m * 2 ** 16))                   # 16 significant bits, exact
            if sig % (1 << 8) == (1 << 7):                  # 8 kept bits, then exactly one half: a tie
                gs.append(gb)
                us.append(u16)
    return np.array(gs, dtype=np.uint16), np.array(us, dtype=np.uint16)


def test_silu_mul_ties_in_the_small_gate_limit():
    """|g| <= 2^-20: g u / 2 exactly on a bf16 tie; the exact value is off it by the
    relative amount tanh(g / 2), so it rounds away from zero for g > 0 and toward
    zero for g < 0 -- checked against the 150-digit value, for both signs of u."""
    gb = np.array([0x3580, 0x35C0, 0x2E40, 0x1FA0, 0x0C60, 0xB580, 0xB5C0, 0xAE40, 0x8C60, 0x3480], dtype=np.uint16)
    g, u = _tie_pairs(gb)
    assert g.size > 20
    u = np.concatenate([u, u | 0x8000])
    g = np.concatenate([g, g])
    bits, n = _pairs_from_bits(g, u)
    h = act.silu_mul_bf16(bits, n)[0]
    gv, uv = bf16_value(g), bf16_value(u)
    for i in range(n):
        _assert_nearest(int(h[i]), _exact_silu_mul(float(gv[i]), float(uv[i])))


def test_silu_mul_ties_in_the_large_gate_limit():
    """g >= 16: g u exactly on a bf16 tie; SiLU(g) < g, so the exact value rounds
    toward zero.  Gates from 16 to 200 (e^-200 is still resolved at 150 digits)."""
    gb = np.array([0x4180, 0x4190, 0x41A0, 0x4240, 0x4280, 0x42C8, 0x4348], dtype=np.uint16)  # 16 .. 200
    g, u = _tie_pairs(gb)
    assert g.size > 20
    bits, n = _pairs_from_bits(g, u)
    h = act.silu_mul_bf16(bits, n)[0]
    gv, uv = bf16_value(g), bf16_value(u)
    for i in range(n):
        _assert_nearest(int(h[i]), _exact_silu_mul(float(gv[i]), float(uv[i])))


def test_silu_mul_fp64_middle_never_near_a_tie():
    """Between the two limits the oracle trusts fp64 (error a few 2^-53).  Over every
    finite gate bit pattern there (g > -700: below that the product is far below
    the smallest bf16 at any up) and every up significand, SiLU(g) u_sig stays more
    than 2^-47 (in significand units) away from every bf16 rounding boundary, at
    every number of kept bits from 0 (the smallest subnormal) to 8 (normal
    numbers); scaling u by a power of two only moves that picture."""
    gbits = np.arange(0x10000, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):
        g = bf16_value(gbits)
    keep = np.isfinite(g) & (np.abs(g) > act.SMALL_G) & (g < act.LARGE_G) & (g > -700.0)
    g = g[keep]
    u = 1.0 + np.arange(128, dtype=np.float64) / 128.0
    with np.errstate(over="ignore"):
        silu = g / (1.0 + np.exp(-g))
    worst = np.inf
    for s in range(9):
        for j in range(0, 128, 32):
            x = np.abs(silu[:, None] * u[None, j:j + 32])
            m, _ = np.frexp(x)
            y = np.ldexp(m * 2.0, s)                     # significand in [1, 2), times 2^s (exact)
            dist = np.abs(y - np.floor(y) - 0.5) / 2.0 ** s
            worst = min(worst, float(dist.min()))
    assert worst > 2.0 ** -47, worst
