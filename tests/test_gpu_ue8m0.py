"""GPU parity of the power-of-two (UE8M0) scale variant (section 2.4.3) against the
CPU oracle: quantiser codes and scales bit for bit (including every group maximum
and every (element, scale exponent) pair), and the dense and grouped GEMMs on the
MX-scaled MFMA within |gpu - ref| <= 4e-3 |ref| + 1e-3 rms(ref) of the fp64 oracle,
on operands quantised by the oracle."""
import numpy as np
import pytest
import torch

import synth
from oracle import cref, gemm, ue8m0
from tests.gpu_util import announce, assert_codes_equal, assert_scales_equal, need_gpu, u8, u16, f32
from tests.test_gpu_gemm import check, dense_attribution, dense_ref_by_rows, grouped_attribution, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fp8rl():
    need_gpu()
    import paper_2601_18150_amd as m
    m.load()
    return m


def test_quant_weight_ue8m0_special_blocks_and_ld(fp8rl):
    announce("quant_weight_ue8m0 special blocks, ldw > k, ldq > k")
    n, k = 384, 640
    w = synth.normal_bf16((n, k), 0.02, 77, "cuda")
    synth.plant_special_blocks(w, 78, frac_zero=2 / 15, frac_large=2 / 15)
    wf = w.float()
    wf[128:256, 0:128] *= 1e-38            # subnormal-range block: clamped exponent
    wf[256:384, 128:256] = 2.0 ** -133
    wf[0:128, 512:640] = 0.0
    wf[5, 515] = -3.0
    w = wf.to(torch.bfloat16)
    wpad = torch.zeros((n, k + 24), dtype=torch.bfloat16, device="cuda")
    wpad[:, :k] = w
    qbuf = torch.full((n, k + 48), 0xAB, dtype=torch.uint8, device="cuda")
    q, s = fp8rl.fp8rl_quant_weight_block128_ue8m0(wpad[:, :k], q=qbuf[:, :k])
    torch.cuda.synchronize()
    qo, so = ue8m0.quant_weight_block128_ue8m0(u16(w))
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s), so, "scales")
    assert np.all(u8(qbuf[:, k:]) == 0xAB), "wrote past k in a padded row"


@pytest.mark.parametrize("m", [1, 37, 129])
def test_quant_act_ue8m0_ragged_and_ld(fp8rl, m):
    announce(f"quant_act_ue8m0 m={m}, lda > k, ld_scale > m")
    k = 384
    x = synth.normal_bf16((m, k + 64), 1.0, 200 + m, "cuda")
    x[:, 7] *= 50
    a = x[:, :k]
    ld = m + 5
    sbuf = torch.full((k // 128, ld), -7.0, dtype=torch.float32, device="cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128_ue8m0(a, scale=sbuf, ld_scale=ld)
    torch.cuda.synchronize()
    qo, so = ue8m0.quant_act_token_group128_ue8m0(u16(a), ld_scale=ld)
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s)[:, :m], so[:, :m], "scales")
    assert np.all(f32(s)[:, m:] == -7.0), "scale padding columns were written"


def test_quant_ue8m0_every_group_maximum(fp8rl):
    """One group per finite bf16 magnitude (0 included): the scale of every amax."""
    announce("quant_act_ue8m0 every group maximum")
    a = synth.sweep_group_maxima("cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128_ue8m0(a)
    torch.cuda.synchronize()
    qo, so = cref.quant_act_token_group128_ue8m0(u16(a))
    assert_scales_equal(f32(s), so, "scales")
    assert_codes_equal(u8(q), qo, "codes")


def test_quant_ue8m0_every_element_for_every_exponent(fp8rl):
    """Codes depend only on (x, k): a group maximum for every scale exponent (every
    binade's 1.75 * 2^e and the largest bf16), each with every |x| <= it, through
    the activation and the weight kernels."""
    announce("quant_ue8m0 exhaustive (x, k) sweep")
    a = synth.sweep_binade_groups("cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128_ue8m0(a)
    torch.cuda.synchronize()
    qo, so = cref.quant_act_token_group128_ue8m0(u16(a))
    assert set(np.unique(ue8m0.e8m0_byte(so))) == set(range(0, 248))
    assert_scales_equal(f32(s), so, "scales")
    assert_codes_equal(u8(q), qo, "codes")
    rows = (a.shape[0] // 128) * 128
    w = a[:rows].reshape(rows // 128, 128, 128).permute(1, 0, 2).reshape(128, -1).contiguous()
    qw, sw = fp8rl.fp8rl_quant_weight_block128_ue8m0(w)
    torch.cuda.synchronize()
    qwo, swo = cref.quant_weight_block128_ue8m0(u16(w))
    assert_scales_equal(f32(sw), swo, "weight scales")
    assert_codes_equal(u8(qw), qwo, "weight codes")


def ue8m0_operands(m, n, k, seed):
    """bf16 N(0,1) activations and N(0,0.02) weights with a gain 2^U(-8,8) per group and
    per block (every scale differs), quantised by the power-of-two oracle."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((m, k)).astype(np.float32)
    a *= np.repeat(2.0 ** rng.uniform(-8, 8, size=(m, k // 128)), 128, axis=1).astype(np.float32)
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    gw = 2.0 ** rng.uniform(-8, 8, size=(n // 128, k // 128))
    w *= np.repeat(np.repeat(gw, 128, axis=0), 128, axis=1).astype(np.float32)
    a16 = torch.from_numpy(a).to(torch.bfloat16)
    w16 = torch.from_numpy(w).to(torch.bfloat16)
    qa, sa = ue8m0.quant_act_token_group128_ue8m0(u16(a16))
    qw, sw = ue8m0.quant_weight_block128_ue8m0(u16(w16))
    return qa, sa, qw, sw


def run_dense_ue8m0(fp8rl, qa, sa, qw, sw, ldsa_pad=0):
    m, k = qa.shape
    sa_d = torch.zeros((k // 128, m + ldsa_pad), dtype=torch.float32, device="cuda")
    sa_d[:, :m] = to_dev(sa[:, :m])
    y = fp8rl.fp8rl_gemm_w8a8_block_ue8m0(to_dev(qa), sa_d, to_dev(qw), to_dev(sw))
    torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("m,n,k", [(1, 128, 128), (37, 384, 256), (129, 640, 384), (256, 1152, 1280), (200, 16512, 256), (300, 512, 256),
                                   (2048, 2048, 256), (2100, 2176, 384), (1000, 16384, 128)])
def test_gemm_ue8m0_shapes(fp8rl, m, n, k):
    announce(f"gemm_ue8m0 m={m} n={n} k={k}")
    qa, sa, qw, sw = ue8m0_operands(m, n, k, m * 5 + n + k)
    y = run_dense_ue8m0(fp8rl, qa, sa, qw, sw, ldsa_pad=3)
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), f"ue8m0 {m}x{n}x{k}")


def test_gemm_ue8m0_scale_per_operand_row_and_k_block(fp8rl):
    """Small-integer codes with a distinct power of two per (token, K block) and per
    (weight block, K block), including the extremes 2^-127 and 2^127 where the
    product stays finite: the result is exact, so any scale slip is visible."""
    announce("gemm_ue8m0 distinct exponents, exact products")
    rng = np.random.default_rng(31)
    m, n, k = 256, 256, 512
    codes = np.array([0x30, 0x38, 0x40, 0x44, 0xB8, 0xC0, 0x00], dtype=np.uint8)     # 0.5 1 2 3 -1 -2 0
    qa = codes[rng.integers(0, codes.size, (m, k))]
    qw = codes[rng.integers(0, codes.size, (n, k))]
    ea = rng.integers(-20, 20, (k // 128, m))
    ew = rng.integers(-20, 20, (n // 128, k // 128))
    # the extremes 2^-127 and 2^127, paired so that every product stays finite
    # (|block sum| <= 128 * 9 < 2^11, so scale products up to 2^117 are safe)
    ea[0, 0], ew[0, 0] = -127, 97
    ea[1, 1], ew[:, 1] = 127, -100
    sa = np.ldexp(1.0, ea).astype(np.float32)
    sw = np.ldexp(1.0, ew).astype(np.float32)
    y = run_dense_ue8m0(fp8rl, qa, sa, qw, sw)
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), "ue8m0 exact exponents")


def test_gemm_ue8m0_prefill_full_size_every_element(fp8rl):
    announce("gemm_ue8m0 prefill 8192x4096x24576, every element")
    a, w = synth.prefill_linear()
    qa, sa = cref.quant_act_token_group128_ue8m0(u16(a))
    qw, sw = cref.quant_weight_block128_ue8m0(u16(w))
    y = run_dense_ue8m0(fp8rl, qa, sa, qw, sw)
    check(y, dense_ref_by_rows(qa, sa, qw, sw), "ue8m0 prefill", dense_attribution(qa, sa, qw, sw, True), budget=32)


def test_gemm_ue8m0_deterministic(fp8rl):
    announce("gemm_ue8m0 determinism")
    qa, sa, qw, sw = ue8m0_operands(2304, 2304, 512, 5)
    args = (to_dev(qa), to_dev(sa), to_dev(qw), to_dev(sw))
    y1 = fp8rl.fp8rl_gemm_w8a8_block_ue8m0(*args)
    y2 = fp8rl.fp8rl_gemm_w8a8_block_ue8m0(*args)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("counts", [[3, 0, 130, 2, 0], [257, 0, 0, 64, 129, 1, 0, 300]])
def test_grouped_ue8m0_small(fp8rl, counts):
    announce(f"grouped_ue8m0 counts={counts}")
    g, n, k = len(counts), 384, 256
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    qa, sa, qw, sw = ue8m0_operands(r, g * n, k, sum(counts))
    qw, sw = qw.reshape(g, n, k), sw.reshape(g, n // 128, k // 128)
    y = fp8rl.fp8rl_grouped_gemm_w8a8_block_ue8m0(to_dev(qa), to_dev(sa), to_dev(qw), to_dev(sw), to_dev(offsets))
    torch.cuda.synchronize()
    check(y, gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, offsets), f"grouped ue8m0 {counts}")


@pytest.mark.parametrize("which", ["gate_up", "down"])
def test_grouped_ue8m0_moe_full_size_every_element(fp8rl, which):
    announce(f"grouped_ue8m0 MoE {which}, every element")
    moe = synth.moe_layer()
    off = moe["routing"].offsets.numpy()
    x = moe["x_gate_up"] if which == "gate_up" else moe["x_down"]
    wts = moe["w_gate_up"] if which == "gate_up" else moe["w_down"]
    g, n, k = wts.shape
    qa, sa = cref.quant_act_token_group128_ue8m0(u16(x))
    qw, sw = cref.quant_weight_block128_ue8m0(u16(wts.reshape(g * n, k)))
    qw, sw = qw.reshape(g, n, k), sw.reshape(g, n // 128, k // 128)
    y = fp8rl.fp8rl_grouped_gemm_w8a8_block_ue8m0(to_dev(qa), to_dev(sa), to_dev(qw), to_dev(sw), to_dev(off))
    torch.cuda.synchronize()
    check(y, gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, off), f"moe ue8m0 {which}",
          grouped_attribution(qa, sa, qw, sw, off, True), budget=8)
