"""GPU parity of the down-projection input step (h = bf16(SiLU(gate) * up), then
1x128 group quantisation) and of the quantised-row gather, against the CPU
oracle (section 2.1.1: down_proj / MoE fc2 quantised like every linear, their
activations dynamically per token and 128-wide group).

h is the correctly rounded bf16 of the exact value on both sides, so h, codes
and scales are all compared bit for bit; codes and scales only where h is
finite (NaN / inf activations are outside the quantiser's domain).

The grouped GEMM over gathered token rows (dispatch and expert product in one
pass) is checked against the oracle's gathered product and bit for bit against
the gather followed by the grouped GEMM."""
import numpy as np
import pytest
import torch

import synth
from oracle import act, cref, gemm, quant
from tests.gpu_util import (announce, assert_codes_equal, assert_scales_equal, bf16_to_f64, need_gpu, u8, u16,
                            f32)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fp8rl():
    need_gpu()
    import paper_2601_18150_amd as m
    m.load()
    return m


def assert_bits_equal(got: np.ndarray, want: np.ndarray, what: str):
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} of {want.size} differ; first at {i}: "
                             f"got {hex(int(got[i]))}, want {hex(int(want[i]))}")


def finite_groups(h: np.ndarray) -> np.ndarray:
    """[M][I/128] mask of groups whose bf16 values are all finite."""
    m, i = h.shape
    return ((h & 0x7F80) != 0x7F80).reshape(m, i // 128, 128).all(axis=2)


def check_fused(gu_t, inter, q, s, h, ld_scale=None, rows=None, big=False):
    """Compare GPU (q, s, h) with the oracle on the given rows (all when None)."""
    gu = u16(gu_t)
    gq, gs, gh = u8(q), f32(s), u16(h)
    if rows is not None:
        gu, gq, gh = gu[rows], gq[rows], gh[rows]
        gs = gs[:, rows]
    wh = act.silu_mul_bf16(gu, inter)
    assert_bits_equal(gh, wh, "h")
    ok = finite_groups(wh)
    m = wh.shape[0]
    if ok.all():
        wq, ws = (cref if big else quant).quant_act_token_group128(wh)
        assert_codes_equal(gq, wq, "codes")
        assert_scales_equal(gs[:, :m], ws[:, :m], "scales")
        return
    wq, ws = cref.quant_act_token_group128(np.where(np.repeat(ok, 128, axis=1), wh, 0).astype(np.uint16))
    mask = np.repeat(ok, 128, axis=1)
    assert_codes_equal(np.where(mask, gq, 0), np.where(mask, wq, 0), "codes (finite groups)")
    okt = ok.T
    assert_scales_equal(np.where(okt, gs[:, :m], 0), np.where(okt, ws[:, :m], 0), "scales (finite groups)")


def test_silu_mul_quant_tiny(fp8rl):
    announce("silu_mul_quant tiny 64x(2x512)")
    gu = synth.gate_up_output(seed=21, device="cuda", m=64, inter=512)
    q, s, h = fp8rl.fp8rl_silu_mul_quant_group128(gu, want_h=True)
    torch.cuda.synchronize()
    check_fused(gu, 512, q, s, h)


@pytest.mark.parametrize("m,inter", [(1, 128), (3, 384), (37, 640), (129, 256), (300, 1536)])
def test_silu_mul_quant_ragged_and_ld(fp8rl, m, inter):
    announce(f"silu_mul_quant ragged m={m} inter={inter}, ld_gu > 2I, ldh/ldq > I, ld_scale > m")
    full = synth.gate_up_output(seed=30 + m, device="cuda", m=m, inter=inter + 64, outlier_cols=4)
    gu = torch.cat([full[:, :inter], full[:, inter + 64:2 * inter + 64]], dim=1)
    gpad = torch.zeros((m, 2 * inter + 40), dtype=torch.bfloat16, device="cuda")
    gpad[:, :2 * inter] = gu
    ld = m + 3
    sbuf = torch.full((inter // 128, ld), -7.0, dtype=torch.float32, device="cuda")
    qbuf = torch.full((m, inter + 32), 0xAB, dtype=torch.uint8, device="cuda")
    hbuf = torch.full((m, inter + 16), -5.0, dtype=torch.bfloat16, device="cuda")
    q, s, h = fp8rl.fp8rl_silu_mul_quant_group128(gpad[:, :2 * inter], q=qbuf[:, :inter], scale=sbuf,
                                                  ld_scale=ld, h=hbuf[:, :inter])
    torch.cuda.synchronize()
    check_fused(gu, inter, q, s, h)
    assert np.all(f32(sbuf)[:, m:] == -7.0), "scale padding columns were written"
    assert np.all(u8(qbuf[:, inter:]) == 0xAB), "wrote codes past I"
    assert np.all(f32(hbuf.float()[:, inter:]) == -5.0), "wrote h past I"


def test_silu_mul_quant_without_h_matches(fp8rl):
    announce("silu_mul_quant h=NULL gives the same codes")
    gu = synth.gate_up_output(seed=22, device="cuda", m=200, inter=768)
    q1, s1, h = fp8rl.fp8rl_silu_mul_quant_group128(gu, want_h=True)
    q2, s2, none = fp8rl.fp8rl_silu_mul_quant_group128(gu)
    torch.cuda.synchronize()
    assert none is None
    assert torch.equal(q1, q2) and torch.equal(s1, s2)


@pytest.mark.parametrize("exponent", [127, None], ids=["up_in_1_2", "up_random_exponent"])
def test_silu_mul_exhaustive_pairs(fp8rl, exponent):
    """Every gate bit pattern against every up significand (2^24 pairs): h bit-exact
    with the correctly rounded value, including NaN / inf / subnormal gates, exp
    overflow and bf16 overflow and underflow of the product."""
    announce(f"silu_mul_quant exhaustive pairs, up exponent {exponent}")
    gu = synth.sweep_silu_pairs("cuda", exponent=exponent)
    q, s, h = fp8rl.fp8rl_silu_mul_quant_group128(gu, want_h=True)
    torch.cuda.synchronize()
    check_fused(gu, gu.shape[1] // 2, q, s, h, big=True)


def test_silu_fast_path_error_bound(fp8rl):
    """The premise of the kernel's fast path: wherever it is taken (|q| >= 2^-100, r
    finite), its fp32 result is within 10 fp32 ulps (the stated error bound) of the
    exact SiLU(g) * u, inside the 12-ulp guard around the bf16 half-way point.
    Measured for every gate bit pattern and up significand (relative error does not
    depend on up's exponent)."""
    import ctypes
    import os
    announce("silu fast-path error bound, 2^24 pairs")
    lib = ctypes.CDLL(os.path.join(os.path.dirname(fp8rl.LIB_PATH), "libfp8rl_probe.so"))
    fn = lib.fp8rl_probe_silu_fast
    fn.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_longlong, ctypes.c_void_p]
    i = np.arange(1 << 24, dtype=np.int64)
    gb = (i & 0xFFFF).astype(np.uint16)
    ub = (0x3F80 | (i >> 16 & 0x7F) | ((i >> 23) << 15)).astype(np.uint16)
    g_t = torch.from_numpy(gb.view(np.int16)).cuda()
    u_t = torch.from_numpy(ub.view(np.int16)).cuda()
    r_t = torch.empty(i.size, dtype=torch.float32, device="cuda")
    q_t = torch.empty_like(r_t)
    assert fn(g_t.data_ptr(), u_t.data_ptr(), r_t.data_ptr(), q_t.data_ptr(), i.size,
              torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    r = r_t.cpu().numpy().astype(np.float64)
    q = q_t.cpu().numpy().astype(np.float64)
    with np.errstate(all="ignore"):
        g = quant.bf16_bits_to_f32(gb).astype(np.float64)
        u = quant.bf16_bits_to_f32(ub).astype(np.float64)
        x = g / (1.0 + np.exp(-g)) * u
        taken = (np.abs(q) >= 2.0 ** -100) & (np.abs(r) <= np.finfo(np.float32).max)
        _, e = np.frexp(np.abs(r[taken]))
        ulp = np.ldexp(1.0, np.maximum(e - 1, -126) - 23)
        err = np.abs(r[taken] - x[taken]) / ulp
    assert taken.mean() > 0.5
    sys_max = float(err.max())
    print(f"fast path taken for {taken.mean():.4f} of pairs; max error {sys_max:.3f} ulp")
    assert sys_max <= 10.0, sys_max


def test_silu_mul_quant_dense_mlp_full_sampled(fp8rl):
    """Full Qwen3-8B MLP shape (8192 tokens, intermediate 12288): the whole step runs
    on the GPU, the oracle checks 256 seeded rows (the step is row-independent)."""
    announce("silu_mul_quant dense MLP 8192 x (2 x 12288), sampled rows")
    gu = synth.gate_up_output(seed=23, device="cuda", m=8192, inter=12288)
    q, s, h = fp8rl.fp8rl_silu_mul_quant_group128(gu, want_h=True)
    torch.cuda.synchronize()
    # 256 seeded rows, plus one row of every 16-row group at a varying offset, so that every
    # workgroup (64 consecutive tokens of one group) and every lane row of it is checked
    rng_rows = np.random.default_rng(23).choice(8192, 256, replace=False)
    grid_rows = np.arange(0, 8192, 16) + (np.arange(512) * 5) % 16
    rows = np.unique(np.concatenate([rng_rows, grid_rows, [8191]]))
    check_fused(gu, 12288, q, s, h, rows=rows)


def test_silu_mul_quant_mid_size_every_row(fp8rl):
    """1000 tokens x intermediate 12288: the launch that puts 32 tokens in a workgroup
    (fewer than 2048 workgroups of 64), with a ragged last block; every row checked."""
    announce("silu_mul_quant 1000 x (2 x 12288), every row")
    gu = synth.gate_up_output(seed=24, device="cuda", m=1000, inter=12288)
    q, s, h = fp8rl.fp8rl_silu_mul_quant_group128(gu, want_h=True)
    torch.cuda.synchronize()
    check_fused(gu, 12288, q, s, h)


def test_silu_mul_quant_zero_rows_is_noop(fp8rl):
    announce("silu_mul_quant m=0")
    gu = torch.empty((0, 512), dtype=torch.bfloat16, device="cuda")
    q, s, h = fp8rl.fp8rl_silu_mul_quant_group128(gu, want_h=True)
    torch.cuda.synchronize()
    assert q.shape == (0, 256) and h.shape == (0, 256)


def test_gather_moe_dispatch_bit_exact(fp8rl):
    """Qwen3-30B-A3B dispatch: 4096 tokens x 2048 quantised once, gathered to the
    32768 expert-grouped rows of a Zipf(1.1) top-8 routing."""
    announce("gather_rows_fp8 MoE dispatch 4096 -> 32768 rows, k=2048")
    routing = synth.moe_routing(seed=6, tokens=4096, experts=128, topk=8)
    x_tok = synth.normal_bf16((4096, 2048), 1.0, 6 + 11, "cpu")
    qo, so = cref.quant_act_token_group128(u16(x_tok))
    index = routing.token_of_row
    gq_want, gs_want = act.gather_rows_fp8(qo, so, index.numpy())
    q = torch.from_numpy(qo).cuda()
    s = torch.from_numpy(so).cuda()
    idx = index.to(torch.int32).cuda()
    gq, gs = fp8rl.fp8rl_gather_rows_fp8(q, s, idx)
    torch.cuda.synchronize()
    assert_codes_equal(u8(gq), gq_want, "gathered codes")
    assert_scales_equal(f32(gs), gs_want, "gathered scales")


@pytest.mark.parametrize("src_rows,rows,k", [(1, 5, 128), (7, 3, 384), (300, 1000, 640), (50, 0, 256)])
def test_gather_ragged_and_ld(fp8rl, src_rows, rows, k):
    announce(f"gather_rows_fp8 src={src_rows} rows={rows} k={k}, padded lds")
    rng = np.random.default_rng(src_rows * 1000 + rows)
    codes = rng.integers(0, 256, (src_rows, k + 48), dtype=np.uint8)
    scales = rng.standard_normal((k // 128, src_rows + 5)).astype(np.float32)
    index = rng.integers(0, src_rows, rows).astype(np.int64)
    qd = torch.full((rows, k + 16), 0xCD, dtype=torch.uint8, device="cuda")
    sd = torch.full((k // 128, rows + 2), -9.0, dtype=torch.float32, device="cuda")
    q_src = torch.from_numpy(codes).cuda()[:, :k]
    s_src = torch.from_numpy(scales).cuda()
    fp8rl.fp8rl_gather_rows_fp8(q_src, s_src, torch.from_numpy(index.astype(np.int32)).cuda(),
                                q_dst=qd[:, :k], s_dst=sd)
    torch.cuda.synchronize()
    wq, ws = act.gather_rows_fp8(codes[:, :k], scales[:, :src_rows], index)
    assert_codes_equal(u8(qd)[:, :k], wq, "codes")
    assert_scales_equal(f32(sd)[:, :rows], ws, "scales")
    assert np.all(u8(qd)[:, k:] == 0xCD), "wrote past k"
    assert np.all(f32(sd)[:, rows:] == -9.0), "wrote scale padding"


def test_gather_then_gemm_equals_gemm_of_gathered_rows(fp8rl):
    """Gathering quantised rows and quantising gathered bf16 rows give the same GEMM
    input, so the grouped GEMM sees identical operands either way."""
    announce("gather vs quantise-after-gather, 512 tokens -> 1024 rows")
    x = synth.normal_bf16((512, 1024), 1.0, 40, "cuda")
    idx = torch.from_numpy(np.random.default_rng(40).integers(0, 512, 1024).astype(np.int32)).cuda()
    q, s = fp8rl.fp8rl_quant_act_token_group128(x)
    gq, gs = fp8rl.fp8rl_gather_rows_fp8(q, s, idx)
    q2, s2 = fp8rl.fp8rl_quant_act_token_group128(x[idx.long()].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(gq, q2) and torch.equal(gs, s2)


def _gathered_case(rng, t, counts, n, k, lda_pad=0, ldsa_pad=0):
    """Token table [t][k] (oracle-quantised bf16 N(0,1) rows), expert weights, a
    routing index with repeats and unused tokens."""
    g = len(counts)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    a16 = torch.from_numpy(rng.standard_normal((t, k)).astype(np.float32)).to(torch.bfloat16)
    w16 = torch.from_numpy((rng.standard_normal((g * n, k)) * 0.02).astype(np.float32)).to(torch.bfloat16)
    qa, sa = cref.quant_act_token_group128(u16(a16))
    qw, sw = cref.quant_weight_block128(u16(w16))
    index = rng.integers(0, t, size=r).astype(np.int32)
    qa_d = torch.zeros((t, k + lda_pad), dtype=torch.uint8, device="cuda")
    qa_d[:, :k] = torch.from_numpy(qa).cuda()
    sa_d = torch.zeros((k // 128, t + ldsa_pad), dtype=torch.float32, device="cuda")
    sa_d[:, :t] = torch.from_numpy(sa).cuda()
    dev = {"qa": qa_d[:, :k], "sa": sa_d, "index": torch.from_numpy(index).cuda(),
           "qw": torch.from_numpy(qw.reshape(g, n, k)).cuda(),
           "sw": torch.from_numpy(sw.reshape(g, n // 128, k // 128)).cuda(),
           "offsets": torch.from_numpy(offsets).cuda()}
    host = (qa, sa, index, qw.reshape(g, n, k), sw.reshape(g, n // 128, k // 128), offsets)
    return dev, host


@pytest.mark.parametrize("t,counts,n,k", [
    (37, [5, 0, 130, 1, 0, 64], 384, 256),            # 256x128 tiles (K <= 1024)
    (300, [257, 0, 3, 129], 256, 1152),               # 128x128 tiles (K > 1024)
    (700, list(range(0, 400, 7)), 640, 384),          # > 512 tiles: several per persistent workgroup
    (700, list(range(0, 400, 7)), 768, 1280),
])
def test_grouped_gathered_matches_oracle(fp8rl, t, counts, n, k):
    """The grouped product over gathered token rows against the oracle: repeated and
    unused tokens, empty and ragged experts, a token-table row pitch > K and ld_sa > T."""
    announce(f"grouped gathered t={t} experts={len(counts)} n={n} k={k}")
    rng = np.random.default_rng(t + n + k)
    dev, host = _gathered_case(rng, t, counts, n, k, lda_pad=32, ldsa_pad=3)
    y = fp8rl.fp8rl_grouped_gemm_w8a8_block_gathered(dev["qa"], dev["sa"], dev["index"], dev["qw"], dev["sw"],
                                                     dev["offsets"])
    torch.cuda.synchronize()
    ref = gemm.grouped_gemm_gathered_ref_fp64(*host)
    ok, worst, _ = gemm.tolerance_check(bf16_to_f64(y), ref)
    assert ok, f"worst |err|/bound {worst:.3f}"


@pytest.mark.parametrize("which", ["gate_up", "down"])
def test_grouped_gathered_bit_identical_to_gather_then_grouped(fp8rl, which):
    """Qwen3-30B-A3B expert shapes, 4096 tokens routed top-8 (Zipf loads, empty experts):
    exactly the bits of fp8rl_gather_rows_fp8 followed by the grouped GEMM."""
    announce(f"grouped gathered vs gather + grouped, MoE {which}")
    lay = synth.moe_layer(device="cuda")
    rt = lay["routing"]
    off = rt.offsets.cuda()
    idx = rt.token_of_row.to(torch.int32).cuda()
    wts = lay["w_gate_up"] if which == "gate_up" else lay["w_down"]
    g, n, k = wts.shape
    tokens = synth.normal_bf16((4096, k), 1.0, 77, "cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128(tokens)
    qw, sw = fp8rl.fp8rl_quant_weight_block128(wts.reshape(g * n, k))
    qw, sw = qw.reshape(g, n, k), sw.reshape(g, n // 128, k // 128)
    y1 = fp8rl.fp8rl_grouped_gemm_w8a8_block_gathered(q, s, idx, qw, sw, off)
    gq, gs = fp8rl.fp8rl_gather_rows_fp8(q, s, idx)
    y2 = fp8rl.fp8rl_grouped_gemm_w8a8_block(gq, gs, qw, sw, off)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_grouped_gathered_out_of_range_index_is_clamped(fp8rl):
    """Indices outside [0, T) read the nearest valid token (never out of bounds)."""
    announce("grouped gathered clamped indices")
    rng = np.random.default_rng(9)
    dev, host = _gathered_case(rng, 50, [40, 24], 256, 256)
    bad = dev["index"].clone()
    bad[::5] = 1000
    bad[1::7] = -3
    y = fp8rl.fp8rl_grouped_gemm_w8a8_block_gathered(dev["qa"], dev["sa"], bad, dev["qw"], dev["sw"],
                                                     dev["offsets"])
    good = bad.clamp(0, 49)
    y2 = fp8rl.fp8rl_grouped_gemm_w8a8_block_gathered(dev["qa"], dev["sa"], good, dev["qw"], dev["sw"],
                                                      dev["offsets"])
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))
