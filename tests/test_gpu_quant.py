"""GPU parity of the quantisation kernels against the CPU oracle: codes and
scales must match bit for bit (section 2.1.1, Eq. (1); 128x128 weight blocks,
1x128 per-token activation groups, fp32 scales)."""
import numpy as np
import pytest
import torch

import synth
from oracle import cref, quant
from tests.gpu_util import announce, assert_codes_equal, assert_scales_equal, need_gpu, u8, u16, f32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fp8rl():
    need_gpu()
    import paper_2601_18150_amd as m
    m.load()
    return m


def test_quant_weight_tiny(fp8rl):
    announce("quant_weight tiny 512x512")
    _, w = synth.tiny_linear(device="cuda")
    q, s = fp8rl.fp8rl_quant_weight_block128(w)
    torch.cuda.synchronize()
    qo, so = quant.quant_weight_block128(u16(w))
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s), so, "scales")


def test_quant_weight_special_blocks_and_ld(fp8rl):
    announce("quant_weight special blocks, ldw > k, ldq > k")
    n, k = 384, 640
    w = synth.normal_bf16((n, k), 0.02, 77, "cuda")
    synth.plant_special_blocks(w, 78, frac_zero=2 / 15, frac_large=2 / 15)
    wf = w.float()
    wf[128:256, 0:128] *= 1e-38            # subnormal scale (amax < 448 * 2^-126)
    wf[256:384, 128:256] = 2.0 ** -133     # smallest bf16 subnormal everywhere
    wf[300, 200] = -(2.0 ** -133)
    wf[0:128, 512:640] = 0.0
    wf[5, 515] = -3.0                      # single nonzero block
    w = wf.to(torch.bfloat16)
    wpad = torch.zeros((n, k + 24), dtype=torch.bfloat16, device="cuda")
    wpad[:, :k] = w
    qbuf = torch.full((n, k + 48), 0xAB, dtype=torch.uint8, device="cuda")
    q, s = fp8rl.fp8rl_quant_weight_block128(wpad[:, :k], q=qbuf[:, :k])
    torch.cuda.synchronize()
    qo, so = quant.quant_weight_block128(u16(w))
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s), so, "scales")
    assert np.all(u8(qbuf[:, k:]) == 0xAB), "wrote past k in a padded row"


@pytest.mark.parametrize("layer", [0, 35])
def test_quant_weight_requant_layers_full(fp8rl, layer):
    """Full matrices of the 36-layer resync workload (first and last layer)."""
    for name in synth.QWEN3_8B_LINEARS:
        announce(f"quant_weight requant layer {layer} {name}")
        w, zeros, larges = synth.requant_matrix(layer, name, device="cuda")
        q, s = fp8rl.fp8rl_quant_weight_block128(w)
        torch.cuda.synchronize()
        qo, so = cref.quant_weight_block128(u16(w))
        assert_codes_equal(u8(q), qo, f"{name} codes")
        assert_scales_equal(f32(s), so, f"{name} scales")
        sh = f32(s)
        for (i, j) in zeros:
            assert sh[i, j] == 1.0
        for (i, j) in larges[:4]:
            assert sh[i, j] > 1e30


def test_quant_weight_exhaustive_element_map(fp8rl):
    """Every (x, amax) bf16 pair with |x| <= amax, through the production weight kernel."""
    announce("quant_weight exhaustive sweep")
    w = synth.sweep_weight_blocks("cuda")
    q, s = fp8rl.fp8rl_quant_weight_block128(w)
    torch.cuda.synchronize()
    qo, so = cref.quant_weight_block128(u16(w))
    assert_scales_equal(f32(s), so, "scales")
    assert_codes_equal(u8(q), qo, "codes")


def test_quant_weight_batched_mixed_jobs(fp8rl):
    """70 matrices (two launches of at most 64 jobs) of assorted shapes, padded
    rows, empty jobs and special blocks: each equal to the oracle, padding untouched."""
    announce("quant_weight batched: 70 mixed jobs")
    rng = np.random.default_rng(5)
    ws, qs, scs, pads, ref = [], [], [], [], []
    for i in range(70):
        n = 0 if i in (3, 40, 69) else 128 * int(rng.integers(1, 5))
        k = 128 * int(rng.integers(1, 6))
        pw, pq = (8 * int(rng.integers(0, 3)), 16 * int(rng.integers(0, 3))) if i % 3 == 0 else (0, 0)
        w = synth.normal_bf16((max(n, 1), k), 0.02, 1000 + i, "cuda")[:n]
        if n and i % 5 == 1:
            synth.plant_special_blocks(w, 2000 + i, frac_zero=0.3, frac_large=0.3)
        wbuf = torch.zeros((n, k + pw), dtype=torch.bfloat16, device="cuda")
        wbuf[:, :k] = w
        qbuf = torch.full((n, k + pq), 0xAB, dtype=torch.uint8, device="cuda")
        ws.append(wbuf[:, :k])
        qs.append(qbuf[:, :k])
        scs.append(torch.full((n // 128, k // 128), -1.0, dtype=torch.float32, device="cuda"))
        pads.append((qbuf, k))
        ref.append(quant.quant_weight_block128(u16(w)) if n else None)
    out = fp8rl.fp8rl_quant_weight_block128_batched(ws, qs, scs)
    torch.cuda.synchronize()
    for i, ((q, s), r, (qbuf, k)) in enumerate(zip(out, ref, pads)):
        if r is None:
            assert q.numel() == 0
            continue
        assert_codes_equal(u8(q), r[0], f"job {i} codes")
        assert_scales_equal(f32(s), r[1], f"job {i} scales")
        assert np.all(u8(qbuf[:, k:]) == 0xAB), f"job {i} wrote past k in a padded row"


def test_quant_weight_batched_requant_layer(fp8rl):
    """The four matrices of one resync layer in one call: equal to the C oracle."""
    announce("quant_weight batched: resync layer 35")
    mats = [synth.requant_matrix(35, name, device="cuda")[0] for name in synth.QWEN3_8B_LINEARS]
    out = fp8rl.fp8rl_quant_weight_block128_batched(mats)
    torch.cuda.synchronize()
    for name, w, (q, s) in zip(synth.QWEN3_8B_LINEARS, mats, out):
        qo, so = cref.quant_weight_block128(u16(w))
        assert_codes_equal(u8(q), qo, f"{name} codes")
        assert_scales_equal(f32(s), so, f"{name} scales")


def test_quant_weight_batched_exhaustive_element_map(fp8rl):
    """The exhaustive (x, amax) sweep through the batched kernel, split into three
    jobs of unequal row ranges."""
    announce("quant_weight batched exhaustive sweep")
    w = synth.sweep_weight_blocks("cuda")
    nb = w.shape[0] // 128
    cuts = [0, 128 * (nb // 3), 128 * (nb // 3 + nb // 5), w.shape[0]]
    parts = [w[a:b] for a, b in zip(cuts, cuts[1:])]
    out = fp8rl.fp8rl_quant_weight_block128_batched(parts)
    torch.cuda.synchronize()
    qo, so = cref.quant_weight_block128(u16(w))
    assert_scales_equal(np.concatenate([f32(s) for _, s in out]), so, "scales")
    assert_codes_equal(np.concatenate([u8(q) for q, _ in out]), qo, "codes")


def test_quant_act_tiny(fp8rl):
    announce("quant_act tiny 64x512")
    a, _ = synth.tiny_linear(device="cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128(a)
    torch.cuda.synchronize()
    qo, so = quant.quant_act_token_group128(u16(a))
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s), so, "scales")


@pytest.mark.parametrize("m", [1, 3, 37, 129])
def test_quant_act_ragged_m_and_ld(fp8rl, m):
    announce(f"quant_act ragged m={m}, lda > k, ld_scale > m")
    k = 384
    x = synth.normal_bf16((m, k + 64), 1.0, 100 + m, "cuda")
    x[:, 7] *= 50
    if m > 2:
        x[2, 128:256] = 0.0
        x[2, 130] = -0.0
    a = x[:, :k]
    ld = m + 5
    sbuf = torch.full((k // 128, ld), -7.0, dtype=torch.float32, device="cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128(a, scale=sbuf, ld_scale=ld)
    torch.cuda.synchronize()
    qo, so = quant.quant_act_token_group128(u16(a), ld_scale=ld)
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s)[:, :m], so[:, :m], "scales")
    assert np.all(f32(s)[:, m:] == -7.0), "scale padding columns were written"


def test_quant_act_prefill_outliers_full(fp8rl):
    """Full 8192x4096 prefill activations with outlier channels (C oracle on all of it)."""
    announce("quant_act prefill 8192x4096")
    a, _ = synth.prefill_linear(device="cuda", n=128)
    q, s = fp8rl.fp8rl_quant_act_token_group128(a)
    torch.cuda.synchronize()
    qo, so = cref.quant_act_token_group128(u16(a))
    assert_codes_equal(u8(q), qo, "codes")
    assert_scales_equal(f32(s), so, "scales")


def test_quant_act_exhaustive_element_map(fp8rl):
    """Every (x, amax) bf16 pair with |x| <= amax, through the production activation kernel."""
    announce("quant_act exhaustive sweep")
    a = synth.sweep_act_groups("cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128(a)
    torch.cuda.synchronize()
    qo, so = cref.quant_act_token_group128(u16(a))
    assert_scales_equal(f32(s), so, "scales")
    assert_codes_equal(u8(q), qo, "codes")


def test_quant_deterministic_and_side_stream(fp8rl):
    announce("quant determinism on a side stream")
    a, w = synth.tiny_linear(device="cuda", m=300, k=1024, n=1024)
    q1, s1 = fp8rl.fp8rl_quant_weight_block128(w)
    p1, t1 = fp8rl.fp8rl_quant_act_token_group128(a)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        q2, s2 = fp8rl.fp8rl_quant_weight_block128(w)
        p2, t2 = fp8rl.fp8rl_quant_act_token_group128(a)
    torch.cuda.synchronize()
    assert torch.equal(q1, q2) and torch.equal(s1, s2)
    assert torch.equal(p1, p2) and torch.equal(t1, t2)


def test_quant_zero_size_is_noop(fp8rl):
    announce("quant zero-size")
    a = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    q, s = fp8rl.fp8rl_quant_act_token_group128(a)
    torch.cuda.synchronize()
    assert q.shape == (0, 256)
