"""GPU parity of the blockwise-scaled FP8 GEMMs (dense and grouped) against the
fp64 oracle on the same FP8 codes and scales.

Codes and scales given to the GPU are made by the oracle (or drawn directly as
random codes), never by the GPU quantisers.  Pass criterion per element:
|gpu - ref| <= 4e-3 |ref| + 1e-3 rms(ref), rms over the call's whole output; every
output element of every call is compared."""
import numpy as np
import pytest
import torch

import synth
from oracle import cref, gemm
from tests import mfma_model
from tests.gpu_util import announce, bf16_to_f64, need_gpu, u16

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fp8rl():
    need_gpu()
    import paper_2601_18150_amd as m
    m.load()
    return m


def to_dev(x: np.ndarray, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to("cuda") if dtype is None else t.to("cuda").to(dtype)


def rand_codes(shape, rng):
    c = rng.integers(0, 256, size=shape, dtype=np.uint8)
    c[(c & 0x7F) == 0x7F] ^= 0x01           # no NaN codes
    return c


def rand_scales(shape, rng):
    return (2.0 ** rng.uniform(-12, -2, size=shape)).astype(np.float32)


def check(y_gpu: torch.Tensor, y_ref: np.ndarray, what: str, attribute=None, budget=0):
    """Every element within |gpu - ref| <= 4e-3 |ref| + 1e-3 rms(ref) of the fp64 oracle.

    The FP8 MFMA truncates products that share a group of 8 K positions with a much
    larger one (tests/test_gpu_mfma_precision.py), so on operands with large in-block
    dynamic range a few elements can miss that tolerance whatever the kernel does.
    Such elements are allowed only where a test names a budget: at most `budget` of
    them, and each must equal, within the same tolerance, `attribute(rows, cols)`:
    the kernel's arithmetic emulated with the instruction's measured summation
    (tests/mfma_model.py)."""
    got = bf16_to_f64(y_gpu)
    ok, worst, rms = gemm.tolerance_check(got, y_ref)
    if ok:
        return
    bound = 4e-3 * np.abs(y_ref) + 1e-3 * rms
    err = np.abs(got - y_ref)
    bad = np.nonzero(err > bound)
    nbad = bad[0].size
    ratio = err[bad] / bound[bad]
    for t in np.argsort(ratio)[::-1][:5]:
        idx = tuple(int(b[t]) for b in bad)
        print(f"  at {idx}: gpu {got[idx]!r} ref {y_ref[idx]!r} err {err[idx]:.4g} ratio {ratio[t]:.3f}")
    assert attribute is not None and nbad <= budget, \
        f"{what}: {nbad} elements outside the tolerance, worst |err|/bound = {worst:.3f} (rms {rms:.4g})"
    emu = attribute(*bad)
    off_model = np.abs(got[bad] - emu) > bound[bad]
    assert not off_model.any(), f"{what}: {int(off_model.sum())} of {nbad} elements outside the tolerance are " \
        "not the instruction's summation either"
    print(f"{what}: {nbad} of {y_ref.size} elements outside the tolerance against the fp64 oracle (worst ratio "
          f"{worst:.3f}), each equal to the emulated FP8 MFMA summation within it")


def dense_attribution(qa, sa, qw, sw, pow2_scales=False):
    """attribute() for check(): the dense kernel emulated with the instruction model."""
    def emulate(rows, cols):
        return mfma_model.gemm_elements(qa[rows], np.asarray(sa)[:, rows].T, qw[cols], np.asarray(sw)[cols // 128],
                                        pow2_scales)
    return emulate


def grouped_attribution(qa, sa, qw, sw, offsets, pow2_scales=False):
    """attribute() for check(): the grouped kernel emulated per element with its expert's weights."""
    def emulate(rows, cols):
        e = np.searchsorted(np.asarray(offsets), rows, side="right") - 1
        return mfma_model.gemm_elements(qa[rows], np.asarray(sa)[:, rows].T, qw[e, cols], sw[e, cols // 128],
                                        pow2_scales)
    return emulate


def dense_ref_by_rows(qa, sa, qw, sw, chunk=1024):
    """The oracle's dense product (dequantise, then an fp64 matmul), evaluated over
    row chunks so that the dequantised weight is formed once: row for row the same
    numbers as gemm.gemm_ref_fp64."""
    wd_t = np.ascontiguousarray(gemm.dequant_weight(qw, sw).T)
    m = qa.shape[0]
    ref = np.empty((m, qw.shape[0]), np.float64)
    for r0 in range(0, m, chunk):
        r1 = min(m, r0 + chunk)
        np.matmul(gemm.dequant_act(qa[r0:r1], sa[:, r0:r1]), wd_t, out=ref[r0:r1])
    return ref


def run_dense(fp8rl, qa, sa, qw, sw, lda_pad=0, ldy_pad=0, ldsa_pad=0):
    m, k = qa.shape
    n = qw.shape[0]
    qa_d = torch.zeros((m, k + lda_pad), dtype=torch.uint8, device="cuda")
    qa_d[:, :k] = to_dev(qa)
    sa_d = torch.zeros((k // 128, m + ldsa_pad), dtype=torch.float32, device="cuda")
    sa_d[:, :m] = to_dev(sa[:, :m])
    y = torch.zeros((m, n + ldy_pad), dtype=torch.bfloat16, device="cuda")
    fp8rl.fp8rl_gemm_w8a8_block(qa_d[:, :k], sa_d, to_dev(qw), to_dev(sw), y=y[:, :n])
    torch.cuda.synchronize()
    if ldy_pad:
        assert torch.all(y[:, n:] == 0), "wrote past n in a padded output row"
    return y[:, :n]


def test_gemm_tiny_config(fp8rl):
    announce("gemm tiny 64x512x512 from oracle-quantised bf16")
    a, w = synth.tiny_linear()
    qa, sa = cref.quant_act_token_group128(u16(a))
    qw, sw = cref.quant_weight_block128(u16(w))
    y = run_dense(fp8rl, qa, sa, qw, sw)
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), "tiny")


def quantised_operands(m, n, k, seed):
    """Realistic FP8 operands: bf16 N(0,1) activations and N(0,0.02) weights, with a
    distinct random gain 2^U(-8,8) per (token, group) and per 128x128 weight block
    so that every scale differs (a wrong scale index is a gross error), quantised
    by the oracle."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((m, k)).astype(np.float32)
    a *= np.repeat(2.0 ** rng.uniform(-8, 8, size=(m, k // 128)), 128, axis=1).astype(np.float32)
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    gw = 2.0 ** rng.uniform(-8, 8, size=(n // 128, k // 128))
    w *= np.repeat(np.repeat(gw, 128, axis=0), 128, axis=1).astype(np.float32)
    a16 = torch.from_numpy(a).to(torch.bfloat16)
    w16 = torch.from_numpy(w).to(torch.bfloat16)
    qa, sa = cref.quant_act_token_group128(u16(a16))
    qw, sw = cref.quant_weight_block128(u16(w16))
    return qa, sa, qw, sw


@pytest.mark.parametrize("m,n,k,pads", [
    (1, 128, 128, (0, 0, 0)),
    (37, 384, 256, (16, 8, 3)),
    (100, 256, 512, (0, 0, 0)),
    (129, 640, 384, (32, 24, 1)),
    (200, 1152, 1280, (16, 8, 2)),
    (256, 256, 128, (0, 0, 0)),
    (160, 33280, 256, (16, 8, 3)),
    (300, 512, 256, (0, 0, 0)),
    (2048, 2048, 256, (0, 0, 0)),
    (2100, 2176, 384, (16, 8, 5)),
])
def test_gemm_shapes(fp8rl, m, n, k, pads):
    announce(f"gemm m={m} n={n} k={k} pads={pads}")
    qa, sa, qw, sw = quantised_operands(m, n, k, m * 7 + n + k)
    y = run_dense(fp8rl, qa, sa, qw, sw, *pads)
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), f"{m}x{n}x{k}")


@pytest.mark.parametrize("m,n,k", [(1000, 16384, 128), (1500, 8192, 384)])
def test_gemm_many_tiles_per_workgroup(fp8rl, m, n, k):
    """More 128x128 tiles than the persistent grid has workgroups (512): each workgroup
    runs several tiles through one pipeline, with ragged last rows; K = 128 makes every
    K step a tile boundary."""
    announce(f"gemm persistent m={m} n={n} k={k}")
    qa, sa, qw, sw = quantised_operands(m, n, k, m + n + k)
    y = run_dense(fp8rl, qa, sa, qw, sw)
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), f"{m}x{n}x{k}")


@pytest.mark.parametrize("m,n,k", [(2048, 2048, 256), (300, 384, 384), (256, 256, 256)])
def test_gemm_largest_row_pitch(fp8rl, m, n, k):
    """Operand row pitches of 2^24 - 16 bytes, the largest the entry point accepts: the
    DMA's 32-bit in-tile offsets reach 255 rows x pitch (256x256 tiles, 4.28e9 of the 2^32
    range), 127 rows (128x128 tiles) and 63 rows (64x64 decode tiles).  Only the first k
    bytes of each row are written; the buffers are 2048 x 16 MiB for the first case."""
    announce(f"gemm largest row pitch m={m} n={n} k={k}")
    pitch = (1 << 24) - 16
    qa, sa, qw, sw = quantised_operands(m, n, k, m + n + 5 * k)
    a_big = torch.empty((m, pitch), dtype=torch.uint8, device="cuda")
    w_big = torch.empty((n, pitch), dtype=torch.uint8, device="cuda")
    a_big[:, :k] = to_dev(qa)
    w_big[:, :k] = to_dev(qw)
    y = fp8rl.fp8rl_gemm_w8a8_block(a_big[:, :k], to_dev(sa), w_big[:, :k], to_dev(sw))
    torch.cuda.synchronize()
    del a_big, w_big
    torch.cuda.empty_cache()
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), f"pitch {pitch} {m}x{n}x{k}")


def test_gemm_full_range_codes(fp8rl):
    """Uniformly random codes over the whole E4M3 range: products from 2^-18 to 448^2 in
    every K group, with heavy cancellation.  The stated tolerance against the fp64
    oracle on every element, except a budgeted handful where the FP8 MFMA's own
    summation (products truncated below the largest one of their group of 8,
    tests/test_gpu_mfma_precision.py) is what misses it."""
    announce("gemm full-range random codes")
    rng = np.random.default_rng(2048 * 7 + 2048 + 256)
    m, n, k = 2048, 2048, 256
    qa, qw = rand_codes((m, k), rng), rand_codes((n, k), rng)
    sa, sw = rand_scales((k // 128, m), rng), rand_scales((n // 128, k // 128), rng)
    y = run_dense(fp8rl, qa, sa, qw, sw)
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), "full-range codes", dense_attribution(qa, sa, qw, sw), budget=16)


def test_gemm_k_block_accumulates_in_fp32(fp8rl):
    """Cancellation inside one 128-wide K block: 448*448 - 448*448 + x*x must leave x*x.

    With fp32 accumulation (24-bit significand) the small term survives in any
    summation order as long as it is >= 2^-6 (half an fp32 ulp of 200704 is
    2^-7); a narrower accumulator would drop it."""
    announce("gemm accumulation precision probe")
    from oracle import e4m3
    small = np.array([4.0, 1.0, 0.5, 0.25, 0.125], np.float32)
    m, n, k = 16, 128, 128
    qa = np.zeros((m, k), np.uint8)
    qw = np.zeros((n, k), np.uint8)
    for i, x in enumerate(small):
        for pos in range(3):                   # put the big pair at different K positions
            r = i * 3 + pos
            c0, c1, c2 = [(pos * 40 + d * 13) % 128 for d in range(3)]
            qa[r, [c0, c1, c2]] = e4m3.encode(np.array([448.0, 448.0, x], np.float32))
            qw[r % n, [c0, c1, c2]] = e4m3.encode(np.array([448.0, -448.0, x], np.float32))
    ones_a = np.ones((1, m), np.float32)
    ones_w = np.ones((1, 1), np.float32)
    y = bf16_to_f64(run_dense(fp8rl, qa, ones_a, qw, ones_w))
    want = gemm.gemm_ref_fp64(qa, ones_a, qw, ones_w)
    diag = [(r, y[r, r % n], want[r, r % n]) for r in range(15)]
    print("probe (row, gpu, exact):", diag)
    assert np.array_equal(y, want)


def test_gemm_exact_small_integers(fp8rl):
    """Integer codes with unit scales: the exact result is an integer < 256, so bf16 holds it exactly."""
    announce("gemm exact integers")
    rng = np.random.default_rng(5)
    m, n, k = 70, 256, 256
    ia = rng.integers(-1, 2, size=(m, k))
    iw = rng.integers(-1, 2, size=(n, k))
    from oracle import e4m3
    qa, qw = e4m3.encode(ia.astype(np.float32)), e4m3.encode(iw.astype(np.float32))
    ones_a = np.ones((k // 128, m), np.float32)
    ones_w = np.ones((n // 128, k // 128), np.float32)
    y = run_dense(fp8rl, qa, ones_a, qw, ones_w)
    want = (ia @ iw.T).astype(np.float64)
    assert np.abs(want).max() < 256
    assert np.array_equal(bf16_to_f64(y), want)


def test_gemm_decode_layer(fp8rl):
    """M=256 decode tokens through the four Qwen3-8B linears of one layer (full outputs)."""
    acts = synth.decode_activations()
    ws = synth.layer_weights(0)
    for name, (k, n) in synth.QWEN3_8B_LINEARS.items():
        announce(f"gemm decode M=256 {name} {k}->{n}")
        x = acts["inter"] if k == 12288 else acts["h"]
        qa, sa = cref.quant_act_token_group128(u16(x))
        qw, sw = cref.quant_weight_block128(u16(ws[name]))
        y = run_dense(fp8rl, qa, sa, qw, sw)
        check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), name)


def run_dense_ws(fp8rl, qa, sa, qw, sw, ws_bytes=None):
    """The split-K entry point with the workspace it asks for (or ws_bytes)."""
    m, k = qa.shape
    n = qw.shape[0]
    need = fp8rl.fp8rl_gemm_w8a8_block_workspace_size(m, n, k)
    nbytes = need if ws_bytes is None else ws_bytes
    ws = torch.full((max(nbytes, 16) // 4,), float("nan"), dtype=torch.float32, device="cuda")
    y = fp8rl.fp8rl_gemm_w8a8_block_ws(to_dev(qa), to_dev(sa), to_dev(qw), to_dev(sw), ws[: nbytes // 4])
    torch.cuda.synchronize()
    return y, need


def test_gemm_split_k_decode_layer(fp8rl):
    """The four decode linears through the split-K entry point (workspace pre-filled with NaN:
    every partial the reduction reads must have been written)."""
    acts = synth.decode_activations()
    ws = synth.layer_weights(35)
    for name, (k, n) in synth.QWEN3_8B_LINEARS.items():
        announce(f"gemm split-K decode M=256 {name} {k}->{n}")
        x = acts["inter"] if k == 12288 else acts["h"]
        qa, sa = cref.quant_act_token_group128(u16(x))
        qw, sw = cref.quant_weight_block128(u16(ws[name]))
        y, need = run_dense_ws(fp8rl, qa, sa, qw, sw)
        assert (need > 0) == (name == "down"), (name, need)   # qkv, o_proj: unsplit 64x64 tiles
        check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), f"split-K {name}")


@pytest.mark.parametrize("m,n,k", [(1, 128, 1024), (37, 384, 13 * 128), (100, 256, 2048), (255, 640, 33 * 128)])
def test_gemm_split_k_ragged(fp8rl, m, n, k):
    """Ragged M and N tails and a K range that does not divide evenly among the splits."""
    announce(f"gemm split-K m={m} n={n} k={k}")
    qa, sa, qw, sw = quantised_operands(m, n, k, m * 11 + n + k)
    y, need = run_dense_ws(fp8rl, qa, sa, qw, sw)
    assert need > 0
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), f"split-K {m}x{n}x{k}")
    y2, _ = run_dense_ws(fp8rl, qa, sa, qw, sw)
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16)), "split-K result not deterministic"


def test_gemm_split_k_short_workspace_runs_unsplit(fp8rl):
    """Less workspace than the query asks for: exactly the unsplit kernel's bits."""
    announce("gemm split-K with a short workspace")
    qa, sa, qw, sw = quantised_operands(100, 256, 2048, 5)
    y_ws, need = run_dense_ws(fp8rl, qa, sa, qw, sw, ws_bytes=1024)
    assert need > 1024
    y = run_dense(fp8rl, qa, sa, qw, sw)
    assert torch.equal(y_ws.view(torch.int16), y.view(torch.int16))


def test_gemm_prefill_full_size_every_element(fp8rl):
    """8192x4096 -> 24576 with outliers: the full GEMM on the GPU against the fp64 oracle
    on every one of its 201M outputs (the oracle runs over row chunks of the same
    codes and scales; rms over the whole output)."""
    announce("gemm prefill 8192x4096x24576, every element")
    a, w = synth.prefill_linear()
    qa, sa = cref.quant_act_token_group128(u16(a))
    qw, sw = cref.quant_weight_block128(u16(w))
    y = run_dense(fp8rl, qa, sa, qw, sw)
    # 1% of the activation channels x50 and 0.1% of the weights x20 put very large and
    # small products into one K group: a few elements carry the instruction's truncation
    check(y, dense_ref_by_rows(qa, sa, qw, sw), "prefill", dense_attribution(qa, sa, qw, sw), budget=32)


def test_gemm_deterministic(fp8rl):
    announce("gemm determinism")
    rng = np.random.default_rng(9)
    m, n, k = 2304, 2304, 512
    qa, qw = to_dev(rand_codes((m, k), rng)), to_dev(rand_codes((n, k), rng))
    sa, sw = to_dev(rand_scales((k // 128, m), rng)), to_dev(rand_scales((n // 128, k // 128), rng))
    y1 = fp8rl.fp8rl_gemm_w8a8_block(qa, sa, qw, sw)
    y2 = fp8rl.fp8rl_gemm_w8a8_block(qa, sa, qw, sw)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def run_grouped(fp8rl, qa, sa, qw, sw, offsets, ldsa_pad=0):
    r = qa.shape[0]
    k = qa.shape[1]
    sa_d = torch.zeros((k // 128, r + ldsa_pad), dtype=torch.float32, device="cuda")
    sa_d[:, :r] = to_dev(sa[:, :r])
    y = fp8rl.fp8rl_grouped_gemm_w8a8_block(to_dev(qa), sa_d, to_dev(qw), to_dev(sw),
                                            to_dev(np.asarray(offsets, np.int32)))
    torch.cuda.synchronize()
    return y


@pytest.mark.parametrize("counts", [
    [3, 0, 130, 2, 0],
    [0, 0, 1],
    [257, 0, 0, 64, 129, 1, 0, 300],
    [5],
])
def test_grouped_small_random(fp8rl, counts):
    announce(f"grouped gemm counts={counts}")
    rng = np.random.default_rng(sum(counts) + len(counts))
    g, n, k = len(counts), 384, 256
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    qa, qw = rand_codes((r, k), rng), rand_codes((g, n, k), rng)
    sa, sw = rand_scales((k // 128, r), rng), rand_scales((g, n // 128, k // 128), rng)
    y = run_grouped(fp8rl, qa, sa, qw, sw, offsets, ldsa_pad=3)
    check(y, gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, offsets), f"grouped {counts}")


def test_grouped_many_experts_matches_dense_per_expert(fp8rl):
    """70 experts (more than one 64-expert scan chunk) vs the dense kernel per expert."""
    announce("grouped gemm 70 experts vs dense")
    rng = np.random.default_rng(70)
    counts = rng.integers(0, 40, size=70)
    counts[[3, 64, 69]] = 0
    g, n, k = 70, 256, 256
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    qa, qw = rand_codes((r, k), rng), rand_codes((g, n, k), rng)
    sa, sw = rand_scales((k // 128, r), rng), rand_scales((g, n // 128, k // 128), rng)
    y = run_grouped(fp8rl, qa, sa, qw, sw, offsets)
    check(y, gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, offsets), "grouped 70")


@pytest.mark.parametrize("k", [128, 384, 1152])
def test_grouped_many_tiles_per_workgroup(fp8rl, k):
    """Over 512 expert tiles (several per persistent workgroup), ragged experts, empty
    experts at both ends, 1, 3 and 9 K blocks per tile (K <= 1024 runs 256x128 tiles,
    K = 1152 the 128x128 ones)."""
    announce(f"grouped gemm persistent k={k}")
    rng = np.random.default_rng(k)
    g, n = 96, 640
    counts = rng.integers(0, 400, size=g)
    counts[[0, 17, 95]] = 0
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    r = int(offsets[-1])
    tiles = int(sum((c + 127) // 128 for c in counts)) * (n // 128)
    assert tiles > 512, tiles
    # realistic operands (bf16 N(0,1) activations, N(0,0.02) weights) quantised by the oracle
    a16 = torch.from_numpy(rng.standard_normal((r, k)).astype(np.float32)).to(torch.bfloat16)
    w16 = torch.from_numpy((rng.standard_normal((g * n, k)) * 0.02).astype(np.float32)).to(torch.bfloat16)
    qa, sa = cref.quant_act_token_group128(u16(a16))
    qw, sw = cref.quant_weight_block128(u16(w16))
    qw, sw = qw.reshape(g, n, k), sw.reshape(g, n // 128, k // 128)
    y = run_grouped(fp8rl, qa, sa, qw, sw, offsets)
    check(y, gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, offsets), f"grouped {g} experts k={k}")


@pytest.mark.parametrize("which", ["gate_up", "down"])
def test_grouped_moe_full_size_every_element(fp8rl, which):
    """Qwen3-30B-A3B-shaped experts, Zipf(1.1) top-8 routing of 4096 tokens (some experts
    empty): every row of every expert against the fp64 oracle."""
    announce(f"grouped gemm MoE {which}, every element")
    moe = synth.moe_layer()
    off = moe["routing"].offsets.numpy()
    x = moe["x_gate_up"] if which == "gate_up" else moe["x_down"]
    wts = moe["w_gate_up"] if which == "gate_up" else moe["w_down"]
    g, n, k = wts.shape
    qa, sa = cref.quant_act_token_group128(u16(x))
    qw, sw = cref.quant_weight_block128(u16(wts.reshape(g * n, k)))
    qw = qw.reshape(g, n, k)
    sw = sw.reshape(g, n // 128, k // 128)
    assert (np.diff(off) == 0).sum() >= 8, "the workload is meant to have empty experts"
    y = run_grouped(fp8rl, qa, sa, qw, sw, off)
    check(y, gemm.grouped_gemm_ref_fp64(qa, sa, qw, sw, off), f"moe {which}",
          grouped_attribution(qa, sa, qw, sw, off), budget=8)


def test_linear_w8a8_end_to_end_tiny(fp8rl):
    """Full forward of the W8A8 linear on the GPU (both quantisers + GEMM) vs the oracle path."""
    announce("linear_w8a8 tiny end to end")
    a, w = synth.tiny_linear(device="cuda")
    qw_d, sw_d = fp8rl.fp8rl_quant_weight_block128(w)
    y = fp8rl.linear_w8a8(a, qw_d, sw_d)
    torch.cuda.synchronize()
    qa, sa = cref.quant_act_token_group128(u16(a))
    qw, sw = cref.quant_weight_block128(u16(w))
    check(y, gemm.gemm_ref_fp64(qa, sa, qw, sw), "linear tiny")
