"""GPU parity of the FP8 KV cache (section 2.3): per-tensor scale calibration and
the quantised cache write bit for bit, decode attention over the paged cache within
|gpu - ref| <= 4e-3 |ref| + 1e-3 rms(ref) of the fp64 oracle (rms over the call)."""
import numpy as np
import pytest
import torch

import synth
from oracle import e4m3, gemm, kv
from tests.gpu_util import announce, assert_codes_equal, assert_scales_equal, need_gpu, u8, u16, f32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fp8rl():
    need_gpu()
    import paper_2601_18150_amd as m
    m.load()
    return m


def check_close(got: torch.Tensor, ref: np.ndarray, what: str):
    g = got.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    ok, worst, rms = gemm.tolerance_check(g, ref)
    assert ok, f"{what}: worst |err|/bound {worst:.3f} (rms {rms:.3g})"


def bf16(rng, shape, std=1.0):
    return torch.from_numpy((rng.standard_normal(shape) * std).astype(np.float32)).to(torch.bfloat16)


@pytest.mark.parametrize("n", [0, 1, 7, 8, 1000, 123457, 4 << 20])
def test_calibrate_scale(fp8rl, n):
    announce(f"kv calibrate n={n}")
    rng = np.random.default_rng(n)
    x = bf16(rng, (n,), 0.7)
    if n > 10:
        x[n // 3] = -37.5
    s = fp8rl.fp8rl_kv_calibrate_scale(x.cuda())
    torch.cuda.synchronize()
    assert_scales_equal(f32(s), np.array([kv.calibrate_scale(u16(x))], np.float32), "scale")


def test_calibrate_all_zero_gives_one(fp8rl):
    announce("kv calibrate zeros")
    x = torch.zeros(4096, dtype=torch.bfloat16)
    x[::3] = -0.0
    s = fp8rl.fp8rl_kv_calibrate_scale(x.cuda())
    torch.cuda.synchronize()
    assert float(s[0]) == 1.0


def test_cache_write_bit_exact_with_saturation_and_padding(fp8rl):
    announce("kv cache write: permuted slots, padding, out-of-range values")
    rng = np.random.default_rng(3)
    t, kvh, nb = 300, 8, 40
    k = bf16(rng, (t, kvh, 128))
    v = bf16(rng, (t, kvh, 128), 0.5)
    k[5, 2, 7] = 1e4                       # beyond the calibrated range: saturates
    v[9, 0, 0] = -1e4
    slots = rng.permutation(nb * 16)[:t].astype(np.int64)
    slots[[3, 77]] = -1                    # padding tokens
    ks, vs = np.float32(2.5 / 448), np.float32(1.25 / 448)
    kc = torch.full((nb, kvh, 16, 128), 0xCD, dtype=torch.uint8, device="cuda")
    vc = torch.full((nb, kvh, 4, 128, 4), 0xCD, dtype=torch.uint8, device="cuda")
    fp8rl.fp8rl_kv_cache_write_fp8(k.cuda(), v.cuda(), torch.from_numpy(slots).cuda(),
                                   torch.tensor([ks]).cuda(), torch.tensor([vs]).cuda(), kc, vc)
    torch.cuda.synchronize()
    kc_ref = np.full((nb, kvh, 16, 128), 0xCD, np.uint8)
    vc_ref = np.full((nb, kvh, 4, 128, 4), 0xCD, np.uint8)
    keep = slots >= 0
    kv.write_cache(kc_ref, vc_ref, u16(k)[keep], u16(v)[keep], slots[keep], ks, vs)
    assert_codes_equal(u8(kc), kc_ref, "k cache")
    assert_codes_equal(u8(vc), vc_ref, "v cache")


def prefill_slots(rng, nb, runs):
    """Token slots of several prefill runs, each (start offset in its first block, tokens),
    over shuffled blocks; padding (-1), an out-of-range slot and a reversed pair mixed in."""
    blocks = list(rng.permutation(nb))
    out = []
    for start, n in runs:
        need = (start + n + 15) // 16
        own, blocks = blocks[:need], blocks[need:]
        out += [int(own[(start + t) // 16]) * 16 + (start + t) % 16 for t in range(n)]
    out = np.array(out, np.int64)
    return out


@pytest.mark.parametrize("runs", [[(0, 64)], [(0, 37), (5, 29), (0, 16), (12, 9), (3, 1)], [(2, 81), (0, 3)]])
def test_cache_write_prefill_runs_bit_exact(fp8rl, runs):
    """Tokens of whole prefills in order (four tokens to four consecutive slots from a
    multiple of 4: whole value dwords) mixed with runs that start mid-dword, ragged
    ends, padding inside a run, a slot past the cache and a swapped pair."""
    announce(f"kv cache write: prefill runs {runs}")
    rng = np.random.default_rng(len(runs))
    kvh, nb = 4, 24
    slots = prefill_slots(rng, nb, runs)
    t = len(slots)
    if t > 20:
        slots[13] = -1                      # padding inside a run
        slots[18] = nb * 16 + 3             # past the cache: skipped
        slots[[8, 9]] = slots[[9, 8]]       # swapped pair
    k = bf16(rng, (t, kvh, 128))
    v = bf16(rng, (t, kvh, 128), 0.5)
    ks, vs = np.float32(3.0 / 448), np.float32(1.5 / 448)
    kc = torch.full((nb, kvh, 16, 128), 0xCD, dtype=torch.uint8, device="cuda")
    vc = torch.full((nb, kvh, 4, 128, 4), 0xCD, dtype=torch.uint8, device="cuda")
    fp8rl.fp8rl_kv_cache_write_fp8(k.cuda(), v.cuda(), torch.from_numpy(slots).cuda(),
                                   torch.tensor([ks]).cuda(), torch.tensor([vs]).cuda(), kc, vc)
    torch.cuda.synchronize()
    kc_ref = np.full((nb, kvh, 16, 128), 0xCD, np.uint8)
    vc_ref = np.full((nb, kvh, 4, 128, 4), 0xCD, np.uint8)
    keep = (slots >= 0) & (slots < nb * 16)
    kv.write_cache(kc_ref, vc_ref, u16(k)[keep], u16(v)[keep], slots[keep], ks, vs)
    assert_codes_equal(u8(kc), kc_ref, "k cache")
    assert_codes_equal(u8(vc), vc_ref, "v cache")


def paged_inputs(rng, seq_lens, q_heads, kv_heads, spare=5, bf16_cache=False):
    pages = [(int(n) + 15) // 16 for n in seq_lens]
    nb = sum(pages) + spare
    perm = rng.permutation(nb)
    max_blocks = max(max(pages), 1)
    table = np.zeros((len(seq_lens), max_blocks), np.int32)
    off = 0
    for b, p in enumerate(pages):
        table[b, :p] = perm[off:off + p]
        off += p
    if bf16_cache:
        kc = bf16(rng, (nb, kv_heads, 16, 128))
        vc = bf16(rng, (nb, kv_heads, 4, 128, 4))
    else:
        kc = rng.integers(0, 256, (nb, kv_heads, 16, 128)).astype(np.uint8)
        vc = rng.integers(0, 256, (nb, kv_heads, 4, 128, 4)).astype(np.uint8)
        kc[(kc & 0x7F) == 0x7F] ^= 1
        vc[(vc & 0x7F) == 0x7F] ^= 1
        # bytes past each sequence's end in its last block: NaN codes, which the kernel must ignore
        for b, n in enumerate(seq_lens):
            if int(n) % 16:
                blk, first = int(table[b, int(n) // 16]), int(n) % 16
                for t in range(first, 16):
                    kc[blk, :, t, :] = 0x7F
                    vc[blk, :, t // 4, :, t % 4] = 0xFF
    q = bf16(rng, (len(seq_lens), q_heads, 128))
    return q, kc, vc, table, max_blocks


def run_fp8(fp8rl, q, kc, vc, table, seq_lens, ks, vs, sm, max_seq_len=None):
    if max_seq_len is None:
        max_seq_len = int(max(seq_lens)) if len(seq_lens) else 0
    out = fp8rl.fp8rl_attention_decode_fp8kv(q.cuda(), torch.from_numpy(kc).cuda(), torch.from_numpy(vc).cuda(),
                                             torch.from_numpy(table).cuda(),
                                             torch.from_numpy(np.asarray(seq_lens, np.int32)).cuda(), max_seq_len,
                                             torch.tensor([ks]).cuda(), torch.tensor([vs]).cuda(), sm)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("q_heads,kv_heads", [(8, 2), (4, 4), (8, 4), (16, 2)])
def test_attention_fp8kv_ragged_short(fp8rl, q_heads, kv_heads):
    announce(f"attention fp8kv short, {q_heads} q heads / {kv_heads} kv heads")
    rng = np.random.default_rng(q_heads * 10 + kv_heads)
    seq_lens = np.array([1, 15, 16, 17, 70, 0, 255, 256, 257], np.int32)
    q, kc, vc, table, _ = paged_inputs(rng, seq_lens, q_heads, kv_heads)
    ks, vs, sm = np.float32(0.0123), np.float32(0.031), float(1 / np.sqrt(128))
    out = run_fp8(fp8rl, q, kc, vc, table, seq_lens, ks, vs, sm)
    ref = kv.attention_decode(u16(q), kc, vc, ks, vs, table, seq_lens, sm)
    check_close(out, ref, "fp8kv short")
    assert torch.all(out[5] == 0), "an empty sequence gives zeros"


def test_attention_fp8kv_long_sequences_many_splits(fp8rl):
    """Sequences of 1 .. 20480 tokens in one batch (many splits per sequence, merged)."""
    announce("attention fp8kv long, 6 sequences up to 20480 tokens")
    rng = np.random.default_rng(7)
    seq_lens = np.array([20480, 1, 7777, 4096, 12345, 300], np.int32)
    q, kc, vc, table, _ = paged_inputs(rng, seq_lens, 32, 8)
    ks, vs, sm = np.float32(0.01), np.float32(0.02), float(1 / np.sqrt(128))
    out = run_fp8(fp8rl, q, kc, vc, table, seq_lens, ks, vs, sm)
    ref = kv.attention_decode(u16(q), kc, vc, ks, vs, table, seq_lens, sm)
    check_close(out, ref, "fp8kv long")


def test_attention_peaked_scores(fp8rl):
    """Large scores (a sharp softmax) exercise the running-max rescaling across pages
    and splits."""
    announce("attention fp8kv peaked softmax")
    rng = np.random.default_rng(8)
    seq_lens = np.array([5000, 999, 64], np.int32)
    q, kc, vc, table, _ = paged_inputs(rng, seq_lens, 8, 2)
    ks, vs = np.float32(0.05), np.float32(0.02)
    out = run_fp8(fp8rl, q, kc, vc, table, seq_lens, ks, vs, 1.0)
    ref = kv.attention_decode(u16(q), kc, vc, ks, vs, table, seq_lens, 1.0)
    check_close(out, ref, "fp8kv peaked")


def test_attention_bf16kv_matches_exact_attention(fp8rl):
    announce("attention bf16kv")
    rng = np.random.default_rng(9)
    seq_lens = np.array([33, 1000, 2049, 16], np.int32)
    q, kc, vc, table, max_blocks = paged_inputs(rng, seq_lens, 16, 4, bf16_cache=True)
    sm = float(1 / np.sqrt(128))
    out = fp8rl.fp8rl_attention_decode_bf16kv(q.cuda(), kc.cuda(), vc.cuda(), torch.from_numpy(table).cuda(),
                                              torch.from_numpy(seq_lens).cuda(), int(seq_lens.max()), sm)
    torch.cuda.synchronize()
    qf = q.double().numpy()
    kf, vf = kc.double().numpy(), vc.double().numpy()
    ref = np.zeros((len(seq_lens), 16, 128))
    for b, n in enumerate(seq_lens):
        k = kv.gather_sequence(kf, table[b], int(n))
        v = kv.gather_sequence(vf, table[b], int(n))
        for h in range(16):
            s = k[:, h // 4, :] @ qf[b, h] * sm
            p = np.exp(s - s.max())
            ref[b, h] = p @ v[:, h // 4, :] / p.sum()
    check_close(out, ref, "bf16kv")


def test_kv_pipeline_calibrate_write_attend(fp8rl):
    """One layer's step: calibrate K and V scales on a calibration pass, write 4 sequences
    of new tokens into the paged cache, then decode: the whole pipeline on the GPU
    against the same pipeline in the oracle."""
    announce("kv pipeline calibrate + write + attention")
    rng = np.random.default_rng(10)
    kvh, qh = 8, 32
    seq_lens = np.array([700, 64, 1999, 3], np.int32)
    calib_k = bf16(rng, (4096, kvh, 128), 1.3)
    calib_v = bf16(rng, (4096, kvh, 128), 0.8)
    ks = fp8rl.fp8rl_kv_calibrate_scale(calib_k.cuda())
    vs = fp8rl.fp8rl_kv_calibrate_scale(calib_v.cuda())
    pages = [(int(n) + 15) // 16 for n in seq_lens]
    nb = sum(pages) + 2
    perm = rng.permutation(nb)
    table = np.zeros((4, max(pages)), np.int32)
    slots, off = [], 0
    for b, p in enumerate(pages):
        table[b, :p] = perm[off:off + p]
        off += p
        slots += [int(table[b, t // 16]) * 16 + t % 16 for t in range(int(seq_lens[b]))]
    slots = np.array(slots, np.int64)
    k_new = bf16(rng, (len(slots), kvh, 128), 1.3)
    v_new = bf16(rng, (len(slots), kvh, 128), 0.8)
    k_new[0, 0, 0] = 50.0                    # beyond the calibrated range
    kc = torch.zeros((nb, kvh, 16, 128), dtype=torch.uint8, device="cuda")
    vc = torch.zeros((nb, kvh, 4, 128, 4), dtype=torch.uint8, device="cuda")
    fp8rl.fp8rl_kv_cache_write_fp8(k_new.cuda(), v_new.cuda(), torch.from_numpy(slots).cuda(), ks, vs, kc, vc)
    q = bf16(rng, (4, qh, 128))
    sm = float(1 / np.sqrt(128))
    out = fp8rl.fp8rl_attention_decode_fp8kv(q.cuda(), kc, vc, torch.from_numpy(table).cuda(),
                                             torch.from_numpy(seq_lens).cuda(), int(seq_lens.max()), ks, vs, sm)
    torch.cuda.synchronize()
    ks_ref, vs_ref = kv.calibrate_scale(u16(calib_k)), kv.calibrate_scale(u16(calib_v))
    assert_scales_equal(f32(ks), np.array([ks_ref]), "k scale")
    assert_scales_equal(f32(vs), np.array([vs_ref]), "v scale")
    kc_ref = np.zeros((nb, kvh, 16, 128), np.uint8)
    vc_ref = np.zeros((nb, kvh, 4, 128, 4), np.uint8)
    kv.write_cache(kc_ref, vc_ref, u16(k_new), u16(v_new), slots, ks_ref, vs_ref)
    assert_codes_equal(u8(kc), kc_ref, "k cache")
    assert_codes_equal(u8(vc), vc_ref, "v cache")
    ref = kv.attention_decode(u16(q), kc_ref, vc_ref, ks_ref, vs_ref, table, seq_lens, sm)
    check_close(out, ref, "pipeline")
