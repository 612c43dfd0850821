"""Pins of oracle/kv.py (FP8 KV cache, per-step scale calibration, decode attention
over the paged cache) against torch's attention and closed forms."""
import numpy as np
import torch

from oracle import e4m3, kv


def bf16_bits(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def random_paged(rng, batch, kv_heads, dim, seq_lens, spare=3):
    pages = [(n + 15) // 16 for n in seq_lens]
    num_blocks = sum(pages) + spare
    perm = rng.permutation(num_blocks)
    table = np.full((batch, max(max(pages), 1) + 2), -1, np.int32)
    k = 0
    for b, p in enumerate(pages):
        table[b, :p] = perm[k:k + p]
        k += p
    codes = lambda shape: (lambda c: np.where((c & 0x7F) == 0x7F, c ^ 1, c))(
        rng.integers(0, 256, shape).astype(np.uint8))
    return codes((num_blocks, kv_heads, 16, dim)), codes((num_blocks, kv_heads, 4, dim, 4)), table


def test_decode_attention_matches_torch_sdpa_with_grouped_heads():
    """Random codes, per-tensor scales, ragged lengths, shuffled pages: the oracle equals
    torch's scaled_dot_product_attention (fp64, grouped query heads) on the
    dequantised, gathered keys and values."""
    rng = np.random.default_rng(1)
    batch, q_heads, kv_heads, dim = 5, 8, 2, 128
    seq_lens = np.array([1, 15, 16, 17, 70], np.int32)
    kc, vc, table = random_paged(rng, batch, kv_heads, dim, seq_lens)
    q = bf16_bits(rng.standard_normal((batch, q_heads, dim)))
    ks, vs, sm = np.float32(0.0123), np.float32(0.031), 1.0 / np.sqrt(dim)
    got = kv.attention_decode(q, kc, vc, ks, vs, table, seq_lens, sm)
    qf = torch.from_numpy(q.view(np.int16)).view(torch.bfloat16).double()
    for b in range(batch):
        n = int(seq_lens[b])
        k = torch.from_numpy(e4m3.decode(kv.gather_sequence(kc, table[b], n)) * float(ks)).permute(1, 0, 2)
        v = torch.from_numpy(e4m3.decode(kv.gather_sequence(vc, table[b], n)) * float(vs)).permute(1, 0, 2)
        ref = torch.nn.functional.scaled_dot_product_attention(qf[b][:, None, :], k, v, scale=sm, enable_gqa=True)
        assert np.allclose(got[b], ref[:, 0, :].numpy(), rtol=1e-12, atol=1e-14)


def test_decode_attention_closed_forms():
    """Identical keys: the output is the mean of the values.  One key far better aligned
    with the query: the output is that token's value row."""
    batch, q_heads, kv_heads, dim = 2, 4, 1, 128
    kc = np.full((4, kv_heads, 16, dim), 0x38, np.uint8)          # every key = 1.0 * scale
    rng = np.random.default_rng(2)
    vc = rng.integers(0, 0x7E, (4, kv_heads, 4, dim, 4)).astype(np.uint8)
    table = np.array([[0, 1, 2, 3], [3, 2, 1, 0]], np.int32)
    seq_lens = np.array([50, 64], np.int32)
    q = bf16_bits(rng.standard_normal((batch, q_heads, dim)))
    out = kv.attention_decode(q, kc, vc, 1.0, 0.5, table, seq_lens, 0.1)
    for b in range(batch):
        v = e4m3.decode(kv.gather_sequence(vc, table[b], int(seq_lens[b]))) * 0.5
        for h in range(q_heads):
            assert np.allclose(out[b, h], v[:, 0, :].mean(axis=0), rtol=1e-12, atol=1e-12)
    kc2 = np.zeros_like(kc)
    kc2[2, 0, 5, :] = 0x70                                        # token 2*16+5 of sequence 0 (one key of 256)
    q2 = bf16_bits(np.ones((1, q_heads, dim)))
    out2 = kv.attention_decode(q2, kc2, vc, 1.0, 0.5, table[:1], seq_lens[:1], 1.0)
    v0 = e4m3.decode(vc[2, 0, 1, :, 1]) * 0.5                      # token 5 of the block: [5 // 4][:][5 % 4]
    assert np.allclose(out2[0, 0], v0, rtol=0, atol=1e-12)


def test_static_quantisation_is_the_library_cast_with_saturation():
    rng = np.random.default_rng(3)
    x = rng.standard_normal(50000).astype(np.float32) * 3
    x[:10] = [1000.0, -1000.0, 448.0, -449.0, 0.0, -0.0, 3e-30, 5.0, -5.0, 1e30]
    bits = bf16_bits(x)
    s = np.float32(0.0125)
    codes = kv.quantize_static(bits, s)
    xv = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float()
    quot = (xv / torch.tensor(s)).numpy()
    inside = np.abs(quot) < 448
    want = torch.from_numpy(quot[inside]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes[inside], want)
    assert np.all(codes[~inside] & 0x7F == 0x7E) and np.array_equal(codes[~inside] >> 7, (quot[~inside] < 0).astype(np.uint8))


def test_calibrated_scale_maps_the_maximum_to_448():
    rng = np.random.default_rng(4)
    x = bf16_bits(rng.standard_normal((64, 1024)) * 0.7)
    s = kv.calibrate_scale(x)
    codes = kv.quantize_static(x, s)
    xv = np.abs(torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).float().numpy())
    assert np.all(codes.reshape(-1)[xv.reshape(-1) == xv.max()] & 0x7F == 0x7E)
    assert np.all(codes & 0x7F != 0x7F)
    assert kv.calibrate_scale(np.zeros(8, np.uint16)) == 1.0


def test_value_page_layout_puts_four_tokens_of_a_dim_together():
    page = np.arange(2 * 16 * 128, dtype=np.int64).reshape(2, 4, 128, 4)    # [kv][4][dim][4]
    tok = kv.page_tokens(page)
    assert tok.shape == (16, 2, 128)
    assert tok[5, 1, 7] == page[1, 1, 7, 1] and tok[12, 0, 127] == page[0, 3, 127, 0]


def test_cache_write_then_gather_round_trips_tokens_in_order():
    rng = np.random.default_rng(5)
    kv_heads, dim = 3, 128
    kc = np.zeros((6, kv_heads, 16, dim), np.uint8)
    vc = np.zeros((6, kv_heads, 4, dim, 4), np.uint8)
    table = np.array([4, 1, 5], np.int32)
    n = 40
    slots = np.array([table[t // 16] * 16 + t % 16 for t in range(n)])
    k = bf16_bits(rng.standard_normal((n, kv_heads, dim)))
    v = bf16_bits(rng.standard_normal((n, kv_heads, dim)))
    kv.write_cache(kc, vc, k, v, slots, 0.01, 0.02)
    assert np.array_equal(kv.gather_sequence(kc, table, n), kv.quantize_static(k, 0.01))
    assert np.array_equal(kv.gather_sequence(vc, table, n), kv.quantize_static(v, 0.02))
