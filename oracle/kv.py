"""FP8 KV cache with per-step scale recalibration, and decode attention over it
-- oracle, test infrastructure only.

Section 2.3: long-context rollouts are memory-bound, so the KV cache is stored
in FP8; because the policy changes at every RL step, the Q/K/V scales are
recalibrated before each rollout (section 2.3.1, inference-side calibration:
the first forward pass of the step measures them).  In the "KV cache FP8 only"
configuration the attention arithmetic itself stays in higher precision.
Readings taken here (listed with their reasons in the project's design notes):

  * one fp32 scale per layer and tensor (K, V; Q for completeness): the
    calibration pass's largest magnitude / 448 (the weight rule), 1.0 if zero;
  * cache codes = E4M3(fl32(x / s)) rounded to nearest even and saturated at
    +-448 (values beyond the calibrated range clip);
  * paged cache, our layout: key codes [num_blocks][kv_heads][16][head_dim]
    (token-major pages), value codes [num_blocks][kv_heads][4][head_dim][4]
    (token 4a + c of dim d at [a][d][c]: four tokens of a dim adjacent), token
    slot = block * 16 + offset, block_table [batch][max_blocks] int32, seq_lens
    [batch] int32;
  * decode attention for one new query token per sequence with grouped query
    heads (query head h reads kv head h // (q_heads / kv_heads)):
    out = softmax(sm_scale * q . dequant(K)^T) . dequant(V), evaluated in fp64
    here from the bf16 query and the dequantised cache (code value x scale).
"""
import numpy as np

from . import e4m3
from .quant import bf16_bits_to_f32

BLOCK_TOKENS = 16


def calibrate_scale(x_bits: np.ndarray) -> np.float32:
    """Per-tensor scale of a calibration pass: fl32(amax / 448), 1.0 when all zero."""
    amax = np.float32(np.abs(bf16_bits_to_f32(np.asarray(x_bits, dtype=np.uint16))).max(initial=0.0))
    if amax == 0:
        return np.float32(1.0)
    return np.float32(amax / np.float32(e4m3.E4M3_MAX))


def quantize_static(x_bits: np.ndarray, scale) -> np.ndarray:
    """E4M3(fl32(x / s)) with saturation at +-448 (satfinite), s a given fp32 scale."""
    x = bf16_bits_to_f32(np.asarray(x_bits, dtype=np.uint16))
    with np.errstate(over="ignore"):
        quotient = (x / np.float32(scale)).astype(np.float32)
    return e4m3.encode(quotient)                          # encode saturates at 448


def write_cache(k_cache: np.ndarray, v_cache: np.ndarray, k_bits, v_bits, slots, k_scale, v_scale):
    """Quantise new tokens' K and V ([T][kv_heads][head_dim] bf16 bits) into the paged
    caches (keys [num_blocks][kv_heads][16][head_dim], values
    [num_blocks][kv_heads][4][head_dim][4]) at the given token slots."""
    kq = quantize_static(k_bits, k_scale)
    vq = quantize_static(v_bits, v_scale)
    for t, slot in enumerate(np.asarray(slots, dtype=np.int64)):
        b, o = divmod(int(slot), BLOCK_TOKENS)
        k_cache[b, :, o, :] = kq[t]
        v_cache[b, :, o // 4, :, o % 4] = vq[t]


def page_tokens(page: np.ndarray) -> np.ndarray:
    """One block of either cache as [16 tokens][kv_heads][head_dim]."""
    if page.ndim == 3:                                   # keys [kv][16][dim]
        return page.transpose(1, 0, 2)
    kvh, _, dim, _ = page.shape                          # values [kv][4][dim][4]
    return page.transpose(1, 3, 0, 2).reshape(BLOCK_TOKENS, kvh, dim)


def gather_sequence(cache: np.ndarray, block_table_row, seq_len: int) -> np.ndarray:
    """Codes of one sequence's tokens in order: [seq_len][kv_heads][head_dim]."""
    pages = [page_tokens(cache[int(b)]) for b in block_table_row[:(seq_len + BLOCK_TOKENS - 1) // BLOCK_TOKENS]]
    if not pages:
        return np.zeros((0, cache.shape[1], cache.shape[-2] if cache.ndim == 5 else cache.shape[-1]), cache.dtype)
    return np.concatenate(pages, axis=0)[:seq_len]


def attention_decode(q_bits, k_cache, v_cache, k_scale, v_scale, block_table, seq_lens, sm_scale):
    """q [batch][q_heads][head_dim] bf16 bits -> out fp64 [batch][q_heads][head_dim]."""
    q = bf16_bits_to_f32(np.asarray(q_bits, dtype=np.uint16)).astype(np.float64)
    batch, q_heads, dim = q.shape
    kv_heads = k_cache.shape[1]
    group = q_heads // kv_heads
    out = np.zeros((batch, q_heads, dim), np.float64)
    for b in range(batch):
        n = int(seq_lens[b])
        if n == 0:
            continue
        k = e4m3.decode(gather_sequence(k_cache, block_table[b], n)) * float(k_scale)   # [n][kv][dim]
        v = e4m3.decode(gather_sequence(v_cache, block_table[b], n)) * float(v_scale)
        for h in range(q_heads):
            kh = h // group
            s = (k[:, kh, :] @ q[b, h]) * float(sm_scale)
            p = np.exp(s - s.max())
            out[b, h] = (p / p.sum()) @ v[:, kh, :]
    return out
