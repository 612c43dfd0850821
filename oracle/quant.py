"""Blockwise / groupwise FP8 quantisation -- oracle, test infrastructure only.

Section 2.1.1, Eq. (1): each code is the FP8 rounding of the element divided by
its block's scale, and the scale comes from the block's largest magnitude
(readings below).  Weights use 128x128 blocks; activations use 1x128 groups per
token, computed dynamically at every forward pass (section 2.1.1 "Static vs
dynamic quantization"; section 3.1 names the 1x128 / 128x128 tiling).  Scales
are fp32 (section 2.4.3 adopts FP32 scaling factors as the default).

Readings of what the paper leaves open (each one is listed with its reason in
the project's design notes):
  * scale = fl32(amax / 448): the block's largest magnitude maps onto the
    largest finite E4M3 value;
  * the quotient x / scale is one IEEE fp32 division (round to nearest even,
    subnormals kept), then rounded once to E4M3 by ``e4m3.encode``;
  * an all-zero block or group gets scale = 1.0 and codes +-0 by input sign;
  * weights are stored [N out][K in] (K contiguous); block (i, j) covers rows
    128i..128i+127 and columns 128j..128j+127; scales are [N/128][K/128];
  * activation scales are stored [K/128][ld_scale] (token index contiguous).

Inputs are bf16 given as uint16 bit patterns; bf16 -> fp32 is exact
(the 16 bits become the high half of the fp32 word).
"""
import numpy as np

from . import e4m3

BLOCK = 128


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact bf16 -> fp32 widening of uint16 bit patterns."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def _scale_from_amax(amax: np.ndarray) -> np.ndarray:
    """fp32 scale per block: amax / 448 in IEEE fp32, 1.0 for all-zero blocks."""
    amax = np.asarray(amax, dtype=np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        s = (amax / np.float32(e4m3.E4M3_MAX)).astype(np.float32)
    return np.where(amax == np.float32(0.0), np.float32(1.0), s).astype(np.float32)


def quantize_with_scale(x: np.ndarray, s) -> np.ndarray:
    """Eq. (1) for one element set sharing scale(s) s: codes = E4M3(fl32(x / s))."""
    x = np.asarray(x, dtype=np.float32)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore", under="ignore"):
        quotient = (x / np.asarray(s, dtype=np.float32)).astype(np.float32)
    return e4m3.encode(quotient)


def quant_weight_block128(w_bits: np.ndarray):
    """bf16 W [N][K] (uint16 bits) -> (codes uint8 [N][K], scales fp32 [N/128][K/128]).

    One block at a time, as Eq. (1) states it: find the block's largest
    magnitude, derive the scale, divide every element by it, round to E4M3.
    """
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    n, k = w_bits.shape
    if n % BLOCK or k % BLOCK:
        raise ValueError("weight dims must be multiples of 128")
    x = bf16_bits_to_f32(w_bits)
    codes = np.empty((n, k), dtype=np.uint8)
    scales = np.empty((n // BLOCK, k // BLOCK), dtype=np.float32)
    for i in range(n // BLOCK):
        for j in range(k // BLOCK):
            blk = x[i * BLOCK:(i + 1) * BLOCK, j * BLOCK:(j + 1) * BLOCK]
            amax = np.max(np.abs(blk))
            s = _scale_from_amax(amax)
            scales[i, j] = s
            codes[i * BLOCK:(i + 1) * BLOCK, j * BLOCK:(j + 1) * BLOCK] = quantize_with_scale(blk, s)
    return codes, scales


def quant_act_token_group128(a_bits: np.ndarray, ld_scale: int | None = None):
    """bf16 A [M][K] (uint16 bits) -> (codes uint8 [M][K], scales fp32 [K/128][ld_scale]).

    Each token (row) is cut into 1x128 groups along K; each group gets its own
    scale from its largest magnitude, then every element is divided and rounded.
    Scale entries in columns m >= M (padding up to ld_scale) are left as 0.
    """
    a_bits = np.asarray(a_bits, dtype=np.uint16)
    m, k = a_bits.shape
    if k % BLOCK:
        raise ValueError("activation K must be a multiple of 128")
    if ld_scale is None:
        ld_scale = m
    if ld_scale < m:
        raise ValueError("ld_scale must be >= M")
    x = bf16_bits_to_f32(a_bits)
    codes = np.empty((m, k), dtype=np.uint8)
    scales = np.zeros((k // BLOCK, ld_scale), dtype=np.float32)
    for g in range(k // BLOCK):
        grp = x[:, g * BLOCK:(g + 1) * BLOCK]                 # [M][128]
        amax = np.max(np.abs(grp), axis=1) if m else np.zeros(0, np.float32)
        s = _scale_from_amax(amax)                            # [M]
        scales[g, :m] = s
        codes[:, g * BLOCK:(g + 1) * BLOCK] = quantize_with_scale(grp, s[:, None])
    return codes, scales
