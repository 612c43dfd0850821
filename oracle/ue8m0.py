"""Power-of-two (UE8M0) scale variant of the blockwise quantisers -- oracle,
test infrastructure only.

Section 2.4.3 ("Scaling Factor: FP32 vs Power-of-2") compares FP32 scaling
factors with power-of-two scales 2^k (UE8M0: an 8-bit biased exponent, no
mantissa) for the same 128x128 weight blocks and 1x128 activation groups.  The
paper does not say how k is derived from the block.  Readings taken here
(listed with their reasons in the project's design notes):

  * k is the smallest integer with amax <= 448 * 2^k: the block maximum lands
    in (224, 448] and nothing saturates; k is clamped below at -127 (the
    smallest UE8M0 value, 2^-127) and an all-zero block gets k = 0;
  * codes = E4M3(x * 2^-k): scaling by a power of two is exact, so E4M3's round
    to nearest even is the only rounding;
  * the scales are returned as fp32 values 2^k, in the same layouts as the
    fp32-scale quantisers ([N/128][K/128] and [K/128][ld_scale]); the byte a
    UE8M0 scale stores is k + 127, the fp32 value's exponent field.

The GEMM with these scales is the ordinary blockwise product (oracle.gemm):
the scales are exact fp32 values.
"""
import numpy as np

from . import e4m3
from .quant import BLOCK, bf16_bits_to_f32

K_MIN = -127


def scale_exponent(amax) -> np.ndarray:
    """Smallest integer k with amax <= 448 * 2^k (clamped at -127; 0 for amax == 0)."""
    a = np.asarray(amax, dtype=np.float64)
    pos = a > 0
    with np.errstate(divide="ignore"):
        k = np.ceil(np.log2(np.where(pos, a, 1.0) / e4m3.E4M3_MAX)).astype(np.int64)
    # log2 is only a first guess: settle k with exact comparisons (448 * 2^k is exact in fp64)
    k = np.where(a > e4m3.E4M3_MAX * np.ldexp(1.0, k), k + 1, k)
    k = np.where(a <= e4m3.E4M3_MAX * np.ldexp(1.0, k - 1), k - 1, k)
    return np.where(pos, np.maximum(k, K_MIN), 0).astype(np.int64)


def quantize_pow2(x: np.ndarray, k) -> np.ndarray:
    """E4M3(x * 2^-k).  x * 2^-k is exact in fp64 and, above 2^-126, in fp32; below
    that E4M3 gives +-0 whatever the fp32 rounding did."""
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    return e4m3.encode(np.ldexp(x, -np.asarray(k)).astype(np.float32))


def quant_weight_block128_ue8m0(w_bits: np.ndarray):
    """bf16 W [N][K] (uint16 bits) -> (codes uint8 [N][K], scales fp32 2^k [N/128][K/128])."""
    w_bits = np.asarray(w_bits, dtype=np.uint16)
    n, k = w_bits.shape
    if n % BLOCK or k % BLOCK:
        raise ValueError("weight dims must be multiples of 128")
    x = bf16_bits_to_f32(w_bits).reshape(n // BLOCK, BLOCK, k // BLOCK, BLOCK)
    amax = np.abs(x).max(axis=(1, 3))                                   # [N/128][K/128]
    e = scale_exponent(amax)
    codes = quantize_pow2(x, e[:, None, :, None]).reshape(n, k)
    return codes, np.ldexp(1.0, e).astype(np.float32)


def quant_act_token_group128_ue8m0(a_bits: np.ndarray, ld_scale: int | None = None):
    """bf16 A [M][K] (uint16 bits) -> (codes uint8 [M][K], scales fp32 2^k [K/128][ld_scale]);
    scale entries of columns m >= M are left 0."""
    a_bits = np.asarray(a_bits, dtype=np.uint16)
    m, k = a_bits.shape
    if k % BLOCK:
        raise ValueError("activation K must be a multiple of 128")
    if ld_scale is None:
        ld_scale = m
    if ld_scale < m:
        raise ValueError("ld_scale must be >= M")
    x = bf16_bits_to_f32(a_bits).reshape(m, k // BLOCK, BLOCK)
    amax = np.abs(x).max(axis=2) if m else np.zeros((0, k // BLOCK), np.float32)   # [M][K/128]
    e = scale_exponent(amax)
    codes = quantize_pow2(x, e[:, :, None]).reshape(m, k)
    scales = np.zeros((k // BLOCK, ld_scale), dtype=np.float32)
    scales[:, :m] = np.ldexp(1.0, e).T
    return codes, scales


def e8m0_byte(scales: np.ndarray) -> np.ndarray:
    """The UE8M0 byte k + 127 of fp32 scales 2^k."""
    _, e = np.frexp(np.asarray(scales, dtype=np.float64))
    return (e - 1 + 127).astype(np.int64)
