"""Down-projection input of the gated MLP, and row gathers of quantised
activations -- oracle, test infrastructure only.

The paper quantises every MLP and MoE expert linear, down_proj / fc2 included
(section 2.1.1 "Quantization scope"), and quantises activations dynamically at
every forward pass with 1x128 groups (section 2.1.1 "Static vs dynamic
quantization"; section 3.1).  The down projection's input is the gated MLP's
hidden state; for the Qwen3 models the paper runs this is SiLU(gate) * up of
the fused gate_up output.  The paper does not spell the activation out; the
readings taken here (listed with their reasons in the project's design notes):

  * gate_up output rows are [gate | up]: columns 0 .. I-1 gate, I .. 2I-1 up;
  * h = SiLU(gate) * up, SiLU(g) = g / (1 + exp(-g)), rounded once to bf16
    (round to nearest even) from its exact value -- the bf16 tensor an
    unfused pipeline would store between the two steps.  The exact value is
    never a bf16 rounding tie for g != 0 (it is transcendental), but in two
    limits it lies closer to an exactly representable product than fp64 can
    resolve, so the side of the tie is taken from the sign of the deviation:
      - |g| <= 2^-20: SiLU(g) u = (g u / 2)(1 + tanh(g / 2)), within 2^-21
        (relative) of the exact 16-bit product g u / 2; at a tie, away from
        zero for g > 0 and toward zero for g < 0;
      - g >= 16: SiLU(g) u = g u (1 - 1 / (1 + e^g)), within e^-16 < 2^-23 of
        g u; at a tie, toward zero;
    everywhere else the fp64 evaluation decides (a pin checks, over every
    gate bit pattern and up significand, that it never lands within 2^-48 of
    a bf16 rounding boundary, far beyond its own error);
  * h is then quantised per token and 1x128 group exactly like any other
    activation (quant.quant_act_token_group128).

MoE dispatch copies each token's activation row to the rows of its experts.
Quantising per row commutes with that copy, so the rows can be quantised once
per token and the codes and scales gathered (gather_rows_fp8).
"""
import numpy as np

from . import quant

BLOCK = 128


SMALL_G = 2.0 ** -20      # at or below |g|: the g u / 2 limit
LARGE_G = 16.0            # at or above g: the g u limit


def f64_to_bf16_bits(x, tie=0) -> np.ndarray:
    """Round fp64 values to bf16 (8 significant bits, subnormals kept, overflow
    to +-inf), once, straight from fp64.  Round to nearest; an exact tie goes to
    the even significand (tie == 0), away from zero (tie > 0) or toward zero
    (tie < 0); `tie` broadcasts against x.  NaN gives 0x7FC0."""
    x = np.asarray(x, dtype=np.float64)
    tie = np.broadcast_to(np.asarray(tie), x.shape)
    with np.errstate(over="ignore", invalid="ignore"):
        return _f64_to_bf16_bits(x, tie)


def _f64_to_bf16_bits(x: np.ndarray, tie: np.ndarray) -> np.ndarray:
    sign = np.where(np.signbit(x), 0x8000, 0).astype(np.uint32)
    a = np.abs(x)
    _, e = np.frexp(a)                                   # a = m * 2^e, m in [0.5, 1)
    q = np.maximum(e - 1, -126) - 7                      # spacing of the bf16 values near a
    t = np.ldexp(a, -q)                                  # exact scaling
    lo = np.floor(t)
    frac = t - lo
    even = np.rint(t)                                    # ties to even
    n = np.where(frac == 0.5, np.where(tie > 0, lo + 1, np.where(tie < 0, lo, even)), even)
    r = np.ldexp(n, q)                                   # representable, or >= 2^128 on overflow
    bits = (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint32)   # exact: <= 8 significant bits
    bits = np.where(r >= 2.0 ** 128, 0x7F80, bits)
    bits = np.where(a == 0.0, 0, bits)
    bits = np.where(np.isnan(x), 0x7FC0, bits | sign)
    return bits.astype(np.uint16)


def silu_mul_bf16(gu_bits: np.ndarray, inter: int) -> np.ndarray:
    """[M][2I] bf16 gate_up (uint16 bits) -> h = bf16(SiLU(gate) * up) [M][I] (uint16 bits)."""
    with np.errstate(over="ignore", invalid="ignore"):         # inf / NaN inputs propagate as IEEE says
        gu = quant.bf16_bits_to_f32(np.asarray(gu_bits, dtype=np.uint16)).astype(np.float64)
        if gu.shape[1] != 2 * inter:
            raise ValueError("gate_up must have 2 * inter columns")
        g, u = gu[:, :inter], gu[:, inter:]
        x = g / (1.0 + np.exp(-g)) * u
        small = np.abs(g) <= SMALL_G
        large = g >= LARGE_G
        x = np.where(small, g * u / 2.0, np.where(large, g * u, x))     # exact products in the two limits
        tie = np.where(small, np.sign(g), np.where(large, -1.0, 0.0))
        return f64_to_bf16_bits(x, tie)


def silu_mul_quant_group128(gu_bits: np.ndarray, inter: int, ld_scale: int | None = None):
    """The fused step: h = bf16(SiLU(gate) * up), then 1x128 group quantisation of h.
    Returns (h bits [M][I], codes [M][I], scales [I/128][ld_scale])."""
    h = silu_mul_bf16(gu_bits, inter)
    codes, scales = quant.quant_act_token_group128(h, ld_scale)
    return h, codes, scales


def gather_rows_fp8(codes: np.ndarray, scales: np.ndarray, index: np.ndarray):
    """Rows index[r] of quantised activations: codes [R][K], scales [K/128][R]."""
    index = np.asarray(index, dtype=np.int64)
    return codes[index], scales[:, index]
