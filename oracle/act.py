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
  * h = SiLU(gate) * up, SiLU(g) = g / (1 + exp(-g)), evaluated exactly (fp64
    here) and rounded once to bf16 (round to nearest even) -- the bf16 tensor
    an unfused pipeline would store between the two steps;
  * h is then quantised per token and 1x128 group exactly like any other
    activation (quant.quant_act_token_group128).

MoE dispatch copies each token's activation row to the rows of its experts.
Quantising per row commutes with that copy, so the rows can be quantised once
per token and the codes and scales gathered (gather_rows_fp8).
"""
import numpy as np

from . import quant

BLOCK = 128


def f64_to_bf16_bits(x) -> np.ndarray:
    """Round fp64 values to bf16 (8 significant bits, round to nearest even,
    subnormals kept, overflow to +-inf), once, straight from fp64."""
    x = np.asarray(x, dtype=np.float64)
    sign = np.where(np.signbit(x), 0x8000, 0).astype(np.uint32)
    a = np.abs(x)
    _, e = np.frexp(a)                                   # a = m * 2^e, m in [0.5, 1)
    q = np.maximum(e - 1, -126) - 7                      # spacing of the bf16 values near a
    n = np.rint(np.ldexp(a, -q))                         # exact scaling, then ties-to-even
    r = np.ldexp(n, q)                                   # representable, or >= 2^128 on overflow
    with np.errstate(over="ignore"):
        bits = (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint32)   # exact: <= 8 significant bits
    bits = np.where(r >= 2.0 ** 128, 0x7F80, bits)
    bits = np.where(a == 0.0, 0, bits)
    bits = np.where(np.isnan(x), 0x7FC0, bits | sign)
    return bits.astype(np.uint16)


def silu_mul_bf16(gu_bits: np.ndarray, inter: int) -> np.ndarray:
    """[M][2I] bf16 gate_up (uint16 bits) -> h = bf16(SiLU(gate) * up) [M][I] (uint16 bits)."""
    gu = quant.bf16_bits_to_f32(np.asarray(gu_bits, dtype=np.uint16)).astype(np.float64)
    if gu.shape[1] != 2 * inter:
        raise ValueError("gate_up must have 2 * inter columns")
    g, u = gu[:, :inter], gu[:, inter:]
    with np.errstate(over="ignore"):
        silu = g / (1.0 + np.exp(-g))
    return f64_to_bf16_bits(silu * u)


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
