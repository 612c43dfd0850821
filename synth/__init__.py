"""Seeded synthetic inputs for the FP8 W8A8 linear-layer workloads.

This module only draws random numbers and lays them out; it performs none of
the quantisation or GEMM arithmetic.  Both the HIP path's tests/bench and the
CPU oracle consume the exact bf16 bytes produced here (copied to the host for
the oracle), so neither side re-derives the inputs.

The shapes and value distributions stand in for the paper's Qwen3-8B-Base and
Qwen3-30B-A3B-Base rollouts (section 2.2.1); no trained weights or evaluation
data are used.

* Qwen3-8B linear shapes: hidden 4096, intermediate 12288, 36 layers,
  q/k/v fused to 6144 outputs (32 query + 8+8 key/value heads of 128).
* Qwen3-30B-A3B expert shapes: hidden 2048, 128 experts of intermediate 768,
  top-8 routing.
"""
from __future__ import annotations

import dataclasses
import math

import torch

BF16_MAX = 3.3895313892515355e38   # largest finite bf16 (0x7F7F)

QWEN3_8B_LINEARS = {            # name: (K in, N out)
    "qkv": (4096, 6144),
    "o_proj": (4096, 4096),
    "gate_up": (4096, 24576),
    "down": (12288, 4096),
}
QWEN3_8B_LAYERS = 36


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def normal_bf16(shape, std: float, seed: int, device="cpu") -> torch.Tensor:
    """~N(0, std^2) drawn in fp32, then rounded to bf16 (RNE)."""
    g = _gen(seed, device)
    x = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(torch.bfloat16)


def bf16_bits(t: torch.Tensor) -> torch.Tensor:
    """Reinterpret a bf16 tensor as its int16 bit patterns (no copy)."""
    return t.view(torch.int16)


def to_numpy_u16(t: torch.Tensor):
    """bf16 tensor -> numpy uint16 array of its bit patterns (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view("uint16")


# --------------------------------------------------------------------------
# tiny blockwise linear: A 64x512 ~N(0,1), W 512x512 ~N(0,0.02)
# --------------------------------------------------------------------------
def tiny_linear(seed: int = 1, device="cpu", m: int = 64, k: int = 512, n: int = 512):
    a = normal_bf16((m, k), 1.0, seed, device)
    w = normal_bf16((n, k), 0.02, seed + 1, device)
    return a, w


# --------------------------------------------------------------------------
# prefill gate_up with outliers: A 8192x4096 ~N(0,1) with 1% of channels x50;
# W 24576x4096 ~N(0,0.02) with 0.1% of entries x20
# --------------------------------------------------------------------------
def prefill_linear(seed: int = 3, device="cpu", m: int = 8192, k: int = 4096, n: int = 24576,
                   outlier_channel_frac: float = 0.01, outlier_channel_gain: float = 50.0,
                   outlier_entry_frac: float = 0.001, outlier_entry_gain: float = 20.0):
    g = _gen(seed, device)
    a = torch.randn(m, k, generator=g, device=device, dtype=torch.float32)
    n_ch = max(1, int(round(outlier_channel_frac * k)))
    ch = torch.randperm(k, generator=g, device=device)[:n_ch]
    a[:, ch] *= outlier_channel_gain
    a = a.to(torch.bfloat16)
    w = torch.randn(n, k, generator=g, device=device, dtype=torch.float32).mul_(0.02)
    n_out = max(1, int(round(outlier_entry_frac * n * k)))
    pos = torch.randint(0, n * k, (n_out,), generator=g, device=device)
    w.view(-1)[pos] *= outlier_entry_gain
    w = w.to(torch.bfloat16)
    return a, w


# --------------------------------------------------------------------------
# decode linears: M tokens through the four Qwen3-8B linears
# --------------------------------------------------------------------------
def decode_activations(seed: int = 2, device="cpu", m: int = 256):
    """{'h': [M][4096], 'inter': [M][12288]} ~N(0,1) bf16."""
    return {
        "h": normal_bf16((m, 4096), 1.0, seed, device),
        "inter": normal_bf16((m, 12288), 1.0, seed + 1, device),
    }


def layer_weights(layer: int, seed: int = 4, device="cpu", names=None):
    """One Qwen3-8B layer's linear weights, [N out][K in] bf16 ~N(0,0.02)."""
    names = names or list(QWEN3_8B_LINEARS)
    out = {}
    for idx, name in enumerate(QWEN3_8B_LINEARS):
        if name not in names:
            continue
        k, n = QWEN3_8B_LINEARS[name]
        out[name] = normal_bf16((n, k), 0.02, seed * 1000003 + layer * 16 + idx, device)
    return out


# --------------------------------------------------------------------------
# weight-resync workload: special blocks planted into a weight matrix
# --------------------------------------------------------------------------
def plant_special_blocks(w: torch.Tensor, seed: int, frac_zero: float = 1 / 256,
                         frac_large: float = 1 / 256):
    """In place: some 128x128 blocks all-zero (a few entries -0), some with huge values.

    Large blocks: the block is multiplied by 1e36 and one entry is set to
    +-bf16-max, so magnitudes reach 3.39e38 without any infinity.
    Returns (zero_blocks, large_blocks) as lists of (i, j) block indices.
    """
    n, k = w.shape
    nb_n, nb_k = n // 128, k // 128
    total = nb_n * nb_k
    g = _gen(seed, "cpu")
    nz = max(1, int(round(frac_zero * total)))
    nl = max(1, int(round(frac_large * total)))
    perm = torch.randperm(total, generator=g)
    zero_ids = perm[:nz].tolist()
    large_ids = perm[nz:nz + nl].tolist()
    for b in zero_ids:
        i, j = divmod(b, nb_k)
        blk = w[i * 128:(i + 1) * 128, j * 128:(j + 1) * 128]
        blk.zero_()
        # a few negative zeros in every zero block
        blk[0, :4] = -0.0
    for b in large_ids:
        i, j = divmod(b, nb_k)
        blk = w[i * 128:(i + 1) * 128, j * 128:(j + 1) * 128]
        big = blk.float().mul_(1e36)
        r, c = divmod(b % (128 * 128), 128)
        big[r, c] = BF16_MAX if (b & 1) else -BF16_MAX
        blk.copy_(big.to(torch.bfloat16))
    return [divmod(b, nb_k) for b in zero_ids], [divmod(b, nb_k) for b in large_ids]


def requant_matrix(layer: int, name: str, seed: int = 5, device="cpu"):
    """One weight matrix of the 36-layer resync workload, with special blocks planted."""
    k, n = QWEN3_8B_LINEARS[name]
    idx = list(QWEN3_8B_LINEARS).index(name)
    s = seed * 1000003 + layer * 16 + idx
    w = normal_bf16((n, k), 0.02, s, device)
    zeros, larges = plant_special_blocks(w, s)
    return w, zeros, larges


# --------------------------------------------------------------------------
# MoE: Qwen3-30B-A3B-shaped experts, Zipf(1.1) routing, some experts empty
# --------------------------------------------------------------------------
@dataclasses.dataclass
class MoERouting:
    token_of_row: torch.Tensor   # int64 [T*topk]: source token for each grouped row
    offsets: torch.Tensor        # int32 [E+1]
    counts: torch.Tensor         # int64 [E]


def moe_routing(seed: int = 6, tokens: int = 4096, experts: int = 128, topk: int = 8,
                zipf_s: float = 1.1, empty_experts: int = 8) -> MoERouting:
    """Zipf(s) expert popularity over a seeded rank order; the `empty_experts`
    least popular ranks get weight 0; each token picks `topk` distinct experts by
    Gumbel-top-k on log-weights.  Rows are grouped by (expert, token)."""
    g = _gen(seed, "cpu")
    ranks = torch.arange(1, experts + 1, dtype=torch.float64)
    weight = ranks.pow(-zipf_s)
    if empty_experts:
        weight[-empty_experts:] = 0.0
    perm = torch.randperm(experts, generator=g)            # rank -> expert id
    w_expert = torch.empty(experts, dtype=torch.float64)
    w_expert[perm] = weight
    logw = torch.where(w_expert > 0, w_expert.log(), torch.full_like(w_expert, -math.inf))
    u = torch.rand(tokens, experts, generator=g, dtype=torch.float64).clamp_(1e-300, 1.0)
    gumbel = -torch.log(-torch.log(u))
    choice = torch.topk(logw[None, :] + gumbel, topk, dim=1).indices   # [T][topk]
    expert_flat = choice.reshape(-1)
    token_flat = torch.arange(tokens).repeat_interleave(topk)
    key = expert_flat * tokens + token_flat
    order = torch.argsort(key)
    expert_sorted = expert_flat[order]
    counts = torch.bincount(expert_sorted, minlength=experts)
    offsets = torch.zeros(experts + 1, dtype=torch.int64)
    offsets[1:] = torch.cumsum(counts, 0)
    return MoERouting(token_of_row=token_flat[order], offsets=offsets.to(torch.int32), counts=counts)


def moe_layer(seed: int = 6, device="cpu", tokens: int = 4096, hidden: int = 2048, experts: int = 128,
              inter: int = 768, topk: int = 8, empty_experts: int = 8):
    """Inputs of one MoE expert block in grouped-row layout.

    Returns dict: routing, x_gate_up [T*topk][hidden] (each token's N(0,1) row
    gathered once per chosen expert), x_down [T*topk][inter] (independent N(0,1),
    standing in for the SiLU*mul output), w_gate_up [E][2*inter][hidden],
    w_down [E][hidden][inter] (~N(0,0.02)).
    """
    routing = moe_routing(seed, tokens, experts, topk, empty_experts=empty_experts)
    x_tok = normal_bf16((tokens, hidden), 1.0, seed + 11, device)
    x_gate_up = x_tok[routing.token_of_row.to(device)]
    x_down = normal_bf16((tokens * topk, inter), 1.0, seed + 12, device)
    w_gate_up = normal_bf16((experts, 2 * inter, hidden), 0.02, seed + 13, device)
    w_down = normal_bf16((experts, hidden, inter), 0.02, seed + 14, device)
    return {"routing": routing, "x_gate_up": x_gate_up, "x_down": x_down,
            "w_gate_up": w_gate_up, "w_down": w_down}


# --------------------------------------------------------------------------
# gated-MLP gate_up outputs (the down projection's input before SiLU * mul)
# --------------------------------------------------------------------------
def gate_up_output(seed: int = 7, device="cpu", m: int = 8192, inter: int = 12288, std_gate: float = 2.0,
                   std_up: float = 1.0, outlier_cols: int = 16, outlier_gain: float = 24.0) -> torch.Tensor:
    """bf16 [m][2*inter] = [gate | up]: gate ~N(0, std_gate^2), up ~N(0, std_up^2),
    `outlier_cols` seeded columns of each half scaled by `outlier_gain` (the
    channel outliers of LLM activations), a few exact zeros per row."""
    g = _gen(seed, device)
    x = torch.randn(m, 2 * inter, generator=g, device=device, dtype=torch.float32)
    x[:, :inter].mul_(std_gate)
    x[:, inter:].mul_(std_up)
    if outlier_cols and m:
        cols = torch.randint(0, inter, (2, outlier_cols), generator=g, device=device)
        x[:, cols[0]] *= outlier_gain
        x[:, inter + cols[1]] *= outlier_gain
    if m:
        zr = torch.randint(0, m, (max(1, m // 8),), generator=g, device=device)
        zc = torch.randint(0, 2 * inter, (max(1, m // 8),), generator=g, device=device)
        x[zr, zc] = 0.0
    return x.to(torch.bfloat16)


def sweep_silu_pairs(device="cpu", exponent: int | None = 127, seed: int = 8, inter: int = 2048) -> torch.Tensor:
    """bf16 gate_up [R][2*inter] covering every (gate bit pattern, up significand)
    pair: element i of the gate half holds bit pattern i mod 2^16, the matching up
    element the sign and 7 mantissa bits i div 2^16 (2^24 pairs in all, R =
    2^24 / inter).  The up exponent is `exponent` (biased, 127: |up| in [1, 2)) or,
    when None, a seeded uniform draw from 1..254 per element."""
    n = 1 << 24
    if n % inter:
        raise ValueError("inter must divide 2^24")
    i = torch.arange(n, dtype=torch.int32, device=device)
    gate = i & 0xFFFF
    sig = i >> 16
    if exponent is None:
        e = torch.randint(1, 255, (n,), generator=_gen(seed, device), device=device, dtype=torch.int32)
    else:
        e = torch.full_like(i, int(exponent))
    up = ((sig >> 7) << 15) | (e << 7) | (sig & 0x7F)
    rows = n // inter
    both = torch.cat([gate.view(rows, inter), up.view(rows, inter)], dim=1)
    bits = torch.where(both >= 0x8000, both - 0x10000, both).to(torch.int16)
    return bits.view(torch.bfloat16)


# --------------------------------------------------------------------------
# exhaustive element-map sweep layouts (bit patterns only)
# --------------------------------------------------------------------------
def _sweep_rows(per: int, device, amax=None) -> torch.Tensor:
    """Rows of `per + 1` bf16 bit patterns: column 0 holds a magnitude a (the row
    maximum), the other columns list every x with |x| <= a, both signs, over as
    many rows as a needs (unused slots are +0).  Every positive finite nonzero a
    appears (or every one of the given patterns), plus one all-zero row mixing +0
    and -0."""
    if amax is None:
        a = torch.arange(1, 0x7F80, dtype=torch.int32, device=device)    # positive finite magnitudes
    else:
        a = torch.as_tensor(amax, dtype=torch.int32).to(device)
    cnt = 2 * (a + 1)                                                    # signed x with |x| <= a
    nb = (cnt + per - 1) // per
    row_a = torch.repeat_interleave(a, nb)
    first = torch.cumsum(nb, 0) - nb
    j = torch.arange(row_a.numel(), dtype=torch.int32, device=device) - torch.repeat_interleave(first, nb)
    i = j[:, None] * per + torch.arange(per, dtype=torch.int32, device=device)[None, :]
    cnt_row = torch.repeat_interleave(cnt, nb)[:, None]
    x = torch.where(i < cnt_row, (i >> 1) | ((i & 1) << 15), torch.zeros_like(i))
    rows = torch.cat([row_a[:, None], x], dim=1)
    zero_row = torch.zeros((1, per + 1), dtype=torch.int32, device=device)
    zero_row[0, 1::2] = 0x8000
    rows = torch.cat([zero_row, rows], dim=0)
    return rows


def sweep_weight_blocks(device="cpu") -> torch.Tensor:
    """bf16 weight [B*128][128] made of 128x128 blocks, each one amax value plus
    16383 x values from the sweep; returned as a bf16 tensor (bit patterns)."""
    rows = _sweep_rows(128 * 128 - 1, device)                           # [B][16384]
    bits = torch.where(rows >= 0x8000, rows - 0x10000, rows).to(torch.int16)
    return bits.view(torch.bfloat16).reshape(-1, 128)


def sweep_act_groups(device="cpu") -> torch.Tensor:
    """bf16 activations [R][128]: each row one amax value plus 127 x values."""
    rows = _sweep_rows(127, device)
    bits = torch.where(rows >= 0x8000, rows - 0x10000, rows).to(torch.int16)
    return bits.view(torch.bfloat16)


def sweep_group_maxima(device="cpu") -> torch.Tensor:
    """bf16 [32640][128]: row r holds the magnitude pattern r (every finite bf16
    magnitude, 0 included) and its negation, zeros elsewhere."""
    a = torch.arange(0, 0x7F80, dtype=torch.int32, device=device)
    rows = torch.zeros((a.numel(), 128), dtype=torch.int32, device=device)
    rows[:, 0] = a
    rows[:, 1] = a | 0x8000
    bits = torch.where(rows >= 0x8000, rows - 0x10000, rows).to(torch.int16)
    return bits.view(torch.bfloat16)


def sweep_binade_groups(device="cpu", mantissas=(0x60,)) -> torch.Tensor:
    """bf16 activations [R][128]: for every exponent field 0..254 and each given
    7-bit mantissa, the magnitude with those bits as the row maximum, followed by
    every x with |x| <= it (127 per row), plus the largest finite bf16 likewise."""
    e = torch.arange(0, 255, dtype=torch.int32)
    m = torch.as_tensor(list(mantissas), dtype=torch.int32)
    amax = ((e[:, None] << 7) | m[None, :]).reshape(-1)
    amax = torch.cat([amax[amax > 0], torch.tensor([0x7F7F], dtype=torch.int32)])
    rows = _sweep_rows(127, device, amax=amax)
    bits = torch.where(rows >= 0x8000, rows - 0x10000, rows).to(torch.int16)
    return bits.view(torch.bfloat16)


# --------------------------------------------------------------------------
# rollout token log-probabilities (TIS weights / mismatch KL)
# --------------------------------------------------------------------------
def rollout_logprobs(seed: int = 9, device="cpu", prompts: int = 32, samples: int = 16, max_len: int = 20480,
                     mismatch_std: float = 0.05):
    """Per-token log-probabilities of a rollout batch laid out [prompts*samples][max_len]
    (flattened): response lengths log-uniform in [256, max_len]; the rollout policy's
    log-probability of each sampled token is -Exp(mean 0.4) (most tokens confident,
    a tail of unlikely ones), the training policy's differs by N(0, mismatch_std^2)
    with 1% of tokens off by N(0, 1).  Returns (logp_train, logp_rollout, mask uint8)."""
    g = _gen(seed, "cpu")
    rows = prompts * samples
    lengths = torch.exp(torch.empty(rows, dtype=torch.float64).uniform_(math.log(256), math.log(max_len), generator=g))
    lengths = lengths.round().clamp(256, max_len).to(torch.int64)
    mask = (torch.arange(max_len)[None, :] < lengths[:, None]).to(torch.uint8).reshape(-1)
    n = rows * max_len
    lr = -torch.empty(n, dtype=torch.float32).exponential_(1.0 / 0.4, generator=g)
    d = torch.randn(n, generator=g, dtype=torch.float32) * mismatch_std
    far = torch.rand(n, generator=g) < 0.01
    d = torch.where(far, torch.randn(n, generator=g, dtype=torch.float32), d)
    lt = (lr + d).clamp(max=0.0)
    return lt.to(device), lr.to(device), mask.to(device)
