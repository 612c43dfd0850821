"""CPU oracle for the blockwise FP8 W8A8 linear layer -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct restatement of what the paper
("FP8-RL", arXiv 2601.18150) computes on its FP8 linear-layer hot path:

* ``e4m3``  -- the OCP E4M3 ("fn") codec, from the format definition
  (section 2.1.1: 4 exponent bits, 3 mantissa bits, range about +-448;
  section 3.1 / ref. [12] for the encoding family).
* ``quant`` -- blockwise weight quantisation with one fp32 scale per
  128x128 block (section 2.1.1, Eq. (1)) and dynamic per-token activation
  quantisation with one fp32 scale per 1x128 group (section 2.1.1 "Static vs
  dynamic quantization", section 3.1 "1x128 tiles for activations").
* ``gemm``  -- the blockwise-scaled FP8 GEMM, dense and grouped by expert
  (section 2.1.4 / section 2.1.1 quantisation scope incl. MoE fc1/fc2),
  evaluated as dequantise-then-matmul in fp64.
* ``act``   -- the down projection's input: SiLU(gate) * up rounded to bf16,
  then 1x128 group quantisation (section 2.1.1: down_proj / fc2 are quantised
  like every linear, activations dynamically), and the row gather of quantised
  activations that MoE dispatch needs.
* ``ue8m0`` -- the power-of-two (UE8M0) scale variant of both quantisers
  (section 2.4.3 "Scaling Factor: FP32 vs Power-of-2").
* ``tis``   -- token-level truncated importance-sampling weights (section
  2.1.3, Eq. (2)-(3)) and the mismatch-KL sums over the sampled tokens.
* ``kv``    -- the FP8 KV cache with per-step scale calibration and decode
  attention over the paged cache (section 2.3).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call or execute anything in this package.  The HIP
product path never does; it shares no code, table or constant generator with
this package.  Everything here is numpy on the CPU, plus one small C file,
``quant_ref.c`` (loaded through ``cref``), a restatement of the quantisers that
the full-size and exhaustive element-map tests use for speed.
"""
from . import e4m3, quant, gemm, act, ue8m0, tis, kv  # noqa: F401
