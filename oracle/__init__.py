"""fp64 CPU oracle for the phase-split decoder forward pass.

TEST INFRASTRUCTURE: only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import it.  The product path never routes through it.

Parity status of each function (pins live in tests/test_oracle_pins.py):
  rmsnorm, rope_frequencies, apply_rope, softmax, causal_gqa_attention, silu/swiglu,
  argmax_lowest, top2_margin, OracleModel (prefill, decode, forward_full) -- all pinned.
  mamba: softplus, causal_depthwise_conv, selective_scan, OracleMamba (prefill, decode,
  forward_full) -- all pinned (tests/test_mamba_oracle_pins.py).
  mamba2: ssd_scan, OracleMamba2 (prefill, extend, decode, forward_full) -- all pinned
  (tests/test_mamba2_oracle_pins.py).
  rglru: gelu_tanh, sigmoid, rms_norm_offset, soft_cap, block_diag_apply, rg_lru, OracleRG
  (prefill, extend, decode, forward_full) -- all pinned (tests/test_rglru_oracle_pins.py).
"""
from .transformer import (  # noqa: F401
    OracleModel, apply_rope, argmax_lowest, causal_gqa_attention, rmsnorm, rope_frequencies,
    silu, softmax, split_prompts, swiglu, teacher_forced_run, top2_margin,
)
