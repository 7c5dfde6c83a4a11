"""Plain, slow CPU oracle of the OLED-MoE block-MoE layer hot path.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check of the build entry point
and the benchmark's CPU-baseline leg may import it; the product path never
does. It shares no code with the HIP library. See oled_oracle for what it
computes and which passages of the paper each function follows.

Parity status: every function is pinned by tests that do not reuse its own
formulas (brute force, closed forms, invariants, high-precision references);
none is "parity unpinned".
"""
from .oled_oracle import (SCORE_SHIFT, SCORE_SCALE, bf16_bits_to_f64, decode, route,
                          permute, classify, silu, expert_ffn, moe_output, score,
                          retain, layer_step, run_schedule)

__all__ = ["SCORE_SHIFT", "SCORE_SCALE", "bf16_bits_to_f64", "decode", "route",
           "permute", "classify", "silu", "expert_ffn", "moe_output", "score",
           "retain", "layer_step", "run_schedule"]
