"""Seeded synthetic inputs shared by the HIP path's tests/bench and by the oracle.

This module only draws random inputs (prompt tokens, forced end-of-sequence
lengths, kernel-sweep data).  It holds none of the method's arithmetic: no
selection, no sampling, no truncation rule, no model math.  Both sides import
it; it imports neither.

Shapes and distributions follow the workload descriptions of the five
configurations (tiny fp32 decoder, kernel sweep, dense-small, a Qwen3-8B-shaped
dense decoder and a Qwen3-30B-A3B-shaped MoE decoder).  The long-tail length
model follows the paper's characterisation of rollout lengths (Sec. 1 and
Sec. 3.2.1: tails 5-10x the median; Sec. 4.3.1: ~5% extreme prompts).
"""
from .configs import CONFIGS, ModelCfg, RunCfg, get_config
from .gen import (rollout_inputs, sweep_attention_inputs, sweep_sampler_logits,
                  sweep_selection_inputs, bf16_bits_from_f32, f32_from_bf16_bits)

__all__ = ["CONFIGS", "ModelCfg", "RunCfg", "get_config", "rollout_inputs",
           "sweep_attention_inputs", "sweep_sampler_logits", "sweep_selection_inputs",
           "bf16_bits_from_f32", "f32_from_bf16_bits"]
