"""CPU oracle (float64 NumPy) of the decoder forward pass.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; never by the product path.
"""
from .backward import loss_and_grads, rms_norm_backward
from .decoder import (OracleDecoder, apply_rope, causal_gqa_attention, gelu_mlp, gelu_tanh, generate_greedy,
                      greedy, layer_norm, rms_norm, rope_cos_sin, rope_inv_freq, round_to_bf16,
                      round_to_f32, silu, softmax, swiglu_mlp, teacher_forced, weights_f64)

__all__ = ["loss_and_grads", "rms_norm_backward", "OracleDecoder", "apply_rope", "causal_gqa_attention", "gelu_mlp", "gelu_tanh", "generate_greedy",
           "greedy", "layer_norm", "rms_norm", "rope_cos_sin", "rope_inv_freq", "round_to_bf16", "round_to_f32",
           "silu", "softmax", "swiglu_mlp", "teacher_forced", "weights_f64"]
