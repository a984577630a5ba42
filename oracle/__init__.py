"""CPU oracle for batched VLA rollout inference -- test infrastructure only.

Imported by the test-suite, the smoke check and the benchmark's CPU-baseline
leg; never by the library.  See ``vla_oracle`` for what it computes, and
``learn_oracle`` for the learning-phase arithmetic (GAE, PPO-clip, log-prob
gradient).
"""
from . import learn_oracle  # noqa: F401
from .vla_oracle import (MODES, Weights, action_logits, apply_rope, as_weights, bf16_round,  # noqa: F401
                         causal_attention, decoder_layer, extract_actions, forward_rows, lora_merge, merge_weights,
                         prefill_logits,
                         prefix_embeddings, rms_norm, rollout, rollout_env, rope_angles,
                         sample_bin, silu, teacher_forced, teacher_forced_env, to_f64,
                         token_stats, values)
