"""Seeded synthetic inputs shared by the CPU oracle, the tests and the bench.

This package holds shapes and random draws only: model shapes, weight and
prompt generators, and the synthetic logits of the vocab-pass workload.  It
contains none of the method's arithmetic (no forward pass, no softmax, no
sampling rule), so that the oracle and the HIP path can both consume it
without sharing any computation.
"""

from .configs import (ModelShape, PairConfig, VocabPassConfig, CONFIGS,
                      TINY_FP32, SMALL_BF16, LLAMA8B_SHAPED, SERVING_8B,
                      VOCAB_STRESS)
from .gen import (bf16_round_u16, bf16_u16_to_f32, model_weights,
                  layer_weights, uniform_prompts, prompt_lengths_uniform,
                  context_lengths_loguniform, draft_lengths, vocab_logits,
                  vocab_temperatures, base_positions, seq_ids_for, mix_draws)

__all__ = [
    "ModelShape", "PairConfig", "VocabPassConfig", "CONFIGS", "TINY_FP32",
    "SMALL_BF16", "LLAMA8B_SHAPED", "SERVING_8B", "VOCAB_STRESS",
    "bf16_round_u16", "bf16_u16_to_f32", "model_weights", "layer_weights",
    "uniform_prompts", "prompt_lengths_uniform", "context_lengths_loguniform",
    "draft_lengths", "vocab_logits", "vocab_temperatures", "base_positions",
    "seq_ids_for", "mix_draws",
]
