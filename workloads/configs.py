"""Model shapes and workload recipes for the draft-and-verify step.

The paper (CacheSpec, Section 4.1 and the small-model choice appendix) pairs a
large target decoder (Qwen3-32B, Llama-3.3-70B) with a small drafter
(Qwen3-1.7B, Llama-3.2-1B/3B) but states no kernel-level shapes, precision or
hardware, and ships no weights here.  The workloads below are synthetic,
random-initialised stand-ins with Llama-style architecture (RMSNorm, rotary
position embedding, SwiGLU MLP, grouped-query attention, untied LM head, no
biases):

* ``TINY_FP32``      2-layer d=256 target / 1-layer drafter, vocab 1024, fp32.
* ``SMALL_BF16``     12-layer d=1024 target / 2-layer d=512 drafter, vocab 32000.
* ``LLAMA8B_SHAPED`` 32-layer d=4096 (32 q / 8 kv heads) target with a
                     16-layer d=2048 drafter, vocab 128256, batch 1.
* ``SERVING_8B``     the same pair serving 64 sequences from a paged cache.
* ``VOCAB_STRESS``   the acceptance / resample pass alone, 256 x 8 rows x 128256.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class ModelShape:
    """Shape of one Llama-style decoder."""

    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rope_theta: float
    rms_eps: float = 1e-5
    dtype: str = "bf16"          # "f32" or "bf16": weights, KV cache, GEMM inputs
    init_std: float = 0.02

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim

    def layer_params(self) -> int:
        d = self.d_model
        return (self.qkv_rows * d + d * self.q_dim + 2 * self.ffn_dim * d
                + d * self.ffn_dim + 2 * d)

    def total_params(self) -> int:
        return (self.n_layers * self.layer_params() + 2 * self.vocab * self.d_model
                + self.d_model)

    def bytes_per_elem(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def weight_bytes_per_forward(self) -> int:
        """Bytes of weights one forward pass with an LM head streams from HBM
        (every layer matrix and the LM head once; embedding rows and norm
        vectors are negligible)."""
        d = self.d_model
        per_layer = (self.qkv_rows * d + d * self.q_dim + 2 * self.ffn_dim * d
                     + d * self.ffn_dim)
        return (self.n_layers * per_layer + self.vocab * d) * self.bytes_per_elem()

    def kv_bytes_per_token(self) -> int:
        return self.n_layers * 2 * self.kv_dim * self.bytes_per_elem()


@dataclass(frozen=True)
class PairConfig:
    """A target/draft pair and the serving recipe around it."""

    name: str
    target: ModelShape
    draft: ModelShape
    batch: int
    # prompt / context recipe: ("fixed", P) | ("uniform", lo, hi) | ("loguniform", lo, hi)
    context: Tuple
    k: Tuple[int, ...]            # draft length choices (one per sequence, seeded)
    temperatures: Tuple[float, ...]
    steps: int
    seed: int = 1234
    page_size: int = 16
    # draft mixing (workload shaping for random-init pairs): the fraction of
    # drafts guided to the target's top-1 token, and the logit boost
    mix_rate: float = 0.0
    mix_boost: float = 2.0


@dataclass(frozen=True)
class VocabPassConfig:
    name: str
    batch: int
    k: int
    vocab: int
    temperatures: Tuple[float, ...]
    p_std: float = 3.0
    q_noise_std: float = 1.0
    base_pos_range: Tuple[int, int] = (512, 4096)
    seed: int = 1234


TINY_TARGET = ModelShape("tiny-target", 2, 256, 4, 4, 64, 688, 1024, 1e4, dtype="f32")
TINY_DRAFT = ModelShape("tiny-draft", 1, 256, 4, 4, 64, 688, 1024, 1e4, dtype="f32")
SMALL_TARGET = ModelShape("small-target", 12, 1024, 16, 16, 64, 2816, 32000, 1e4)
SMALL_DRAFT = ModelShape("small-draft", 2, 512, 8, 8, 64, 1408, 32000, 1e4)
L8B_TARGET = ModelShape("8b-shaped-target", 32, 4096, 32, 8, 128, 14336, 128256, 5e5)
L1B_DRAFT = ModelShape("1b-shaped-draft", 16, 2048, 32, 8, 64, 8192, 128256, 5e5)

TINY_FP32 = PairConfig("tiny-fp32", TINY_TARGET, TINY_DRAFT, batch=1,
                       context=("fixed", 128), k=(4,), temperatures=(1.0, 0.0),
                       steps=32)
SMALL_BF16 = PairConfig("small-bf16", SMALL_TARGET, SMALL_DRAFT, batch=8,
                        context=("uniform", 256, 512), k=(5,),
                        temperatures=(0.7,), steps=64)
LLAMA8B_SHAPED = PairConfig("8b-shaped", L8B_TARGET, L1B_DRAFT, batch=1,
                            context=("fixed", 2048), k=(5,),
                            temperatures=(0.0, 0.8), steps=64)
SERVING_8B = PairConfig("8b-serving", L8B_TARGET, L1B_DRAFT, batch=64,
                        context=("loguniform", 512, 4096), k=(3, 5, 7),
                        temperatures=(0.8,), steps=256, mix_rate=0.7, mix_boost=2.0)
VOCAB_STRESS = VocabPassConfig("vocab-stress", batch=256, k=7, vocab=128256,
                               temperatures=(0.3, 1.0, 1.5))

CONFIGS = {c.name: c for c in (TINY_FP32, SMALL_BF16, LLAMA8B_SHAPED,
                               SERVING_8B, VOCAB_STRESS)}
