"""Seeded generators for the synthetic workloads.

Every draw comes from a NumPy PCG64 stream keyed by ``(seed, tag, indices...)``
so that any single tensor, prompt or logit row can be regenerated on its own
(the oracle's sampled checks at full size rely on that).  Weights are
N(0, std^2) with std 0.02; bf16 weights are the fp32 draw rounded to the
nearest bf16 (ties to even) and stored as uint16 bit patterns; norm weights are
ones.  Nothing here evaluates the decoder or the sampling rule.
"""

from __future__ import annotations

import zlib
from typing import Dict, List, Sequence

import numpy as np

from .configs import ModelShape


def _key(tag: str) -> int:
    return zlib.crc32(tag.encode("utf-8"))


def rng_for(seed: int, tag: str, *idx: int) -> np.random.Generator:
    """Independent PCG64 stream for ``(seed, tag, idx...)``."""
    ss = np.random.SeedSequence([int(seed) & 0xFFFFFFFF, int(seed) >> 32,
                                 _key(tag)] + [int(i) for i in idx])
    return np.random.Generator(np.random.PCG64(ss))


def bf16_round_u16(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest, ties to even.
    Inputs here are finite normal draws, so NaN handling is not needed."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_u16_to_f32(u: np.ndarray) -> np.ndarray:
    """bf16 bit pattern -> fp32 (exact widening), for generating derived inputs."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal(seed: int, shape: ModelShape, tensor: str, layer: int, size) -> np.ndarray:
    g = rng_for(seed, f"{shape.name}/{tensor}", layer)
    w = g.standard_normal(size, dtype=np.float32)
    w *= np.float32(shape.init_std)
    if shape.dtype == "bf16":
        return bf16_round_u16(w)
    return w


def _ones(shape: ModelShape, n: int) -> np.ndarray:
    one = np.ones(n, dtype=np.float32)
    return bf16_round_u16(one) if shape.dtype == "bf16" else one


def layer_weights(shape: ModelShape, seed: int, layer: int) -> Dict[str, np.ndarray]:
    """One decoder layer's weights, row-major with the reduction dim innermost.

    wqkv      [(Hq + 2 Hkv) * hd, d]  rows: all q heads, then k heads, then v heads
    wo        [d, Hq * hd]
    w_gate_up [2 * ffn, d]            rows 0..ffn-1 gate, ffn..2 ffn-1 up
    w_down    [d, ffn]
    attn_norm, mlp_norm [d]
    """
    d, f = shape.d_model, shape.ffn_dim
    return {
        "attn_norm": _ones(shape, d),
        "wqkv": _normal(seed, shape, "wqkv", layer, (shape.qkv_rows, d)),
        "wo": _normal(seed, shape, "wo", layer, (d, shape.q_dim)),
        "mlp_norm": _ones(shape, d),
        "w_gate_up": _normal(seed, shape, "w_gate_up", layer, (2 * f, d)),
        "w_down": _normal(seed, shape, "w_down", layer, (d, f)),
    }


def model_weights(shape: ModelShape, seed: int, n_layers: int | None = None) -> Dict:
    """All weights of one model (``n_layers`` overrides the depth, for reduced-depth
    checks at full width)."""
    L = shape.n_layers if n_layers is None else n_layers
    return {
        "embed": _normal(seed, shape, "embed", 0, (shape.vocab, shape.d_model)),
        "final_norm": _ones(shape, shape.d_model),
        "lm_head": _normal(seed, shape, "lm_head", 0, (shape.vocab, shape.d_model)),
        "layers": [layer_weights(shape, seed, l) for l in range(L)],
    }


def uniform_prompts(seed: int, lengths: Sequence[int], vocab: int) -> List[np.ndarray]:
    """Uniform-random token ids, one independent stream per sequence."""
    return [rng_for(seed, "prompt", s).integers(0, vocab, size=int(n), dtype=np.int64).astype(np.int32)
            for s, n in enumerate(lengths)]


def prompt_lengths_uniform(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """Lengths uniform on the integers [lo, hi]."""
    return rng_for(seed, "prompt-len").integers(lo, hi + 1, size=batch).astype(np.int32)


def context_lengths_loguniform(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """floor(exp(U(ln lo, ln hi))): the log-uniform context-length mix."""
    g = rng_for(seed, "ctx-len")
    x = g.uniform(np.log(lo), np.log(hi), size=batch)
    return np.clip(np.floor(np.exp(x)), lo, hi).astype(np.int32)


def draft_lengths(seed: int, batch: int, choices: Sequence[int]) -> np.ndarray:
    """Per-sequence draft length k_s drawn uniformly from ``choices``."""
    if len(choices) == 1:
        return np.full(batch, choices[0], dtype=np.int32)
    g = rng_for(seed, "draft-len")
    return np.asarray(choices, dtype=np.int32)[g.integers(0, len(choices), size=batch)]


def seq_ids_for(seed: int, batch: int) -> np.ndarray:
    """Stable caller-chosen 64-bit sequence ids (they key the random streams, so
    they deliberately use bits above 32)."""
    g = rng_for(seed, "seq-ids")
    ids = g.integers(1, 1 << 44, size=batch, dtype=np.int64)
    return ids


def vocab_logits(seed: int, seqs: Sequence[int], k: int, vocab: int,
                 p_std: float = 3.0, q_noise_std: float = 1.0):
    """Synthetic target and draft logits for the vocab-pass workload.

    For each listed sequence index s: target rows p[s] ~ N(0, p_std^2), shape
    (k+1, V); draft rows q[s] = p[s, :k] + N(0, q_noise_std^2), shape (k, V).
    Returns (p, q) as fp32 arrays of shape (len(seqs), k+1, V) and (len(seqs), k, V).
    """
    n = len(seqs)
    p = np.empty((n, k + 1, vocab), dtype=np.float32)
    q = np.empty((n, k, vocab), dtype=np.float32)
    for i, s in enumerate(seqs):
        gp = rng_for(seed, "vocab-p", int(s))
        p[i] = gp.standard_normal((k + 1, vocab), dtype=np.float32) * np.float32(p_std)
        gq = rng_for(seed, "vocab-q", int(s))
        q[i] = p[i, :k] + gq.standard_normal((k, vocab), dtype=np.float32) * np.float32(q_noise_std)
    return p, q


def vocab_temperatures(batch: int, temps: Sequence[float]) -> np.ndarray:
    """T_s cycles through ``temps`` by sequence index."""
    return np.asarray([temps[s % len(temps)] for s in range(batch)], dtype=np.float32)


def base_positions(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """Seeded absolute position n_s of each sequence's pending token, in [lo, hi)."""
    return rng_for(seed, "base-pos").integers(lo, hi, size=batch).astype(np.int32)


def mix_draws(seed: int, seq_ids, positions, rate: float) -> np.ndarray:
    """Bernoulli(rate) per (sequence, drafted position): whether draft mixing
    guides that draft to the target's top-1 token (workload shaping)."""
    return np.array([rng_for(seed, "mix", int(s), int(p)).random() < rate
                     for s, p in zip(seq_ids, positions)], dtype=bool)
