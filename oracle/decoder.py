"""Float64 forward pass of a Llama-style decoder with a per-sequence KV list.

The paper runs its drafter and target as ordinary autoregressive decoders
(Section 4.1: Qwen3-32B with Qwen3-1.7B; the small-model appendix, Table 10:
Llama-3.3-70B with Llama-3.2-1B/3B).  It prints no architecture details; the
stand-in models use the Llama layer, written out here by its definition:

  h   = E[token]
  per layer:
    y   = RMSNorm(h) * w_attn           RMSNorm(x) = x / sqrt(mean(x^2) + eps)
    q, k, v = y Wqkv^T                  (q: Hq heads, k/v: Hkv heads of size hd)
    q, k = RoPE(q, pos), RoPE(k, pos)   rotate-half pairs (i, i + hd/2),
                                        angle pos * theta^(-2i/hd)
    o   = softmax(q K^T / sqrt(hd) + causal mask) V, query head h reading kv
          head h // (Hq / Hkv) (grouped-query attention)
    h  += o Wo^T
    y   = RMSNorm(h) * w_mlp
    h  += (silu(y Wg^T) * (y Wu^T)) Wd^T          silu(x) = x / (1 + e^-x)
  logits = (RMSNorm(h) * w_final) Wlm^T

Weights arrive as fp32 arrays or bf16 bit patterns (uint16) and are widened
exactly to float64; every operation below is float64.  Matrix products against
large weights are taken in row blocks of the weight only to bound memory; the
block split changes no arithmetic beyond float64 summation order.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List

import numpy as np

_BLOCK_ROWS = 8192


def widen(w: np.ndarray) -> np.ndarray:
    """fp32 array or bf16 bit pattern (uint16) -> float64, exactly."""
    w = np.asarray(w)
    if w.dtype == np.uint16:
        return (w.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return w.astype(np.float64)


def matmul_wt(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """x @ W^T for W stored [N, K] (fp32 or bf16 bits), float64 result."""
    n = w.shape[0]
    if n <= _BLOCK_ROWS:
        return x @ widen(w).T
    out = np.empty((x.shape[0], n), dtype=np.float64)
    for s in range(0, n, _BLOCK_ROWS):
        out[:, s:s + _BLOCK_ROWS] = x @ widen(w[s:s + _BLOCK_ROWS]).T
    return out


def rms_norm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * widen(w)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [n, H, hd] at absolute positions pos [n]."""
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-2.0 * np.arange(half, dtype=np.float64) / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, qpos: np.ndarray) -> np.ndarray:
    """Causal grouped-query attention.

    q [n, Hq, hd] at absolute positions qpos; K, V [T, Hkv, hd] hold positions
    0..T-1.  Query row r sees keys 0..qpos[r].  Returns [n, Hq, hd]."""
    n, hq, hd = q.shape
    hkv = K.shape[1]
    group = hq // hkv
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for r in range(n):
        L = int(qpos[r]) + 1
        for h in range(hq):
            g = h // group
            s = (K[:L, g, :] @ q[r, h]) * scale
            s = np.exp(s - s.max())
            out[r, h] = (s / s.sum()) @ V[:L, g, :]
    return out


@dataclass
class KVList:
    """Per-sequence, per-layer keys (after RoPE) and values, float64, in position order."""

    n_layers: int
    K: List[np.ndarray] = field(default_factory=list)
    V: List[np.ndarray] = field(default_factory=list)

    def __post_init__(self):
        if not self.K:
            self.K = [None] * self.n_layers
            self.V = [None] * self.n_layers

    @property
    def length(self) -> int:
        return 0 if self.K[0] is None else self.K[0].shape[0]

    def append(self, layer: int, k: np.ndarray, v: np.ndarray):
        if self.K[layer] is None:
            self.K[layer], self.V[layer] = k.copy(), v.copy()
        else:
            self.K[layer] = np.concatenate([self.K[layer], k], axis=0)
            self.V[layer] = np.concatenate([self.V[layer], v], axis=0)

    def truncate(self, new_len: int):
        for l in range(self.n_layers):
            if self.K[l] is not None:
                self.K[l] = self.K[l][:new_len]
                self.V[l] = self.V[l][:new_len]


class Decoder:
    """A decoder given by its shape and (raw) weights from ``workloads.gen``."""

    def __init__(self, shape, weights: Dict):
        self.shape = shape
        self.w = weights
        self.n_layers = len(weights["layers"])

    def new_kv(self) -> KVList:
        return KVList(self.n_layers)

    def forward(self, kv: KVList, tokens, positions, logits: bool = True) -> np.ndarray:
        """Run rows ``tokens`` at ``positions`` (which must continue the cache:
        positions == kv.length, kv.length + 1, ...), appending their K/V.
        Returns logits [n, V] (or the final hidden state if ``logits`` is False)."""
        sh = self.shape
        tokens = np.asarray(tokens, dtype=np.int64)
        positions = np.asarray(positions, dtype=np.int64)
        n = tokens.shape[0]
        assert np.array_equal(positions, kv.length + np.arange(n)), "positions must extend the cache"
        hq, hkv, hd = sh.n_heads, sh.n_kv_heads, sh.head_dim
        h = widen(self.w["embed"][tokens])
        for l, lw in enumerate(self.w["layers"]):
            y = rms_norm(h, lw["attn_norm"], sh.rms_eps)
            qkv = matmul_wt(y, lw["wqkv"])
            q = qkv[:, :hq * hd].reshape(n, hq, hd)
            k = qkv[:, hq * hd:(hq + hkv) * hd].reshape(n, hkv, hd)
            v = qkv[:, (hq + hkv) * hd:].reshape(n, hkv, hd)
            q = rope(q, positions, sh.rope_theta)
            k = rope(k, positions, sh.rope_theta)
            kv.append(l, k, v)
            o = attention(q, kv.K[l], kv.V[l], positions)
            h = h + matmul_wt(o.reshape(n, hq * hd), lw["wo"])
            y = rms_norm(h, lw["mlp_norm"], sh.rms_eps)
            gu = matmul_wt(y, lw["w_gate_up"])
            f = sh.ffn_dim
            h = h + matmul_wt(silu(gu[:, :f]) * gu[:, f:], lw["w_down"])
        y = rms_norm(h, self.w["final_norm"], sh.rms_eps)
        if not logits:
            return y
        return matmul_wt(y, self.w["lm_head"])

    def kv_at(self, tokens, rows):
        """Every layer's K (after RoPE) and V at the listed positions of the
        no-cache forward over ``tokens``: a list over layers of (K [r, Hkv,
        hd], V [r, Hkv, hd]).  The same arithmetic as ``forward``, restricted
        to what those values depend on: a layer's K/V at a row depend on the
        layer's input at that row only, and its output at a row on its K/V
        at the rows up to it.  So the last layer runs only at ``rows``, the
        one before it outputs only at ``rows`` (attending over its K/V of
        every row up to the last of them), and earlier layers run in full up
        to that row.  (Used to check long prefills at sampled positions.)"""
        sh = self.shape
        tokens = np.asarray(tokens, dtype=np.int64)
        rows = np.asarray(sorted(int(r) for r in rows), dtype=np.int64)
        top = int(rows[-1]) + 1
        hq, hkv, hd = sh.n_heads, sh.n_kv_heads, sh.head_dim
        L = self.n_layers
        idx = np.arange(top)         # rows whose layer input is known
        h = widen(self.w["embed"][tokens[:top]])
        out = []
        for l, lw in enumerate(self.w["layers"]):
            # K/V of every row of idx (all rows up to `top`, or `rows` in the last layer)
            y = rms_norm(h, lw["attn_norm"], sh.rms_eps)
            qkv = matmul_wt(y, lw["wqkv"])
            n = len(idx)
            q = rope(qkv[:, :hq * hd].reshape(n, hq, hd), idx, sh.rope_theta)
            k = rope(qkv[:, hq * hd:(hq + hkv) * hd].reshape(n, hkv, hd), idx, sh.rope_theta)
            v = qkv[:, (hq + hkv) * hd:].reshape(n, hkv, hd)
            sel = np.searchsorted(idx, rows)
            out.append((k[sel], v[sel]))
            if l == L - 1:
                break
            # outputs: at `rows` when the next layer is the last, else at every row
            orow = rows if l == L - 2 else idx
            osel = np.searchsorted(idx, orow)
            o = attention(q[osel], k, v, orow)
            hh = h[osel] + matmul_wt(o.reshape(len(orow), hq * hd), lw["wo"])
            y = rms_norm(hh, lw["mlp_norm"], sh.rms_eps)
            gu = matmul_wt(y, lw["w_gate_up"])
            f = sh.ffn_dim
            h = hh + matmul_wt(silu(gu[:, :f]) * gu[:, f:], lw["w_down"])
            idx = orow
        return out

    def full_logits(self, tokens) -> np.ndarray:
        """No-cache forward over a whole token sequence (positions 0..n-1)."""
        kv = self.new_kv()
        return self.forward(kv, tokens, np.arange(len(tokens)))
