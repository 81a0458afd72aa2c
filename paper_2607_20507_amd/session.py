"""Device-side setup around the C ABI: model weights and descriptors, KV pools,
workspace, and a session object whose methods call the library one to one.

Marshalling only: weights are copied (or drawn, for the large random-init
models) into device tensors that the library reads through raw pointers.
"""

from __future__ import annotations

import ctypes
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import binding as B

_TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}
_SPEC_DTYPE = {"f32": B.SPEC_F32, "bf16": B.SPEC_BF16}


def to_device(a: np.ndarray, device) -> torch.Tensor:
    """numpy fp32 array or bf16 bit pattern (uint16) -> device tensor (bits kept)."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class DeviceModel:
    """A decoder's weights on the GPU and its spec_model_desc.

    weights: the dict of ``workloads.gen.model_weights`` (numpy), uploaded and,
    for bf16, converted in place to the library's tiled weight layout;
    or None with ``seed`` to draw N(0, std^2) weights on the device (torch's
    generator; used for the large random-init models where host generation and
    upload would dominate set-up time)."""

    def __init__(self, shape, weights: Optional[Dict] = None, device="cuda", seed: int = 0,
                 n_layers: Optional[int] = None):
        self.shape = shape
        self.device = torch.device(device)
        L = shape.n_layers if n_layers is None else n_layers
        self.n_layers = L
        if weights is not None:
            self.t = {
                "embed": to_device(weights["embed"], self.device),
                "final_norm": to_device(weights["final_norm"], self.device),
                "lm_head": to_device(weights["lm_head"], self.device),
                "layers": [{k: to_device(v, self.device) for k, v in lw.items()} for lw in weights["layers"][:L]],
            }
        else:
            self.t = self._draw(seed, L)
        self._layers = (B.spec_layer_weights * L)()
        for l, lw in enumerate(self.t["layers"]):
            self._layers[l] = B.spec_layer_weights(*(lw[k].data_ptr() for k in
                                                     ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gate_up", "w_down")))
        sh = shape
        self.desc = B.spec_model_desc(L, sh.d_model, sh.n_heads, sh.n_kv_heads, sh.head_dim, sh.ffn_dim,
                                      sh.vocab, _SPEC_DTYPE[sh.dtype], sh.rope_theta, sh.rms_eps,
                                      self.t["embed"].data_ptr(), self.t["final_norm"].data_ptr(),
                                      self.t["lm_head"].data_ptr(),
                                      ctypes.cast(self._layers, ctypes.POINTER(B.spec_layer_weights)),
                                      B.SPEC_LAYOUT_ROWMAJOR)
        # bf16 projections go to the tiled layout the kernels stream (in place)
        B.spec_pack_model(self.desc)

    def _draw(self, seed: int, L: int):
        sh = self.shape
        dt = _TORCH_DTYPE[sh.dtype]
        g = torch.Generator(device=self.device)

        def normal(tag: int, rows: int, cols: int) -> torch.Tensor:
            g.manual_seed(seed * 1_000_003 + tag)
            out = torch.empty(rows, cols, dtype=dt, device=self.device)
            step = max(1, (1 << 26) // cols)
            for s in range(0, rows, step):
                e = min(rows, s + step)
                out[s:e] = (torch.randn(e - s, cols, generator=g, device=self.device) * sh.init_std).to(dt)
            return out

        ones = lambda: torch.ones(sh.d_model, dtype=dt, device=self.device)
        d, f = sh.d_model, sh.ffn_dim
        layers = []
        for l in range(L):
            layers.append({
                "attn_norm": ones(), "mlp_norm": ones(),
                "wqkv": normal(10 * l + 1, sh.qkv_rows, d),
                "wo": normal(10 * l + 2, d, sh.q_dim),
                "w_gate_up": normal(10 * l + 3, 2 * f, d),
                "w_down": normal(10 * l + 4, d, f),
            })
        return {"embed": normal(7_000_001, sh.vocab, d), "final_norm": ones(),
                "lm_head": normal(7_000_002, sh.vocab, d), "layers": layers}


class SpecSession:
    """One library context with its pools and workspace; methods mirror the C calls."""

    def __init__(self, target: DeviceModel, draft: Optional[DeviceModel], *, max_seqs: int, k_max: int,
                 max_pages_per_seq: int, num_pages_target: Optional[int] = None,
                 num_pages_draft: Optional[int] = None, max_rows: int = 2048, graphs: bool = True):
        """draft None: a decode-only context over `target` (decode())."""
        self.target, self.draft = target, draft
        self.k_max = k_max
        dev = target.device
        npt = num_pages_target or max_seqs * max_pages_per_seq
        npd = (num_pages_draft or max_seqs * max_pages_per_seq) if draft is not None else 0
        self.kv_target = torch.zeros(B.spec_kv_pool_bytes(target.desc, npt), dtype=torch.uint8, device=dev)
        self.kv_draft = (torch.zeros(B.spec_kv_pool_bytes(draft.desc, npd), dtype=torch.uint8, device=dev)
                         if draft is not None else None)
        self.cache = B.spec_cache_desc(16, npt, npd, max_seqs, max_pages_per_seq, k_max, max_rows,
                                       self.kv_target.data_ptr(),
                                       self.kv_draft.data_ptr() if draft is not None else None)
        self.ctx = B.spec_ctx_create(target.desc, draft.desc if draft is not None else None, self.cache)
        nbytes = B.spec_workspace_bytes(self.ctx)
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=dev)
        off = (-self.workspace.data_ptr()) % 256
        self.ws_view = self.workspace[off:off + nbytes]
        B.spec_set_workspace(self.ctx, self.ws_view)
        B.spec_set_graphs(self.ctx, graphs)

    def close(self):
        if self.ctx:
            B.spec_ctx_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prefill(self, seq_ids, prompts, stream=None):
        B.spec_prefill(self.ctx, seq_ids, prompts, stream)

    def set_graphs(self, enable: bool):
        B.spec_set_graphs(self.ctx, enable)

    def draft_step(self, seq_ids, temps, seed: int, stream=None):
        B.spec_draft_step(self.ctx, seq_ids, temps, seed, stream)

    def draft_step_guided(self, seq_ids, temps, seed: int, guide, boost: float, stream=None):
        B.spec_draft_step_guided(self.ctx, seq_ids, temps, seed, guide, boost, stream)

    def draft_loop(self, seq_ids, temps, seed: int, steps, stream=None):
        """steps[i] draft steps for sequence i in one call (one graph)."""
        B.spec_draft_loop(self.ctx, seq_ids, temps, seed, steps, stream)

    def target_forward(self, seq_ids, stream=None):
        B.spec_target_forward(self.ctx, seq_ids, stream)

    def set_drafts(self, seq_id: int, tokens, q_logits, stream=None):
        B.spec_set_drafts(self.ctx, seq_id, tokens, q_logits, stream)

    def set_draft_tree(self, seq_id: int, parents, tokens, q_logits, stream=None):
        B.spec_set_draft_tree(self.ctx, seq_id, parents, tokens, q_logits, stream)

    def verify(self, seq_ids, temps, seed: int, stream=None):
        return B.spec_verify(self.ctx, seq_ids, temps, seed, self.k_max, stream)

    def verify_commit_draft(self, seq_ids, temps, verify_seed: int, draft_seed: int, steps, stream=None):
        """verify, commit with the accepted counts, then draft_loop of the next round, in one call."""
        return B.spec_verify_commit_draft(self.ctx, seq_ids, temps, verify_seed, self.k_max, draft_seed, steps,
                                          stream)

    def decode(self, seq_ids, temps, seed: int, steps: int, stream=None):
        """Plain decoding of the target model: tokens [n, steps]."""
        return B.spec_decode(self.ctx, seq_ids, temps, seed, steps, stream)

    def commit(self, seq_ids, n_accepted, stream=None):
        B.spec_kv_commit(self.ctx, seq_ids, n_accepted, stream)

    def rollback(self, seq_id: int, new_len: int, stream=None):
        B.spec_kv_rollback(self.ctx, seq_id, new_len, stream)

    def release(self, seq_id: int):
        B.spec_seq_release(self.ctx, seq_id)

    def seq_info(self, seq_id: int):
        return B.spec_seq_info(self.ctx, seq_id)

    def draft_tokens(self, seq_id: int, stream=None):
        """The sequence's current draft tokens (list of int)."""
        return [int(x) for x in B.spec_draft_tokens(self.ctx, seq_id, self.k_max, stream)]

    def draft_logits(self, seq_id: int, j: int) -> torch.Tensor:
        """Copy of the draft logits row [V] (fp32) behind draft j of seq_id
        (drafts made by draft_step live in this session's workspace)."""
        ptr = B.spec_draft_logits(self.ctx, seq_id, j)
        V = self.target.shape.vocab
        off = ptr - self.ws_view.data_ptr()
        return self.ws_view[off:off + V * 4].view(torch.float32).clone()

    def last_logits(self) -> torch.Tensor:
        """Copy of the last verify's target logits [rows, V] (fp32)."""
        ptr, rows = B.spec_last_logits(self.ctx)
        V = self.target.shape.vocab
        base = self.ws_view.data_ptr()
        off = ptr - base
        flat = self.ws_view[off:off + rows * V * 4].view(torch.float32)
        return flat.view(rows, V).clone()
