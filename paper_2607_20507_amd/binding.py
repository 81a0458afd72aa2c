"""ctypes binding of libspecverify.so (include/spec.h, include/spec_ops.h).

Argument marshalling only: every step of the verify path runs in the HIP
library.  PyTorch supplies device memory and the stream.  If the library is
not built this module raises on first use; there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_int64, c_size_t, c_uint64, c_void_p
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspecverify.so")

SPEC_OK, SPEC_E_INVALID, SPEC_E_NOPAGES, SPEC_E_HIP, SPEC_E_STATE, SPEC_E_UNSUPPORTED = range(6)
SPEC_F32, SPEC_BF16 = 0, 1
SPEC_LAYOUT_ROWMAJOR, SPEC_LAYOUT_TILED = 0, 1
SPEC_DRAFT, SPEC_ACCEPT, SPEC_RESAMPLE, SPEC_BONUS = range(4)
SPEC_EPI_STORE_F32, SPEC_EPI_ADD_F32, SPEC_EPI_SWIGLU = range(3)

STATUS_NAMES = {0: "SPEC_OK", 1: "SPEC_E_INVALID", 2: "SPEC_E_NOPAGES", 3: "SPEC_E_HIP",
                4: "SPEC_E_STATE", 5: "SPEC_E_UNSUPPORTED"}


class SpecError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class spec_layer_weights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gate_up", "w_down")]


class spec_model_desc(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("ffn_dim", c_int32),
                ("vocab", c_int32), ("dtype", c_int32), ("rope_theta", c_float),
                ("rms_eps", c_float), ("embed", c_void_p), ("final_norm", c_void_p),
                ("lm_head", c_void_p), ("layers", POINTER(spec_layer_weights)),
                ("weight_layout", c_int32)]


class spec_cache_desc(ctypes.Structure):
    _fields_ = [("page_size", c_int32), ("num_pages_target", c_int32), ("num_pages_draft", c_int32),
                ("max_seqs", c_int32), ("max_pages_per_seq", c_int32), ("k_max", c_int32),
                ("max_rows", c_int32), ("kv_target", c_void_p), ("kv_draft", c_void_p)]


_P = c_void_p
_I32P = POINTER(c_int32)
_I64P = POINTER(c_int64)
_F32P = POINTER(c_float)

# name -> (restype, argtypes); mirrors the headers
SIGNATURES = {
    "spec_kv_pool_bytes": (c_size_t, [POINTER(spec_model_desc), c_int32]),
    "spec_ctx_create": (c_int32, [POINTER(spec_model_desc), POINTER(spec_model_desc),
                                  POINTER(spec_cache_desc), POINTER(c_void_p)]),
    "spec_ctx_destroy": (None, [_P]),
    "spec_last_error": (ctypes.c_char_p, [_P]),
    "spec_workspace_bytes": (c_size_t, [_P]),
    "spec_set_workspace": (c_int32, [_P, _P, c_size_t]),
    "spec_prefill": (c_int32, [_P, c_int32, _I64P, _I32P, _I32P, _P]),
    "spec_draft_step": (c_int32, [_P, c_int32, _I64P, _F32P, c_uint64, _P]),
    "spec_set_drafts": (c_int32, [_P, c_int64, c_int32, _I32P, _P, _P]),
    "spec_set_draft_tree": (c_int32, [_P, c_int64, c_int32, _I32P, _I32P, _P, _P]),
    "spec_verify": (c_int32, [_P, c_int32, _I64P, _F32P, c_uint64, _I32P, _I32P, _P]),
    "spec_kv_commit": (c_int32, [_P, c_int32, _I64P, _I32P, _P]),
    "spec_kv_rollback": (c_int32, [_P, c_int64, c_int32, _P]),
    "spec_seq_release": (c_int32, [_P, c_int64]),
    "spec_seq_info": (c_int32, [_P, c_int64, _I32P, _I32P, _I32P, _I32P, _I32P, _I32P, _I32P, c_int32]),
    "spec_last_logits": (c_int32, [_P, POINTER(c_void_p), _I32P]),
    "spec_set_graphs": (c_int32, [_P, c_int32]),
    "spec_draft_step_guided": (c_int32, [_P, c_int32, _I64P, _F32P, c_uint64, _I32P, c_float, _P]),
    "spec_draft_loop": (c_int32, [_P, c_int32, _I64P, _F32P, c_uint64, _I32P, _P]),
    "spec_verify_commit_draft": (c_int32, [_P, c_int32, _I64P, _F32P, c_uint64, _I32P, _I32P, c_uint64, _I32P,
                                           _P]),
    "spec_decode": (c_int32, [_P, c_int32, _I64P, _F32P, c_uint64, c_int32, _I32P, _P]),
    "spec_target_forward": (c_int32, [_P, c_int32, _I64P, _P]),
    "spec_draft_logits": (c_int32, [_P, c_int64, c_int32, _P]),
    "spec_draft_tokens": (c_int32, [_P, c_int64, _P, _P, _P]),
    "spec_timing_enable": (c_int32, [_P, ctypes.c_char_p]),
    "spec_timing_read": (c_int32, [_P, POINTER(ctypes.c_double), _I64P, POINTER(ctypes.c_double),
                                   POINTER(ctypes.c_double)]),
    "spec_sample_workspace_bytes": (c_size_t, [c_int32, c_int32, c_int32]),
    "spec_sample_verify": (c_int32, [c_int32, _I32P, _F32P, _I64P, _I32P, _P, _P, _P, c_int32,
                                     c_uint64, _P, _P, _P, c_size_t, _P]),
    "spec_sample_verify_noalloc": (c_int32, [c_int32, c_int32, _P, _P, _P, _P, _P, _P, _P, c_int32, c_uint64,
                                             _P, _P, _P]),
    "spec_sample_draft": (c_int32, [c_int32, _P, c_int32, _F32P, _I64P, _I32P, c_uint64, _P, _P,
                                    c_size_t, _P]),
    "spec_philox_uniform": (c_int32, [c_uint64, c_int64, c_int32, c_int32, c_int32, _P, _P]),
    "spec_pack_model": (c_int32, [POINTER(spec_model_desc), _P]),
    "spec_pack_weight": (c_int32, [_P, c_int32, c_int32, c_int32, c_int32, _P]),
    "spec_op_gemm_workspace_bytes": (c_size_t, [c_int32, c_int32]),
    "spec_op_gemm": (c_int32, [c_int32, c_int32, c_int32, c_int32, _P, _P, _P, c_int32, _P, c_size_t, _P]),
    "spec_op_rmsnorm": (c_int32, [c_int32, c_int32, c_int32, _P, _P, c_float, _P, _P]),
    "spec_op_rope_kv": (c_int32, [c_int32, c_int32, c_int32, c_int32, c_int32, c_float, _P, _P, _P,
                                  _P, _P, _P, _P]),
    "spec_op_attention_workspace_bytes": (c_size_t, [c_int32, c_int32, c_int32, c_int32, c_int32]),
    "spec_op_attention": (c_int32, [c_int32, c_int32, _I32P, _I32P, _I32P, c_int32, c_int32, c_int32,
                                    c_int32, _P, _P, _P, _P, _P, c_size_t, _P]),
}

_lib = None


def lib():
    """Load the in-tree HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2607_20507_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


# ---------------------------------------------------------------------------
# marshalling helpers

def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def _ptr(a: np.ndarray, t):
    return a.ctypes.data_as(t)


def dptr(t) -> Optional[int]:
    """Device address of a torch tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def stream_ptr(stream=None) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def check(status: int, ctx=None):
    if status != SPEC_OK:
        msg = lib().spec_last_error(ctx)
        raise SpecError(status, msg.decode() if msg else "")


# ---------------------------------------------------------------------------
# thin wrappers with the C names

def spec_kv_pool_bytes(desc: spec_model_desc, num_pages: int) -> int:
    return lib().spec_kv_pool_bytes(ctypes.byref(desc), num_pages)


def spec_ctx_create(target: spec_model_desc, draft: Optional[spec_model_desc], cache: spec_cache_desc) -> int:
    """draft None: a decode-only context over the target model (spec_decode)."""
    out = c_void_p()
    check(lib().spec_ctx_create(ctypes.byref(target), ctypes.byref(draft) if draft is not None else None,
                                ctypes.byref(cache), ctypes.byref(out)))
    return out.value


def spec_ctx_destroy(ctx: int):
    lib().spec_ctx_destroy(ctx)


def spec_workspace_bytes(ctx: int) -> int:
    return lib().spec_workspace_bytes(ctx)


def spec_set_workspace(ctx: int, ws) -> None:
    check(lib().spec_set_workspace(ctx, dptr(ws), ws.numel() * ws.element_size()), ctx)


def spec_prefill(ctx: int, seq_ids, prompts: Sequence[Sequence[int]], stream=None):
    ids = _i64(seq_ids)
    lens = _i32([len(p) for p in prompts])
    toks = _i32(np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts]) if len(prompts) else [])
    check(lib().spec_prefill(ctx, len(ids), _ptr(ids, _I64P), _ptr(lens, _I32P), _ptr(toks, _I32P),
                             stream_ptr(stream)), ctx)


def spec_draft_step(ctx: int, seq_ids, temperature, seed: int, stream=None):
    ids = _i64(seq_ids)
    t = _f32(temperature)
    check(lib().spec_draft_step(ctx, len(ids), _ptr(ids, _I64P), _ptr(t, _F32P), seed,
                                stream_ptr(stream)), ctx)


def spec_draft_step_guided(ctx: int, seq_ids, temperature, seed: int, guide, boost: float, stream=None):
    ids = _i64(seq_ids)
    t = _f32(temperature)
    g = np.ascontiguousarray(np.asarray(guide, dtype=np.int32))
    check(lib().spec_draft_step_guided(ctx, len(ids), _ptr(ids, _I64P), _ptr(t, _F32P), seed, _ptr(g, _I32P),
                                       float(boost), stream_ptr(stream)), ctx)


def spec_draft_loop(ctx: int, seq_ids, temperature, seed: int, steps, stream=None):
    ids = _i64(seq_ids)
    t = _f32(temperature)
    k = np.ascontiguousarray(np.asarray(steps, dtype=np.int32))
    check(lib().spec_draft_loop(ctx, len(ids), _ptr(ids, _I64P), _ptr(t, _F32P), seed, _ptr(k, _I32P),
                                stream_ptr(stream)), ctx)


def spec_target_forward(ctx: int, seq_ids, stream=None):
    ids = _i64(seq_ids)
    check(lib().spec_target_forward(ctx, len(ids), _ptr(ids, _I64P), stream_ptr(stream)), ctx)


def spec_set_drafts(ctx: int, seq_id: int, tokens, q_logits, stream=None):
    tk = _i32(tokens)
    check(lib().spec_set_drafts(ctx, int(seq_id), len(tk), _ptr(tk, _I32P), dptr(q_logits),
                                stream_ptr(stream)), ctx)


def spec_set_draft_tree(ctx: int, seq_id: int, parents, tokens, q_logits, stream=None):
    """q_logits: device fp32 [m + 1, V] (row 0 the root's children's draft logits)."""
    pa = _i32(parents)
    tk = _i32(tokens)
    check(lib().spec_set_draft_tree(ctx, int(seq_id), len(tk), _ptr(pa, _I32P), _ptr(tk, _I32P), dptr(q_logits),
                                    stream_ptr(stream)), ctx)


def spec_verify(ctx: int, seq_ids, temperature, seed: int, k_max: int, stream=None):
    """Returns (n_accepted [n], out_tokens [n, k_max + 1])."""
    ids = _i64(seq_ids)
    t = _f32(temperature)
    n = len(ids)
    na = np.zeros(n, dtype=np.int32)
    ot = np.full((n, k_max + 1), -1, dtype=np.int32)
    check(lib().spec_verify(ctx, n, _ptr(ids, _I64P), _ptr(t, _F32P), seed, _ptr(na, _I32P),
                            _ptr(ot, _I32P), stream_ptr(stream)), ctx)
    return na, ot


def spec_verify_commit_draft(ctx: int, seq_ids, temperature, verify_seed: int, k_max: int, draft_seed: int,
                             steps, stream=None):
    """spec_verify, spec_kv_commit and spec_draft_loop in one call.
    Returns (n_accepted [n], out_tokens [n, k_max + 1])."""
    ids = _i64(seq_ids)
    t = _f32(temperature)
    n = len(ids)
    k = np.ascontiguousarray(np.asarray(steps, dtype=np.int32))
    na = np.zeros(n, dtype=np.int32)
    ot = np.full((n, k_max + 1), -1, dtype=np.int32)
    check(lib().spec_verify_commit_draft(ctx, n, _ptr(ids, _I64P), _ptr(t, _F32P), verify_seed, _ptr(na, _I32P),
                                         _ptr(ot, _I32P), draft_seed, _ptr(k, _I32P), stream_ptr(stream)), ctx)
    return na, ot


def spec_decode(ctx: int, seq_ids, temperature, seed: int, steps: int, stream=None):
    """Plain decoding of the context's target model; returns tokens [n, steps]."""
    ids = _i64(seq_ids)
    t = _f32(temperature)
    out = np.full((len(ids), max(steps, 0)), -1, dtype=np.int32)
    check(lib().spec_decode(ctx, len(ids), _ptr(ids, _I64P), _ptr(t, _F32P), seed, steps, _ptr(out, _I32P),
                            stream_ptr(stream)), ctx)
    return out


def spec_kv_commit(ctx: int, seq_ids, n_accepted, stream=None):
    ids = _i64(seq_ids)
    na = _i32(n_accepted)
    check(lib().spec_kv_commit(ctx, len(ids), _ptr(ids, _I64P), _ptr(na, _I32P), stream_ptr(stream)), ctx)


def spec_kv_rollback(ctx: int, seq_id: int, new_len: int, stream=None):
    check(lib().spec_kv_rollback(ctx, int(seq_id), int(new_len), stream_ptr(stream)), ctx)


def spec_seq_release(ctx: int, seq_id: int):
    check(lib().spec_seq_release(ctx, int(seq_id)), ctx)


def spec_seq_info(ctx: int, seq_id: int, max_pages: int = 4096):
    tl, dl, pp, nt, nd = (c_int32() for _ in range(5))
    pt = np.zeros(max_pages, dtype=np.int32)
    pd = np.zeros(max_pages, dtype=np.int32)
    check(lib().spec_seq_info(ctx, int(seq_id), ctypes.byref(tl), ctypes.byref(dl), ctypes.byref(pp),
                              _ptr(pt, _I32P), ctypes.byref(nt), _ptr(pd, _I32P), ctypes.byref(nd),
                              max_pages), ctx)
    return {"target_len": tl.value, "draft_len": dl.value, "pending_pos": pp.value,
            "pages_target": pt[:nt.value].tolist(), "pages_draft": pd[:nd.value].tolist()}


def spec_last_logits(ctx: int):
    p = c_void_p()
    r = c_int32()
    check(lib().spec_last_logits(ctx, ctypes.byref(p), ctypes.byref(r)), ctx)
    return p.value, r.value


def spec_draft_logits(ctx: int, seq_id: int, j: int) -> int:
    """Device address of the draft logits row that drew draft j of seq_id."""
    p = c_void_p()
    check(lib().spec_draft_logits(ctx, seq_id, j, ctypes.byref(p)), ctx)
    return p.value


def spec_draft_tokens(ctx: int, seq_id: int, k_max: int, stream=None) -> np.ndarray:
    """The sequence's current draft tokens (host int32 [k])."""
    out = np.zeros(max(1, k_max), dtype=np.int32)
    k = c_int32()
    check(lib().spec_draft_tokens(ctx, seq_id, out.ctypes.data, ctypes.byref(k), stream_ptr(stream)), ctx)
    return out[:k.value].copy()


def spec_set_graphs(ctx: int, enable: bool) -> None:
    check(lib().spec_set_graphs(ctx, 1 if enable else 0), ctx)


def spec_timing_enable(ctx: int, kernel_name: Optional[str]):
    check(lib().spec_timing_enable(ctx, kernel_name.encode() if kernel_name else None), ctx)


def spec_timing_read(ctx: int):
    """-> (total_ms, launches, bytes, flops) of the timed kernel since enable."""
    ms, b, f = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    n = c_int64()
    check(lib().spec_timing_read(ctx, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(b), ctypes.byref(f)), ctx)
    return ms.value, n.value, b.value, f.value


def spec_sample_workspace_bytes(B: int, total_rows: int, V: int) -> int:
    return lib().spec_sample_workspace_bytes(B, total_rows, V)


def spec_sample_verify(k, temperature, seq_ids, base_pos, p_logits, q_logits, draft_tokens, V: int,
                       seed: int, n_accepted, out_tokens, workspace, stream=None):
    kk = _i32(k)
    t = _f32(temperature)
    ids = _i64(seq_ids)
    bp = _i32(base_pos)
    check(lib().spec_sample_verify(len(kk), _ptr(kk, _I32P), _ptr(t, _F32P), _ptr(ids, _I64P),
                                   _ptr(bp, _I32P), dptr(p_logits), dptr(q_logits), dptr(draft_tokens),
                                   V, seed, dptr(n_accepted), dptr(out_tokens), dptr(workspace),
                                   workspace.numel() * workspace.element_size(), stream_ptr(stream)))


def spec_sample_verify_noalloc(k_max: int, k, temperature, seq_ids, base_pos, p_logits, q_logits, draft_tokens,
                               V: int, seed: int, n_accepted, out_tokens, stream=None):
    """k, temperature, seq_ids, base_pos: device tensors (int32, float32, int64, int32)."""
    check(lib().spec_sample_verify_noalloc(k.numel(), k_max, dptr(k), dptr(temperature), dptr(seq_ids),
                                           dptr(base_pos), dptr(p_logits), dptr(q_logits), dptr(draft_tokens),
                                           V, seed, dptr(n_accepted), dptr(out_tokens), stream_ptr(stream)))


def spec_sample_draft(logits, V: int, temperature, seq_ids, pos, seed: int, tokens, workspace, stream=None):
    t = _f32(temperature)
    ids = _i64(seq_ids)
    ps = _i32(pos)
    check(lib().spec_sample_draft(len(t), dptr(logits), V, _ptr(t, _F32P), _ptr(ids, _I64P), _ptr(ps, _I32P),
                                  seed, dptr(tokens), dptr(workspace),
                                  workspace.numel() * workspace.element_size(), stream_ptr(stream)))


def spec_philox_uniform(seed: int, seq_id: int, pos: int, purpose: int, n: int, out, stream=None):
    check(lib().spec_philox_uniform(seed, int(seq_id), pos, purpose, n, dptr(out), stream_ptr(stream)))


def spec_pack_model(desc: spec_model_desc, stream=None) -> None:
    check(lib().spec_pack_model(ctypes.byref(desc), stream_ptr(stream)))


def spec_pack_weight(w, rows: int, K: int, rot_rows: int = 0, head_dim: int = 0, stream=None) -> None:
    check(lib().spec_pack_weight(dptr(w), rows, K, rot_rows, head_dim, stream_ptr(stream)))


def spec_op_gemm_workspace_bytes(R: int, Nw: int) -> int:
    return lib().spec_op_gemm_workspace_bytes(R, Nw)


def spec_op_gemm(dtype: int, R: int, N: int, K: int, X, W, Y, epilogue: int, workspace=None, stream=None):
    wb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    check(lib().spec_op_gemm(dtype, R, N, K, dptr(X), dptr(W), dptr(Y), epilogue, dptr(workspace), wb,
                             stream_ptr(stream)))


def spec_op_rmsnorm(dtype: int, R: int, d: int, h, w, eps: float, y, stream=None):
    check(lib().spec_op_rmsnorm(dtype, R, d, dptr(h), dptr(w), eps, dptr(y), stream_ptr(stream)))


def spec_op_rope_kv(dtype: int, R: int, n_heads: int, n_kv_heads: int, head_dim: int, theta: float,
                    qkv, pos, slot, q_out, k_pages, v_pages, stream=None):
    check(lib().spec_op_rope_kv(dtype, R, n_heads, n_kv_heads, head_dim, theta, dptr(qkv), dptr(pos),
                                dptr(slot), dptr(q_out), dptr(k_pages), dptr(v_pages), stream_ptr(stream)))


def spec_op_attention_workspace_bytes(n_seqs: int, total_rows: int, max_pages: int, n_kv_heads: int,
                                      head_dim: int) -> int:
    return lib().spec_op_attention_workspace_bytes(n_seqs, total_rows, max_pages, n_kv_heads, head_dim)


def spec_op_attention(dtype: int, rows, pos0, page_table, n_heads: int, n_kv_heads: int, head_dim: int,
                      q, k_pages, v_pages, out, workspace, stream=None):
    r = _i32(rows)
    p = _i32(pos0)
    pt = _i32(page_table)
    check(lib().spec_op_attention(dtype, len(r), _ptr(r, _I32P), _ptr(p, _I32P), _ptr(pt, _I32P),
                                  pt.shape[1], n_heads, n_kv_heads, head_dim, dptr(q), dptr(k_pages),
                                  dptr(v_pages), dptr(out), dptr(workspace),
                                  workspace.numel() * workspace.element_size(), stream_ptr(stream)))
