"""KV commit / rollback clear rejected slots in place (spec_kv_commit,
spec_kv_rollback): after a verify and a commit with a accepted drafts, the
target cache slots of positions n+a+1 .. n+k and the draft cache slots past
n+a hold zeros in every layer, kv head and dim, for K and V, while the kept
positions still hold their entries; a rollback to new_len clears positions
new_len .. of both caches.  The pools are read back and indexed by the
documented page layouts: the fp32 cache keeps K [16][hd] and V^T [hd][16]
per (page, kv head) block; the bf16 cache uses the attention kernel's
operand order (the two index formulas below restate the layout comment of
the library's kv_layout.h)."""

import numpy as np
import pytest

from tests.gpu_util import device, say, torch
from workloads import SMALL_BF16, TINY_FP32, model_weights, uniform_prompts

pytestmark = pytest.mark.gpu


def _k_off_bf16(k, d):
    c = d >> 3
    s, g = c >> 2, c & 3
    h, j = (k >> 2) & 1, (k & 3) + 4 * (k >> 3)
    return ((((s * 2 + h) * 4 + g) * 8 + j) << 3) + (d & 7)


def _v_off_bf16(k, d):
    return (((((d >> 4) * 2 + (k >> 3)) * 16) + (d & 15)) << 3) + (k & 7)


class _Pool:
    """Raw bit view of one model's paged KV pool."""

    def __init__(self, pool_u8, shape, n_layers, num_pages):
        self.bf16 = shape.dtype == "bf16"
        self.bits = pool_u8.view(torch.int16 if self.bf16 else torch.int32).cpu().numpy()
        self.L, self.P, self.H, self.hd = n_layers, num_pages, shape.n_kv_heads, shape.head_dim
        self.block = 16 * self.hd
        self.layer = self.P * self.H * self.block * 2
        assert self.bits.size == self.L * self.layer

    def token_bits(self, page, off):
        """All K and V elements (every layer, kv head, dim) of token `off` of `page`."""
        d = np.arange(self.hd)
        if self.bf16:
            ko = np.array([_k_off_bf16(off, x) for x in d])
            vo = np.array([_v_off_bf16(off, x) for x in d])
        else:
            ko, vo = off * self.hd + d, d * 16 + off
        out = []
        for l in range(self.L):
            for h in range(self.H):
                base = l * self.layer + (page * self.H + h) * self.block
                out.append(self.bits[base + ko])
                out.append(self.bits[base + self.layer // 2 + vo])
        return np.concatenate(out)


def _slot(pages, pos):
    return pages[pos // 16], pos % 16


def _session(which, n_seqs):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    cfg, lt, ld = (TINY_FP32, None, None) if which == "fp32" else (SMALL_BF16, 2, 1)
    dev = device()
    tw = model_weights(cfg.target, cfg.seed, lt)
    dw = model_weights(cfg.draft, cfg.seed + 1, ld)
    pages = 24
    gpu = SpecSession(DeviceModel(cfg.target, tw, dev, n_layers=lt), DeviceModel(cfg.draft, dw, dev, n_layers=ld),
                      max_seqs=n_seqs, k_max=max(cfg.k), max_pages_per_seq=pages, max_rows=256)
    Lt = cfg.target.n_layers if lt is None else lt
    Ld = cfg.draft.n_layers if ld is None else ld
    return gpu, cfg, (Lt, Ld), n_seqs * pages


# two sequences: the slots to clear travel in the kernel arguments; four or
# five: more than 16 per pool, uploaded as call metadata
@pytest.mark.parametrize("which,n_seqs", [("fp32", 2), ("bf16", 2), ("fp32", 5), ("bf16", 4)])
def test_commit_and_rollback_clear_rejected_slots(which, n_seqs):
    gpu, cfg, (Lt, Ld), npages = _session(which, n_seqs)
    k = max(cfg.k)
    ids = [11 + i for i in range(n_seqs)]
    prompts = uniform_prompts(cfg.seed + 8, [37 + 13 * i for i in range(n_seqs)], cfg.target.vocab)
    say("kv clear", which, ": prefill, draft", k, "steps, verify, commit with a = 0")
    gpu.prefill(ids, prompts)
    n = {sid: gpu.seq_info(sid)["target_len"] for sid in ids}
    for _ in range(k):
        gpu.draft_step(ids, [1.0] * n_seqs, 3)
    gpu.verify(ids, [1.0] * n_seqs, 3)
    before = {sid: gpu.seq_info(sid) for sid in ids}
    gpu.commit(ids, [0] * n_seqs)
    torch.cuda.synchronize()
    tp = _Pool(gpu.kv_target, cfg.target, Lt, npages)
    dp = _Pool(gpu.kv_draft, cfg.draft, Ld, npages)
    for sid in ids:
        pt, pd = before[sid]["pages_target"], before[sid]["pages_draft"]
        ln_d = before[sid]["draft_len"]
        assert ln_d == n[sid] + k  # the last draft is not in the draft cache
        assert np.any(tp.token_bits(*_slot(pt, n[sid])) != 0), "kept target position lost"
        assert np.any(dp.token_bits(*_slot(pd, n[sid])) != 0), "kept draft position lost"
        for pos in range(n[sid] + 1, n[sid] + k + 1):
            assert not np.any(tp.token_bits(*_slot(pt, pos))), f"seq {sid}: target position {pos} not cleared"
        for pos in range(n[sid] + 1, ln_d):
            assert not np.any(dp.token_bits(*_slot(pd, pos))), f"seq {sid}: draft position {pos} not cleared"
    # rollback of the second sequence by 6 positions
    sid = ids[1]
    info = gpu.seq_info(sid)
    assert (info["target_len"], info["draft_len"]) == (n[sid] + 1, n[sid] + 1)
    new_len = info["target_len"] - 6
    pt, pd = info["pages_target"], info["pages_draft"]
    say("kv clear", which, ": rollback to", new_len)
    gpu.rollback(sid, new_len)
    torch.cuda.synchronize()
    tp = _Pool(gpu.kv_target, cfg.target, Lt, npages)
    dp = _Pool(gpu.kv_draft, cfg.draft, Ld, npages)
    assert np.any(tp.token_bits(*_slot(pt, new_len - 1)) != 0)
    assert np.any(dp.token_bits(*_slot(pd, new_len - 1)) != 0)
    for pos in range(new_len, info["target_len"]):
        assert not np.any(tp.token_bits(*_slot(pt, pos))), f"target position {pos} not cleared by rollback"
        assert not np.any(dp.token_bits(*_slot(pd, pos))), f"draft position {pos} not cleared by rollback"
    gpu.close()
