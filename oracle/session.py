"""End-to-end draft-and-verify on the float64 oracle decoders.

State of one sequence (the pending-token model):

* ``history`` holds every committed token x_0..x_n; the last one, x_n at
  position n, is *pending*: it is not yet in the target's KV cache, whose
  length is n.
* the draft cache has length len_d <= n; its pending tokens are
  history[len_d..n] (one token normally, two after a step that accepted all
  drafts).
* draft step j feeds the draft model its pending tokens (j = 1) or x~_{j-1}
  (j > 1) and draws x~_j at position n+j from the last row's logits.
* verify feeds the target x_n, x~_1..x~_k at positions n..n+k (their K/V are
  written first, then each row attends causally) and applies the rule.
* commit with a accepted: the a+1 emitted tokens join the history; the target
  cache keeps positions <= n+a (length n+a+1); the draft cache keeps
  min(len_d, n+a+1); rejected positions are dropped in place.

A prompt of P tokens is prefilled into both caches for positions 0..P-2, and
x_{P-1} is pending.

With no draft model (``draft=None``) the session decodes the target alone
(``decode``): each step is a verify of no drafts, whose one row's bonus draw is
the next token, and its commit.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

from .decoder import Decoder, KVList
from .paging import PagePool
from . import rule, tree


@dataclass
class SeqState:
    history: List[int]
    kv_t: KVList
    kv_d: Optional[KVList]
    drafts: List[int] = field(default_factory=list)
    zq: List[np.ndarray] = field(default_factory=list)
    draft_excluded: bool = False
    tree_parents: Optional[List[int]] = None   # drafts form a tree (set_draft_tree)

    @property
    def n(self) -> int:            # position of the pending token
        return len(self.history) - 1


class Session:
    def __init__(self, target: Decoder, draft: Optional[Decoder], num_pages_target: int,
                 num_pages_draft: int, page_size: int = 16):
        self.target = target
        self.draft = draft
        self.pool_t = PagePool(num_pages_target, page_size)
        self.pool_d = PagePool(num_pages_draft if draft is not None else 0, page_size)
        self.seqs: Dict[int, SeqState] = {}

    # ------------------------------------------------------------------
    def prefill(self, seq_ids: Sequence[int], prompts: Sequence[Sequence[int]]):
        for sid, prompt in zip(seq_ids, prompts):
            sid = int(sid)
            prompt = [int(t) for t in prompt]
            assert len(prompt) >= 1 and sid not in self.seqs
            st = SeqState(prompt, self.target.new_kv(), self.draft.new_kv() if self.draft else None)
            P = len(prompt)
            self.pool_t.ensure(sid, P - 1)
            if self.draft:
                self.pool_d.ensure(sid, P - 1)
            if P > 1:
                self.target.forward(st.kv_t, prompt[:-1], np.arange(P - 1), logits=False)
                if self.draft:
                    self.draft.forward(st.kv_d, prompt[:-1], np.arange(P - 1), logits=False)
            self.seqs[sid] = st

    def draft_step(self, seq_ids: Sequence[int], temps: Sequence[float], seed: int,
                   margins: rule.Margins = rule.Margins(), guide: Sequence[int] = None,
                   boost: float = 0.0) -> List[int]:
        """One draft token per sequence.  With guide[i] >= 0 the guide token's
        logit is first raised to the row maximum + boost (workload shaping: the
        raised row is the proposal q that the draw and the rule use)."""
        out = []
        for i, (sid, T) in enumerate(zip(seq_ids, temps)):
            st = self.seqs[int(sid)]
            if st.drafts:
                toks = [st.drafts[-1]]
            else:
                toks = st.history[st.kv_d.length:]
            start = st.kv_d.length
            self.pool_d.ensure(int(sid), start + len(toks))
            z = self.draft.forward(st.kv_d, toks, start + np.arange(len(toks)))[-1]
            if guide is not None and guide[i] >= 0:
                z = z.copy()
                z[int(guide[i])] = z.max() + boost
            pos = st.n + len(st.drafts) + 1
            x, bad = rule.sample_draft(z, float(T), seed, int(sid), pos, margins)
            st.drafts.append(x)
            st.zq.append(z)
            st.draft_excluded |= bad
            out.append(x)
        return out

    def draft_loop(self, seq_ids: Sequence[int], temps: Sequence[float], seed: int,
                   steps: Sequence[int], margins: rule.Margins = rule.Margins()):
        """steps[i] draft steps of sequence i as one call: the draft pages of
        all of a call's steps are taken first, sequence by sequence in list
        order, then the steps run (step j for every sequence that takes part
        in it, in list order), each exactly draft_step."""
        for sid, n_steps in zip(seq_ids, steps):
            if n_steps > 0:
                st = self.seqs[int(sid)]
                first = 1 if st.drafts else st.n + 1 - st.kv_d.length
                self.pool_d.ensure(int(sid), st.kv_d.length + first + n_steps - 1)
        for j in range(max(steps, default=0)):
            part = [(s, t) for s, t, n_s in zip(seq_ids, temps, steps) if n_s > j]
            self.draft_step([s for s, _ in part], [t for _, t in part], seed, margins)

    def set_drafts(self, sid: int, drafts: Sequence[int], zq: np.ndarray):
        """Install externally supplied drafts (tokens and their draft logits)."""
        st = self.seqs[int(sid)]
        st.drafts = [int(x) for x in drafts]
        st.zq = [np.asarray(r, dtype=np.float64) for r in zq]

    def set_draft_tree(self, sid: int, parents: Sequence[int], tokens: Sequence[int], zq: np.ndarray):
        """Install a draft tree: node i has token tokens[i] and parent
        parents[i] (-1: the pending token); zq [m+1, V] holds the draft logits
        each node's children were drawn from (row 0: the root's)."""
        st = self.seqs[int(sid)]
        tree.depths(parents)
        st.drafts = [int(x) for x in tokens]
        st.zq = [np.asarray(r, dtype=np.float64) for r in zq]
        st.tree_parents = [int(p) for p in parents]

    def _verify_tree(self, sid: int, st: SeqState, T: float, seed: int, margins: rule.Margins):
        """Target logits of every tree node by the plain causal forward over the
        node's path (the root row first), then the tree rule; the cache then
        holds the pending token and the accepted path."""
        n, parents = st.n, st.tree_parents

        def copy(kv):
            return KVList(kv.n_layers, [None if x is None else x.copy() for x in kv.K],
                          [None if x is None else x.copy() for x in kv.V])

        def path_tokens(i):
            out = []
            while i >= 0:
                out.append(st.drafts[i])
                i = parents[i]
            return out[::-1]

        root_kv = copy(st.kv_t)
        rows = [self.target.forward(root_kv, [st.history[-1]], [n])[0]]
        for i in range(len(parents)):
            pt = path_tokens(i)
            rows.append(self.target.forward(copy(root_kv), pt, n + 1 + np.arange(len(pt)))[-1])
        zp = np.stack(rows)
        res = tree.verify_tree(zp, np.stack(st.zq), parents, st.drafts, T, seed, sid, n, margins)
        acc = [st.drafts[i] for i in res.path]
        if acc:
            self.target.forward(root_kv, acc, n + 1 + np.arange(len(acc)), logits=False)
        st.kv_t = root_kv
        return res, zp

    def verify(self, seq_ids: Sequence[int], temps: Sequence[float], seed: int,
               margins: rule.Margins = rule.Margins()):
        """Returns a list of (VerifyResult or TreeResult, target logits [k+1, V])."""
        out = []
        for sid, T in zip(seq_ids, temps):
            sid = int(sid)
            st = self.seqs[sid]
            n, k = st.n, len(st.drafts)
            self.pool_t.ensure(sid, n + k + 1)
            if st.tree_parents is not None:
                out.append(self._verify_tree(sid, st, float(T), seed, margins))
                continue
            rows = [st.history[-1]] + st.drafts
            zp = self.target.forward(st.kv_t, rows, n + np.arange(k + 1))
            zq = np.stack(st.zq) if k else np.zeros((0, zp.shape[1]))
            res = rule.verify(zp, zq, st.drafts, float(T), seed, sid, n, margins)
            if st.draft_excluded:
                res.excluded = True
                res.first_excluded = 0 if res.first_excluded is None else res.first_excluded
            out.append((res, zp))
        return out

    def undo_verify(self, seq_ids: Sequence[int]):
        """Take back the last verify of the listed sequences: drop the K/V it
        wrote (positions n..n+k) and the target pages that only it needed, so
        that the cache and the page pool are as before the verify.  The drafts
        stay."""
        for sid in seq_ids:
            sid = int(sid)
            st = self.seqs[sid]
            st.kv_t.truncate(st.n)
            self.pool_t.truncate(sid, st.n)

    def commit(self, seq_ids: Sequence[int], results: Sequence[rule.VerifyResult]):
        for sid, res in zip(seq_ids, results):
            sid = int(sid)
            st = self.seqs[sid]
            n, a = st.n, res.n_accepted
            st.history.extend(res.tokens)
            new_t = n + a + 1
            st.kv_t.truncate(new_t)
            self.pool_t.truncate(sid, new_t)
            if st.kv_d is not None:
                new_d = min(st.kv_d.length, new_t)
                st.kv_d.truncate(new_d)
                self.pool_d.truncate(sid, new_d)
            st.drafts, st.zq, st.draft_excluded, st.tree_parents = [], [], False, None

    def rollback(self, sid: int, new_len: int):
        """Truncate both caches to ``new_len`` positions; history[new_len] becomes
        the pending token.  Outstanding drafts are dropped."""
        st = self.seqs[int(sid)]
        assert 0 <= new_len <= st.kv_t.length
        del st.history[new_len + 1:]
        st.kv_t.truncate(new_len)
        self.pool_t.truncate(int(sid), new_len)
        if st.kv_d is not None:
            st.kv_d.truncate(min(st.kv_d.length, new_len))
            self.pool_d.truncate(int(sid), st.kv_d.length)
        st.drafts, st.zq, st.draft_excluded, st.tree_parents = [], [], False, None

    def decode(self, seq_ids: Sequence[int], temps: Sequence[float], seed: int, steps: int,
               margins: rule.Margins = rule.Margins()):
        """Plain decoding of the target: ``steps`` tokens per sequence, each a
        verify with no drafts (the bonus draw from p at position n + 1, or its
        argmax for T = 0) and its commit, step by step over the list.  Returns
        (tokens [n][steps], excluded [n][steps], logits [steps] of [n, V])."""
        toks = [[] for _ in seq_ids]
        excl = [[] for _ in seq_ids]
        logits = []
        for _ in range(steps):
            for sid in seq_ids:
                assert not self.seqs[int(sid)].drafts, "decode needs sequences with no drafts"
            out = self.verify(seq_ids, temps, seed, margins)
            self.commit(seq_ids, [r for r, _ in out])
            for i, (r, _) in enumerate(out):
                toks[i].append(r.tokens[0])
                excl[i].append(bool(r.excluded))
            logits.append(np.stack([z[0] for _, z in out]))
        return toks, excl, logits

    def release(self, sid: int):
        self.pool_t.release(int(sid))
        self.pool_d.release(int(sid))
        del self.seqs[int(sid)]

    # ------------------------------------------------------------------
    def lengths(self, sid: int):
        st = self.seqs[int(sid)]
        return st.kv_t.length, (st.kv_d.length if st.kv_d is not None else 0)

    def pages(self, sid: int):
        return list(self.pool_t.tables.get(int(sid), [])), list(self.pool_d.tables.get(int(sid), []))
