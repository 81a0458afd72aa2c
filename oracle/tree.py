"""Tree (multi-candidate) verification, in float64.

Test infrastructure: a plain CPU statement of what the GPU path computes; the
product path never imports it.

Section 2 of the paper lists tree-structured and multi-candidate
verification (SpecInfer, Medusa, EAGLE) among the variants of speculative
decoding; the exact rule for a tree of sampled candidates is SpecInfer's
multi-step speculative sampling (Miao et al. 2024), the chain rule of
Leviathan et al. / Chen et al. applied to one candidate after another with
the target distribution replaced by the residual after each rejection.

A draft tree of m nodes hangs below the pending token x_n (the root, depth
0).  Node i carries token x_i, its parent parents[i] (-1 for the root, else
a node with a smaller index) and depth d_i = depth of its parent + 1, so x_i
would sit at position n + d_i.  Siblings are ordered by index.  Every node
u's children were drawn independently from one draft distribution q_u =
softmax(zq_u / T); the target scores node u with p_u = softmax(zp_u / T)
(the distribution of the token after u's path).

Rule, from the root:
1. at node u of depth d, let r = p_u;
2. for each child c of u in order (candidate number j = 0, 1, ...): accept
   x_c iff v_j * q_u(x_c) < r(x_c), v_j = U(seed, seq, n + d + 1, ACCEPT,
   block j); if accepted emit x_c and continue at c (step 1); otherwise
   replace r by norm(max(0, r - q_u)) (kept as is if that has no mass);
3. if u has children and all are rejected, emit t ~ r (Gumbel-max with
   RESAMPLE noise at n + d + 1) and stop; if u has no children, emit
   t ~ p_u (BONUS noise at n + d + 1) and stop.
Greedy (T = 0): accept the first child whose token is argmax zp_u (lowest id
on ties), else emit argmax zp_u.

A chain (parents[i] = i - 1) is the chain rule exactly: one candidate per
position uses block 0, the scalar draw of the chain rule.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import philox, rule
from .philox import ACCEPT, BONUS, RESAMPLE


def children_of(parents: Sequence[int], u: int) -> List[int]:
    """Children (node indices, in order) of node u (-1: the root)."""
    return [i for i, p in enumerate(parents) if int(p) == u]


def depths(parents: Sequence[int]) -> List[int]:
    d = []
    for i, p in enumerate(parents):
        assert -1 <= int(p) < i, "parents must precede their children"
        d.append(1 if p < 0 else d[p] + 1)
    return d


def residual_step(r: np.ndarray, q: np.ndarray) -> np.ndarray:
    """norm(max(0, r - q)), or r if that has no mass."""
    w = np.maximum(r - q, 0.0)
    s = w.sum()
    return w / s if s > 0.0 else r


@dataclass
class TreeResult:
    n_accepted: int                   # depth of the last accepted node (0: none)
    tokens: List[int]                 # the accepted path's tokens, then t
    path: List[int] = field(default_factory=list)   # accepted node indices, root to leaf
    excluded: bool = False
    first_excluded: Optional[int] = None


def verify_tree(zp: np.ndarray, zq: np.ndarray, parents: Sequence[int], tokens: Sequence[int], T: float,
                seed: int, seq: int, n: int, m: rule.Margins = rule.Margins()) -> TreeResult:
    """zp [m+1, V]: row 0 the root's target logits, row i+1 node i's;
    zq [m+1, V]: row 0 the draft logits the root's children were drawn from,
    row i+1 those of node i's children (rows of leaves are not read)."""
    mm = len(parents)
    assert zp.shape[0] == mm + 1 and len(tokens) == mm
    depths(parents)
    V = zp.shape[1]
    res = TreeResult(0, [])

    def mark(bad: bool):
        if bad and not res.excluded:
            res.excluded = True
            res.first_excluded = len(res.tokens)

    u, d = -1, 0
    while True:
        kids = children_of(parents, u)
        row = u + 1
        if T == 0.0:
            t, bad = rule.greedy_pick(zp[row], m)
            mark(bad)
            nxt = next((c for c in kids if int(tokens[c]) == t), None)
            if nxt is None:
                res.tokens.append(t)
                return res
            res.tokens.append(t)
            res.path.append(nxt)
            u, d = nxt, d + 1
            res.n_accepted = d
            continue
        r = rule.softmax_t(zp[row], T)
        if not kids:
            t, bad = rule.draw_categorical(r, philox.gumbel(seed, seq, n + d + 1, BONUS, V), m)
            mark(bad)
            res.tokens.append(t)
            return res
        q = rule.softmax_t(zq[row], T)
        accepted = None
        for j, c in enumerate(kids):
            x = int(tokens[c])
            v = philox.uniform_block(seed, seq, n + d + 1, ACCEPT, j)
            ratio = 1.0 if q[x] <= 0.0 else min(1.0, r[x] / q[x])
            mark(abs(v - ratio) < m.accept)
            if v * q[x] < r[x]:
                accepted = c
                break
            r = residual_step(r, q)
        if accepted is None:
            t, bad = rule.draw_categorical(r, philox.gumbel(seed, seq, n + d + 1, RESAMPLE, V), m)
            mark(bad)
            res.tokens.append(t)
            return res
        res.tokens.append(int(tokens[accepted]))
        res.path.append(accepted)
        u, d = accepted, d + 1
        res.n_accepted = d


def outcome_law_tree(p_rows: Sequence[np.ndarray], q_rows: Sequence[Optional[np.ndarray]],
                     parents: Sequence[int], tokens: Sequence[int]) -> Dict[Tuple[int, ...], float]:
    """Exact law of the emitted tokens of one tree verify for a fixed tree:
    {tuple(tokens): probability}; p_rows[u + 1] / q_rows[u + 1] are node u's
    normalised target / draft distributions (u = -1: the root)."""
    law: Dict[Tuple[int, ...], float] = {}

    def emit(prefix, prob, r):
        for t in np.nonzero(r)[0]:
            key = prefix + (int(t),)
            law[key] = law.get(key, 0.0) + prob * float(r[t])

    def walk(u, prefix, prob):
        kids = children_of(parents, u)
        r = p_rows[u + 1]
        if not kids:
            emit(prefix, prob, r)
            return
        q = q_rows[u + 1]
        for c in kids:
            x = int(tokens[c])
            acc = (1.0 if r[x] > 0.0 else 0.0) if q[x] <= 0.0 else min(1.0, r[x] / q[x])
            if acc > 0.0:
                walk(c, prefix + (x,), prob * acc)
            prob *= 1.0 - acc
            if prob == 0.0:
                return
            r = residual_step(r, q)
        emit(prefix, prob, r)

    walk(-1, (), 1.0)
    return law
