"""Brute-force output law of repeated draft-and-verify steps on tiny vocabularies.

The guarantee of speculative sampling (Leviathan et al. 2023, Theorem 1; the
method CacheSpec's drafter relies on in Section 3.4) is that the emitted tokens
follow exactly the target's autoregressive distribution, whatever the drafter.
This module enumerates every draft string (weight = product of draft
probabilities) and every verify outcome (``rule.outcome_law``), step after step
until N tokens have been emitted, and returns the joint law of the first N
emitted tokens.  Comparing it with the target's own joint law pins the rule.
"""

from __future__ import annotations

import itertools
from typing import Callable, Dict, Tuple

import numpy as np

from . import rule, tree

Dist = Callable[[Tuple[int, ...]], np.ndarray]


def speculative_law(target: Dist, draft: Dist, k: int, N: int, V: int) -> Dict[Tuple[int, ...], float]:
    """Joint law of the first N tokens emitted by draft-and-verify with k drafts."""
    final: Dict[Tuple[int, ...], float] = {}
    frontier: Dict[Tuple[int, ...], float] = {(): 1.0}
    while frontier:
        nxt: Dict[Tuple[int, ...], float] = {}
        for prefix, w in frontier.items():
            for d in itertools.product(range(V), repeat=k):
                pr = w
                qs = []
                for j in range(k):
                    q = draft(prefix + d[:j])
                    qs.append(q)
                    pr *= q[d[j]]
                    if pr == 0.0:
                        break
                if pr == 0.0:
                    continue
                ps = [target(prefix + d[:j]) for j in range(k + 1)]
                for toks, pt in rule.outcome_law(ps, qs, d).items():
                    full = prefix + toks
                    if len(full) >= N:
                        key = full[:N]
                        final[key] = final.get(key, 0.0) + pr * pt
                    else:
                        nxt[full] = nxt.get(full, 0.0) + pr * pt
        frontier = nxt
    return final


def tree_shape(branching) -> list:
    """Parents of a tree with branching[l] children under every node of depth
    l (the root has depth 0), nodes numbered level by level."""
    parents, level = [], [-1]
    for b in branching:
        nxt = []
        for u in level:
            for _ in range(b):
                parents.append(u)
                nxt.append(len(parents) - 1)
        level = nxt
    return parents


def tree_law(target: Dist, draft: Dist, branching, N: int, V: int) -> Dict[Tuple[int, ...], float]:
    """Joint law of the first N tokens emitted by tree verification, every
    node's children drawn independently from the draft distribution after the
    node's path (``tree.outcome_law_tree`` for each drawn tree)."""
    parents = tree_shape(branching)
    m = len(parents)

    def path(i, toks):
        out = []
        while i >= 0:
            out.append(toks[i])
            i = parents[i]
        return tuple(reversed(out))

    final: Dict[Tuple[int, ...], float] = {}
    frontier: Dict[Tuple[int, ...], float] = {(): 1.0}
    while frontier:
        nxt: Dict[Tuple[int, ...], float] = {}
        for prefix, w in frontier.items():
            for toks in itertools.product(range(V), repeat=m):
                pr = w
                for i in range(m):
                    u = parents[i]
                    pr *= draft(prefix + (path(u, toks) if u >= 0 else ()))[toks[i]]
                    if pr == 0.0:
                        break
                if pr == 0.0:
                    continue
                ps = [target(prefix)] + [target(prefix + path(i, toks)) for i in range(m)]
                qs = [draft(prefix)] + [draft(prefix + path(i, toks)) for i in range(m)]
                for out, pt in tree.outcome_law_tree(ps, qs, parents, toks).items():
                    full = prefix + out
                    if len(full) >= N:
                        key = full[:N]
                        final[key] = final.get(key, 0.0) + pr * pt
                    else:
                        nxt[full] = nxt.get(full, 0.0) + pr * pt
        frontier = nxt
    return final


def target_law(target: Dist, N: int, V: int) -> Dict[Tuple[int, ...], float]:
    """Autoregressive joint law of N tokens under the target."""
    law = {}
    for s in itertools.product(range(V), repeat=N):
        pr = 1.0
        for i in range(N):
            pr *= target(s[:i])[s[i]]
            if pr == 0.0:
                break
        if pr > 0.0:
            law[s] = pr
    return law


def max_abs_diff(a: Dict, b: Dict) -> float:
    keys = set(a) | set(b)
    return max(abs(a.get(x, 0.0) - b.get(x, 0.0)) for x in keys)


def table_model(seed: int, V: int, depth: int, sparsity: float = 0.0) -> Dist:
    """An arbitrary conditional table prefix -> distribution over V (random
    Dirichlet rows, some entries zeroed with probability ``sparsity``),
    memoised per prefix.  Test input only."""
    g = np.random.default_rng(seed)
    cache: Dict[Tuple[int, ...], np.ndarray] = {}

    def dist(prefix: Tuple[int, ...]) -> np.ndarray:
        if prefix not in cache:
            p = g.dirichlet(np.full(V, 0.7))
            if sparsity > 0.0:
                keep = g.random(V) >= sparsity
                keep[g.integers(V)] = True
                p = np.where(keep, p, 0.0)
                p = p / p.sum()
            cache[prefix] = p
        return cache[prefix]

    return dist


def decoder_model(dec, context, T: float) -> Dist:
    """prefix -> softmax(z/T) of a decoder's next-token logits after context+prefix."""
    cache: Dict[Tuple[int, ...], np.ndarray] = {}

    def dist(prefix: Tuple[int, ...]) -> np.ndarray:
        if prefix not in cache:
            z = dec.full_logits(list(context) + list(prefix))[-1]
            cache[prefix] = rule.softmax_t(z, T)
        return cache[prefix]

    return dist
