"""The speculative sampling rule, in float64.

CacheSpec (Section 3.4 and the speculative-decoding paragraph of Section 2)
uses the draft-and-verify scheme of Leviathan et al. 2023 / Chen et al. 2023
without restating it.  Written out, for a sequence whose last committed token
x_n sits at position n, drafts x~_1..x~_k (x~_j at position n+j, drawn from the
draft distribution q_j) and target distributions p_1..p_{k+1} (p_j scores
position n+j, from the target row fed the token at position n+j-1):

1. p_j = softmax(zp_j / T), q_j = softmax(zq_j / T), the same T for both models.
2. For j = 1..k: draw u_j ~ U(0,1); accept x~_j iff u_j * q_j(x~_j) < p_j(x~_j)
   (that is, with probability min(1, p_j/q_j)).  At the first rejection emit
   x~_1..x~_{j-1} and one token t ~ norm(max(0, p_j - q_j)), and stop.
3. If all k drafts are accepted, emit them and a bonus token t ~ p_{k+1}.
4. T = 0 (greedy): draft x~_j = argmax zq_j; accept iff x~_j = argmax zp_j; on
   rejection emit argmax zp_j; the bonus is argmax zp_{k+1}.  Ties go to the
   lowest token id.

Readings where the paper is silent (each is listed with its reason in the
design notes): categorical draws use the Gumbel-max trick with per-token
Philox noise keyed by (seed, seq, position, purpose); u_j uses the ACCEPT
stream at position n+j, the residual draw the RESAMPLE stream at n+j, the
bonus draw the BONUS stream at n+k+1 and the draft draw the DRAFT stream at
n+j; if the residual has no mass the draw falls back to p_j.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import philox
from .philox import ACCEPT, BONUS, DRAFT, RESAMPLE


def softmax_t(z: np.ndarray, T: float) -> np.ndarray:
    """softmax(z / T) in float64."""
    s = np.asarray(z, dtype=np.float64) / float(T)
    e = np.exp(s - s.max())
    return e / e.sum()


def residual(p: np.ndarray, q: np.ndarray) -> np.ndarray:
    """norm(max(0, p - q)); falls back to p when the residual has no mass."""
    r = np.maximum(p - q, 0.0)
    tot = r.sum()
    if tot <= 0.0:
        return p.copy()
    return r / tot


def argmax_first(x: np.ndarray) -> int:
    """Index of the maximum, lowest index on ties."""
    return int(np.argmax(x))


def gumbel_argmax(w: np.ndarray, G: np.ndarray) -> int:
    """Gumbel-max draw from the (unnormalised) weights ``w`` >= 0: argmax of
    log w_i + G_i; zero-weight tokens score -inf and are never chosen."""
    with np.errstate(divide="ignore"):
        s = np.log(w) + G
    return argmax_first(s)


# --------------------------------------------------------------------------
# decision margins (which decisions an fp32 implementation may legitimately flip)
# --------------------------------------------------------------------------

@dataclass
class Margins:
    """Exclusion rules for comparing an fp32 implementation with this oracle.

    accept:   an acceptance decision is excluded when |u - min(1, p/q)| < accept.
    rel:      relative error budget of the other side's probabilities; a
              categorical draw is excluded unless its winner beats every other
              token under every perturbation within that budget.
    gumbel:   absolute error budget of the other side's Gumbel noise.
    greedy:   an argmax is excluded when its top-2 logit gap is below this.
    """

    accept: float = 1e-4
    rel: float = 1e-4
    gumbel: float = 1e-5
    greedy: float = 0.0


def _draw_is_robust(w_hi: np.ndarray, w_lo: np.ndarray, G: np.ndarray, win: int, m: Margins) -> bool:
    with np.errstate(divide="ignore"):
        hi = np.log(w_hi) + G + m.gumbel
        lo_w = np.log(w_lo[win]) + G[win] - m.gumbel if w_lo[win] > 0 else -np.inf
    hi[win] = -np.inf
    return bool(lo_w > hi.max())


def draw_categorical(p: np.ndarray, G: np.ndarray, m: Margins) -> Tuple[int, bool]:
    """Gumbel-max draw from distribution p; returns (token, excluded)."""
    t = gumbel_argmax(p, G)
    ok = _draw_is_robust(p * (1 + m.rel), p * (1 - m.rel), G, t, m)
    return t, not ok


def draw_residual(p: np.ndarray, q: np.ndarray, G: np.ndarray, m: Margins) -> Tuple[int, bool]:
    """Gumbel-max draw from norm(max(0, p - q)); returns (token, excluded)."""
    r = np.maximum(p - q, 0.0)
    if r.sum() <= 0.0:
        return draw_categorical(p, G, m)
    t = gumbel_argmax(r, G)
    err = m.rel * (p + q)
    ok = _draw_is_robust(r + err, np.maximum(r - err, 0.0), G, t, m)
    return t, not ok


def greedy_pick(z: np.ndarray, m: Margins) -> Tuple[int, bool]:
    t = argmax_first(z)
    if m.greedy <= 0.0 or z.shape[0] < 2:
        return t, False
    rest = np.delete(np.asarray(z, dtype=np.float64), t)
    return t, bool(z[t] - rest.max() < m.greedy)


# --------------------------------------------------------------------------
# draft sampling and the verify rule
# --------------------------------------------------------------------------

def sample_draft(zq: np.ndarray, T: float, seed: int, seq: int, pos: int,
                 m: Margins = Margins()) -> Tuple[int, bool]:
    """Draft token at absolute position ``pos`` from draft logits zq."""
    if T == 0.0:
        return greedy_pick(zq, m)
    q = softmax_t(zq, T)
    return draw_categorical(q, philox.gumbel(seed, seq, pos, DRAFT, q.shape[0]), m)


@dataclass
class VerifyResult:
    n_accepted: int
    tokens: List[int]                 # x~_1..x~_a, t  (a + 1 tokens)
    excluded: bool = False            # some decision on the path was within its margin
    first_excluded: Optional[int] = None   # index into tokens of the first unsafe decision
    accept_margins: List[float] = field(default_factory=list)


def verify(zp: np.ndarray, zq: np.ndarray, drafts: Sequence[int], T: float,
           seed: int, seq: int, n: int, m: Margins = Margins()) -> VerifyResult:
    """Apply the rule to target logits zp [k+1, V], draft logits zq [k, V] and
    drafts x~_1..x~_k of a sequence whose pending token is at position n."""
    k = len(drafts)
    assert zp.shape[0] == k + 1 and (k == 0 or zq.shape[0] == k)
    V = zp.shape[1]
    res = VerifyResult(0, [])

    def mark(idx: int, bad: bool):
        if bad and not res.excluded:
            res.excluded = True
            res.first_excluded = idx

    if T == 0.0:
        for j in range(1, k + 1):
            t, bad = greedy_pick(zp[j - 1], m)
            mark(j - 1, bad)
            if drafts[j - 1] != t:
                res.n_accepted = j - 1
                res.tokens = [int(x) for x in drafts[:j - 1]] + [t]
                return res
        t, bad = greedy_pick(zp[k], m)
        mark(k, bad)
        res.n_accepted = k
        res.tokens = [int(x) for x in drafts] + [t]
        return res

    for j in range(1, k + 1):
        x = int(drafts[j - 1])
        p = softmax_t(zp[j - 1], T)
        q = softmax_t(zq[j - 1], T)
        u = philox.uniform(seed, seq, n + j, ACCEPT)
        ratio = 1.0 if q[x] <= 0.0 else min(1.0, p[x] / q[x])
        res.accept_margins.append(abs(u - ratio))
        mark(j - 1, abs(u - ratio) < m.accept)
        if u * q[x] < p[x]:
            continue
        t, bad = draw_residual(p, q, philox.gumbel(seed, seq, n + j, RESAMPLE, V), m)
        mark(j - 1, bad)
        res.n_accepted = j - 1
        res.tokens = [int(v) for v in drafts[:j - 1]] + [t]
        return res
    p = softmax_t(zp[k], T)
    t, bad = draw_categorical(p, philox.gumbel(seed, seq, n + k + 1, BONUS, V), m)
    mark(k, bad)
    res.n_accepted = k
    res.tokens = [int(v) for v in drafts] + [t]
    return res


def outcome_law(p_rows: Sequence[np.ndarray], q_rows: Sequence[np.ndarray],
                drafts: Sequence[int]) -> dict:
    """Exact law of the emitted tokens of one verify step for fixed drafts:
    {tuple(tokens): probability}, with p_rows the k+1 target distributions and
    q_rows the k draft distributions (already normalised)."""
    k = len(drafts)
    law = {}
    reach = 1.0
    for j in range(1, k + 1):
        x = int(drafts[j - 1])
        p, q = p_rows[j - 1], q_rows[j - 1]
        acc = 1.0 if q[x] <= 0.0 else min(1.0, p[x] / q[x])
        rej = reach * (1.0 - acc)
        if rej > 0.0:
            r = residual(p, q)
            prefix = tuple(int(v) for v in drafts[:j - 1])
            for t in np.nonzero(r)[0]:
                key = prefix + (int(t),)
                law[key] = law.get(key, 0.0) + rej * r[t]
        reach *= acc
    if reach > 0.0:
        p = p_rows[k]
        prefix = tuple(int(v) for v in drafts)
        for t in np.nonzero(p)[0]:
            key = prefix + (int(t),)
            law[key] = law.get(key, 0.0) + reach * p[t]
    return law


def acceptance_rate(p: np.ndarray, q: np.ndarray) -> float:
    """P(accept) of one draft position when x~ ~ q: sum_i min(p_i, q_i)."""
    return float(np.minimum(p, q).sum())
