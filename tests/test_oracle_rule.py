"""Pins of the oracle's speculative sampling rule against what the method fixes:

* the emitted tokens follow the target's joint law exactly (brute force, 1e-9);
* greedy speculative decoding reproduces greedy target decoding token for token;
* a drafter identical to the target is always accepted;
* per-position acceptance probability is sum_i min(p_i, q_i) (Monte Carlo);
* the accepted-length law is the product of per-position acceptance rates;
* the Gumbel-max sampler draws from its normalised weights, never a zero weight.
"""

import numpy as np
import pytest

from oracle import brute, philox, rule
from oracle.decoder import Decoder
from oracle.session import Session
from workloads import ModelShape, model_weights


@pytest.mark.parametrize("V,k,N,sparsity,seed", [
    (16, 2, 2, 0.0, 1),
    (8, 3, 3, 0.0, 2),
    (8, 4, 2, 0.0, 3),
    (6, 2, 3, 0.4, 4),     # zero-probability entries on both sides
    (16, 1, 2, 0.5, 5),
])
def test_brute_force_marginal_tables(V, k, N, sparsity, seed):
    tgt = brute.table_model(seed, V, N, sparsity)
    drf = brute.table_model(seed + 1000, V, N + k, sparsity)
    spec = brute.speculative_law(tgt, drf, k, N, V)
    ref = brute.target_law(tgt, N, V)
    assert abs(sum(spec.values()) - 1.0) < 1e-12
    assert brute.max_abs_diff(spec, ref) < 1e-9


def _tiny_pair(V=8):
    t = ModelShape("brute-target", 2, 16, 2, 1, 8, 24, V, 1e4, dtype="f32", init_std=0.5)
    d = ModelShape("brute-draft", 1, 16, 2, 2, 8, 24, V, 1e4, dtype="f32", init_std=0.5)
    return Decoder(t, model_weights(t, 21)), Decoder(d, model_weights(d, 22))


@pytest.mark.parametrize("T", [1.0, 0.6])
def test_brute_force_marginal_decoders(T):
    tdec, ddec = _tiny_pair(8)
    ctx = [1, 5, 2]
    tgt = brute.decoder_model(tdec, ctx, T)
    drf = brute.decoder_model(ddec, ctx, T)
    spec = brute.speculative_law(tgt, drf, 2, 3, 8)
    ref = brute.target_law(tgt, 3, 8)
    assert brute.max_abs_diff(spec, ref) < 1e-9


def test_outcome_law_detects_planted_mistakes():
    """The brute-force check is sharp: a residual without the max(0, .) clamp or
    an acceptance test on the wrong ratio breaks the marginal."""
    V, k, N = 6, 2, 2
    tgt = brute.table_model(9, V, N)
    drf = brute.table_model(10, V, N + k)
    ref = brute.target_law(tgt, N, V)
    good = brute.speculative_law(tgt, drf, k, N, V)
    assert brute.max_abs_diff(good, ref) < 1e-9
    orig = rule.residual
    try:
        def no_clamp(p, q):
            r = np.abs(p - q)
            return r / r.sum()
        rule.residual = no_clamp
        bad = brute.speculative_law(tgt, drf, k, N, V)
    finally:
        rule.residual = orig
    assert brute.max_abs_diff(bad, ref) > 1e-3


def test_verify_sampler_matches_outcome_law():
    """Monte Carlo over Philox seeds of ``rule.verify`` against the exact law."""
    g = np.random.default_rng(3)
    V, k = 5, 3
    zp = g.standard_normal((k + 1, V)) * 1.5
    zq = zp[:k] + g.standard_normal((k, V))
    drafts = [1, 3, 0]
    T = 1.0
    law = rule.outcome_law([rule.softmax_t(z, T) for z in zp], [rule.softmax_t(z, T) for z in zq], drafts)
    counts = {}
    n = 6000
    for s in range(n):
        r = rule.verify(zp, zq, drafts, T, seed=s, seq=77, n=100)
        key = tuple(r.tokens)
        counts[key] = counts.get(key, 0) + 1
    assert set(counts) <= set(law)
    chi2 = 0.0
    dof = 0
    for key, pr in law.items():
        e = n * pr
        if e < 5:
            continue
        chi2 += (counts.get(key, 0) - e) ** 2 / e
        dof += 1
    assert chi2 < dof + 5 * np.sqrt(2 * dof)


def test_greedy_speculation_equals_greedy_target():
    """Greedy draft-and-verify emits exactly the target's greedy continuation."""
    t = ModelShape("g-target", 2, 32, 4, 2, 8, 48, 50, 1e4, dtype="f32", init_std=0.3)
    d = ModelShape("g-draft", 1, 32, 4, 4, 8, 48, 50, 1e4, dtype="f32", init_std=0.3)
    tdec, ddec = Decoder(t, model_weights(t, 31)), Decoder(d, model_weights(d, 32))
    prompt = [3, 14, 15, 9, 2, 6]
    sess = Session(tdec, ddec, 64, 64, page_size=4)
    sess.prefill([9], [prompt])
    emitted = []
    accepted = []
    while len(emitted) < 24:
        for _ in range(3):
            sess.draft_step([9], [0.0], seed=1)
        (res, _), = sess.verify([9], [0.0], seed=1)
        sess.commit([9], [res])
        emitted += res.tokens
        accepted.append(res.n_accepted)
    # reference: plain greedy decoding with the target, one token at a time
    seq = list(prompt)
    for _ in range(len(emitted)):
        seq.append(int(np.argmax(tdec.full_logits(seq)[-1])))
    assert emitted == seq[len(prompt):]
    assert sess.lengths(9)[0] == len(prompt) + len(emitted) - 1


def test_identical_draft_always_accepted():
    sh = ModelShape("same", 2, 32, 4, 2, 8, 48, 40, 1e4, dtype="f32", init_std=0.3)
    w = model_weights(sh, 41)
    sess = Session(Decoder(sh, w), Decoder(sh, w), 64, 64, page_size=4)
    sess.prefill([5], [[1, 2, 3]])
    for step in range(4):
        for _ in range(3):
            sess.draft_step([5], [0.9], seed=step)
        (res, _), = sess.verify([5], [0.9], seed=step)
        assert res.n_accepted == 3
        sess.commit([5], [res])
    assert sess.lengths(5) == (3 + 4 * 4 - 1, 3 + 4 * 4 - 2)


def test_acceptance_rate_and_length_law():
    """P(accept_j) = sum_i min(p_i, q_i) and P(a >= j) = prod_{i<=j} alpha_i when
    drafts are drawn from q (vocab-stress style rows, small V)."""
    g = np.random.default_rng(8)
    V, k, T = 300, 3, 1.0
    zp = g.standard_normal((k + 1, V)) * 3
    zq = zp[:k] + g.standard_normal((k, V))
    alpha = [rule.acceptance_rate(rule.softmax_t(zp[j], T), rule.softmax_t(zq[j], T)) for j in range(k)]
    n = 4000
    ge = np.zeros(k + 1)
    for s in range(n):
        drafts = [rule.sample_draft(zq[j], T, s, 3, 50 + j + 1)[0] for j in range(k)]
        a = rule.verify(zp, zq, drafts, T, s, 3, 50).n_accepted
        ge[:a + 1] += 1
    for j in range(1, k + 1):
        pj = np.prod(alpha[:j])
        est = ge[j] / n
        assert abs(est - pj) < 4 * np.sqrt(pj * (1 - pj) / n) + 1e-3


def test_gumbel_sampler_chi2_and_zero_weights():
    w = np.array([0.0, 0.1, 0.0, 0.3, 0.05, 0.55, 0.0])
    counts = np.zeros(len(w))
    n = 20000
    for pos in range(n):
        counts[rule.gumbel_argmax(w, philox.gumbel(17, 4, pos, philox.RESAMPLE, len(w)))] += 1
    assert counts[w == 0].sum() == 0
    e = n * w[w > 0]
    chi2 = ((counts[w > 0] - e) ** 2 / e).sum()
    assert chi2 < 20  # 3 dof


def test_emitted_token_at_rejection_follows_target():
    """First emitted token of a step is distributed as p_1, whatever the drafter."""
    g = np.random.default_rng(12)
    V, T = 7, 0.8
    zp = g.standard_normal((2, V))
    zq = g.standard_normal((1, V)) * 2
    p1 = rule.softmax_t(zp[0], T)
    counts = np.zeros(V)
    n = 20000
    for s in range(n):
        d = rule.sample_draft(zq[0], T, s, 1, 11)[0]
        counts[rule.verify(zp, zq, [d], T, s, 1, 10).tokens[0]] += 1
    e = n * p1
    assert ((counts - e) ** 2 / e).sum() < 6 + 5 * np.sqrt(12)


def test_margins_flag_near_ties():
    V = 10
    G = np.zeros(V)
    p = np.full(V, 0.05)
    p[3] = 0.275
    p[7] = 0.275 * (1 + 1e-6)
    t, bad = rule.draw_categorical(p / p.sum(), G, rule.Margins())
    assert t == 7 and bad
    p[7] = 0.4
    t, bad = rule.draw_categorical(p / p.sum(), G, rule.Margins())
    assert t == 7 and not bad
    z = np.zeros(5)
    z[2], z[4] = 1.0, 1.0 - 1e-7
    assert rule.greedy_pick(z, rule.Margins(greedy=1e-5)) == (2, True)
    assert rule.greedy_pick(z, rule.Margins()) == (2, False)
