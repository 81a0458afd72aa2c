"""Pins of the oracle's tree (multi-candidate) verification.

* exactness: with every node's children drawn independently from the draft
  distribution, the joint law of the first N emitted tokens equals the
  target's autoregressive law (enumerated on tiny vocabularies, 1e-12);
* the sampled rule follows its own exact outcome law (Monte Carlo, 4 sigma);
* a chain is the chain rule: bit-identical decisions and tokens;
* greedy follows the argmax path;
* the session's tree rows are the no-cache forward over each node's path, and
  the cache after commit holds the accepted path (the next verify's logits are
  the no-cache forward's).
"""

import numpy as np
import pytest

from oracle import brute, rule, tree
from oracle.decoder import Decoder
from oracle.session import Session
from workloads import TINY_FP32, model_weights, uniform_prompts


@pytest.mark.parametrize("V,branching,N,sparsity", [
    (3, [2], 2, 0.0), (3, [2, 2], 2, 0.0), (4, [3], 2, 0.3), (3, [2, 1], 3, 0.3), (2, [3, 2], 3, 0.0)])
def test_tree_law_equals_target_law(V, branching, N, sparsity):
    tg = brute.table_model(10 + V, V, 4, sparsity)
    dr = brute.table_model(20 + V, V, 4, sparsity)
    a = brute.tree_law(tg, dr, branching, N, V)
    b = brute.target_law(tg, N, V)
    assert abs(sum(a.values()) - 1.0) < 1e-12
    assert brute.max_abs_diff(a, b) < 1e-12


def test_tree_law_on_a_tiny_decoder_pair():
    shape = TINY_FP32.target.__class__("t", 1, 16, 2, 2, 8, 24, 4, 1e4, dtype="f32", init_std=0.5)
    dshape = shape.__class__("d", 1, 16, 2, 2, 8, 24, 4, 1e4, dtype="f32", init_std=0.5)
    tgt = brute.decoder_model(Decoder(shape, model_weights(shape, 3)), [1, 2], 1.0)
    drf = brute.decoder_model(Decoder(dshape, model_weights(dshape, 4)), [1, 2], 1.0)
    a = brute.tree_law(tgt, drf, [2, 2], 2, 4)
    b = brute.target_law(tgt, 2, 4)
    assert brute.max_abs_diff(a, b) < 1e-12


def test_sampled_tree_rule_follows_its_outcome_law():
    V, T = 6, 1.0
    g = np.random.default_rng(5)
    parents = brute.tree_shape([3, 2])
    m = len(parents)
    zp = g.standard_normal((m + 1, V)) * 1.5
    zq = zp + g.standard_normal((m + 1, V))
    qs = [rule.softmax_t(z, T) for z in zq]
    ps = [rule.softmax_t(z, T) for z in zp]
    # candidate tokens drawn from their parent's q (fixed for the test)
    toks = [int(g.choice(V, p=qs[p + 1])) for p in parents]
    law = tree.outcome_law_tree(ps, qs, parents, toks)
    n_draws = 6000
    counts = {}
    for s in range(n_draws):
        r = tree.verify_tree(zp, zq, parents, toks, T, seed=1000 + s, seq=7, n=50)
        counts[tuple(r.tokens)] = counts.get(tuple(r.tokens), 0) + 1
    assert set(counts) <= set(law)
    for key, p in law.items():
        f = counts.get(key, 0) / n_draws
        assert abs(f - p) <= 4 * np.sqrt(p * (1 - p) / n_draws) + 1e-3, (key, f, p)


@pytest.mark.parametrize("T", [0.0, 0.7, 1.0])
def test_chain_tree_is_the_chain_rule(T):
    V, k = 40, 4
    g = np.random.default_rng(9)
    same = 0
    for s in range(150):
        zp = g.standard_normal((k + 1, V)) * 2.0
        zq = zp[:k] + g.standard_normal((k, V)) * 0.7
        drafts = [int(np.argmax(z + g.gumbel(size=V))) for z in zq]
        a = rule.verify(zp, zq, drafts, T, 3, 11, 100 + s)
        zq_tree = np.concatenate([zq, np.zeros((1, V))])
        b = tree.verify_tree(zp, zq_tree, list(range(-1, k - 1)), drafts, T, 3, 11, 100 + s)
        assert (a.n_accepted, a.tokens, a.excluded) == (b.n_accepted, b.tokens, b.excluded)
        assert b.path == list(range(b.n_accepted))
        same += a.n_accepted > 0
    assert same > 10  # some drafts were accepted


def test_greedy_tree_follows_the_argmax_path():
    V = 8
    g = np.random.default_rng(2)
    parents = [-1, -1, 0, 0, 1, 3]
    zp = g.standard_normal((7, V))
    zq = g.standard_normal((7, V))
    top = [int(np.argmax(z)) for z in zp]
    # root's second child and node 0's second child carry the argmax tokens
    toks = [(top[0] + 1) % V, top[0], (top[1] + 1) % V, top[1], 0, top[4]]
    r = tree.verify_tree(zp, zq, parents, toks, 0.0, 1, 1, 10)
    # root -> node 1 (argmax of row 0); node 1's child is node 4 (token 0)
    if toks[4] == top[2]:
        assert r.path[:2] == [1, 4]
    else:
        assert r.path == [1] and r.tokens == [top[0], top[2]]


def test_session_tree_rows_and_committed_cache():
    shape = TINY_FP32.target
    w = model_weights(shape, 21)
    dec = Decoder(shape, w)
    sess = Session(dec, None, 64, 0)
    prompt = [int(x) for x in uniform_prompts(21, [30], shape.vocab)[0]]
    sess.prefill([4], [prompt])
    V = shape.vocab
    g = np.random.default_rng(21)
    parents = [-1, -1, 0, 1, 1, 3]
    toks = [int(x) for x in g.integers(0, V, size=6)]
    zq = g.standard_normal((7, V))
    sess.set_draft_tree(4, parents, toks, zq)
    ((res, zp),) = sess.verify([4], [1.0], 8)

    def path(i):
        out = []
        while i >= 0:
            out.append(toks[i])
            i = parents[i]
        return out[::-1]

    np.testing.assert_allclose(zp[0], dec.full_logits(prompt)[-1], atol=1e-12)
    for i in range(6):
        np.testing.assert_allclose(zp[i + 1], dec.full_logits(prompt + path(i))[-1], atol=1e-12)
    sess.commit([4], [res])
    hist = sess.seqs[4].history
    assert hist == prompt + res.tokens
    assert sess.lengths(4)[0] == len(hist) - 1
    # the next verify (no drafts) sees the committed path in the cache
    ((res2, zp2),) = sess.verify([4], [1.0], 9)
    np.testing.assert_allclose(zp2[0], dec.full_logits(hist)[-1], atol=1e-12)
