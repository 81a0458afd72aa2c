"""Pins of the oracle's plain decoding (a session with no draft model).

Plain decoding is the rule with no drafts: each step's token is the bonus
draw from p_1 = softmax(z / T) of the pending row, with BONUS noise at the
next position, or its argmax at T = 0.  These tests check the cached,
paged decode against the no-cache forward over the growing history and
against the categorical draw written out directly from the Gumbel-max trick.
"""

import numpy as np

from oracle import philox
from oracle.decoder import Decoder
from oracle.session import Session
from workloads import TINY_FP32, model_weights, seq_ids_for, uniform_prompts


def _session():
    shape = TINY_FP32.target
    dec = Decoder(shape, model_weights(shape, 11))
    return dec, Session(dec, None, num_pages_target=64, num_pages_draft=0)


def _prompts(n):
    return uniform_prompts(11, [9, 23, 16][:n], TINY_FP32.target.vocab)


def test_greedy_decode_is_the_argmax_chain_of_the_no_cache_forward():
    dec, sess = _session()
    ids = [int(x) for x in seq_ids_for(11, 3)]
    prompts = _prompts(3)
    sess.prefill(ids, prompts)
    toks, excl, logits = sess.decode(ids, [0.0] * 3, seed=5, steps=10)
    for i, p in enumerate(prompts):
        hist = [int(t) for t in p]
        for j in range(10):
            z = dec.full_logits(hist)[-1]
            np.testing.assert_allclose(logits[j][i], z, rtol=0, atol=1e-12 * np.abs(z).max())
            t = int(np.argmax(z))  # first maximum: the lowest id on ties
            assert toks[i][j] == t
            hist.append(t)
        assert sess.seqs[ids[i]].history == hist
        assert sess.lengths(ids[i]) == (len(hist) - 1, 0)


def test_sampled_decode_draws_with_bonus_noise_at_the_next_position():
    dec, sess = _session()
    ids = [int(x) for x in seq_ids_for(12, 2)]
    prompts = _prompts(2)
    sess.prefill(ids, prompts)
    T, seed = 0.9, 77
    toks, _, _ = sess.decode(ids, [T, T], seed=seed, steps=8)
    V = dec.shape.vocab
    for i, p in enumerate(prompts):
        hist = [int(t) for t in p]
        for j in range(8):
            z = dec.full_logits(hist)[-1] / T
            logp = z - (z.max() + np.log(np.exp(z - z.max()).sum()))
            n = len(hist) - 1  # the pending token's position; the draw decides n + 1
            g = philox.gumbel(seed, ids[i], n + 1, philox.BONUS, V)
            t = int(np.argmax(logp + g))
            assert toks[i][j] == t
            hist.append(t)


def test_decode_pages_grow_lowest_free_first():
    _, sess = _session()
    ids = [int(x) for x in seq_ids_for(13, 2)]
    sess.prefill(ids, _prompts(2))
    sess.decode(ids, [1.0, 0.0], seed=3, steps=20)
    (t0, d0), (t1, d1) = sess.pages(ids[0]), sess.pages(ids[1])
    assert d0 == [] and d1 == []
    # prompts of 9 and 23 tokens: 8 and 22 cached positions, then 20 steps
    # interleaved sequence by sequence
    assert len(t0) == (8 + 20 + 15) // 16 and len(t1) == (22 + 20 + 15) // 16
    assert sorted(t0 + t1) == list(range(len(t0) + len(t1)))
