"""Pins of the page-assignment simulation and of the session's cache bookkeeping."""

import numpy as np
import pytest

from oracle.paging import PageOOM, PagePool
from oracle.decoder import Decoder
from oracle.session import Session
from workloads import ModelShape, model_weights


def test_lowest_free_first_and_eager_free():
    p = PagePool(8, page_size=16)
    p.ensure(1, 33)          # 3 pages
    p.ensure(2, 16)          # 1 page
    assert p.tables[1] == [0, 1, 2] and p.tables[2] == [3]
    p.truncate(1, 17)        # keeps pages for positions 0..16 -> 2 pages
    assert p.tables[1] == [0, 1]
    p.ensure(2, 40)          # needs 2 more: lowest free are 2 and 4
    assert p.tables[2] == [3, 2, 4]
    assert p.slot(2, 17) == 2 * 16 + 1
    p.truncate(1, 0)
    assert p.tables[1] == [] and sorted(p.free) == [0, 1, 5, 6, 7]


def test_oom_leaves_state_unchanged():
    p = PagePool(4, page_size=16)
    p.ensure(1, 48)
    before = (list(p.free), {k: list(v) for k, v in p.tables.items()})
    with pytest.raises(PageOOM):
        p.ensure(2, 33)
    assert (list(p.free), {k: list(v) for k, v in p.tables.items()}) == before


def test_boundaries():
    p = PagePool(4, page_size=16)
    p.ensure(1, 16)
    assert len(p.tables[1]) == 1
    p.ensure(1, 17)
    assert len(p.tables[1]) == 2
    p.truncate(1, 16)
    assert len(p.tables[1]) == 1
    p.ensure(3, 0)
    assert p.tables[3] == []


def test_session_lengths_pages_and_history():
    """Scripted steps: lengths after commit follow n+a+1 / min(len_d, n+a+1), and
    page tables cover exactly the cached positions."""
    sh = ModelShape("pg", 1, 16, 2, 2, 8, 16, 20, 1e4, dtype="f32", init_std=0.3)
    dec = Decoder(sh, model_weights(sh, 51))
    sess = Session(dec, dec, 32, 32, page_size=4)
    sess.prefill([1, 2], [[1, 2, 3, 4, 5], [6, 7]])
    assert sess.lengths(1) == (4, 4) and sess.lengths(2) == (1, 1)
    for _ in range(3):
        sess.draft_step([1, 2], [0.7, 0.7], seed=3)
    assert sess.lengths(1) == (4, 7)
    out = sess.verify([1, 2], [0.7, 0.7], seed=3)
    res = [r for r, _ in out]
    sess.commit([1, 2], res)
    for sid, r, n0 in ((1, res[0], 4), (2, res[1], 1)):
        lt, ld = sess.lengths(sid)
        assert lt == n0 + r.n_accepted + 1
        assert ld == min(n0 + 3, n0 + r.n_accepted + 1)
        pt, pd = sess.pages(sid)
        assert len(pt) == (lt + 3) // 4 and len(pd) == (ld + 3) // 4
    sess.rollback(1, 2)
    assert sess.lengths(1) == (2, 2)
    assert sess.seqs[1].history == [1, 2, 3]
    used = sum(len(v) for v in sess.pool_t.tables.values())
    assert used + len(sess.pool_t.free) == 32


def test_undo_verify_restores_cache_and_pages():
    """A verify taken back leaves target lengths, page tables and the free
    pool as before it; verifying a subset afterwards allocates as if the
    other sequence had never been verified."""
    sh = ModelShape("pg", 1, 16, 2, 2, 8, 16, 20, 1e4, dtype="f32", init_std=0.3)
    dec = Decoder(sh, model_weights(sh, 52))
    sess = Session(dec, dec, 32, 32, page_size=4)
    sess.prefill([1, 2, 3], [[1, 2, 3, 4], [5, 6, 7, 8], [9, 10]])
    for _ in range(3):
        sess.draft_step([1, 2, 3], [0.7] * 3, seed=4)
    before = {s: (sess.lengths(s), sess.pages(s)) for s in (1, 2, 3)}
    free = sorted(sess.pool_t.free)
    out1 = sess.verify([1, 2, 3], [0.7] * 3, seed=4)
    assert sess.pages(2)[0] != before[2][1][0]
    sess.undo_verify([1, 2, 3])
    assert {s: (sess.lengths(s), sess.pages(s)) for s in (1, 2, 3)} == before
    assert sorted(sess.pool_t.free) == free
    # without sequence 1, sequence 2 takes the pages sequence 1 took before
    taken1 = [p for p in sess.pages(1)[0]]
    sess.release(1)
    out2 = sess.verify([2, 3], [0.7] * 2, seed=4)
    assert [r.tokens for r, _ in out2] == [r.tokens for r, _ in out1[1:]]
    assert set(sess.pages(2)[0]) & set(taken1)


def test_guided_draft_row_and_draw():
    """Draft guidance raises the guide token to max + boost in the kept q row;
    with a large boost the draw is the guide token, with guide -1 nothing changes."""
    import numpy as np
    from oracle.decoder import Decoder
    from oracle.session import Session
    from workloads import TINY_FP32, model_weights, uniform_prompts
    cfg = TINY_FP32
    tw = model_weights(cfg.target, cfg.seed, 1)
    dw = model_weights(cfg.draft, cfg.seed, 1)
    a = Session(Decoder(cfg.target, tw), Decoder(cfg.draft, dw), 64, 64)
    b = Session(Decoder(cfg.target, tw), Decoder(cfg.draft, dw), 64, 64)
    prompt = uniform_prompts(3, [20], cfg.target.vocab)[0]
    a.prefill([1], [prompt])
    b.prefill([1], [prompt])
    x_a = a.draft_step([1], [1.0], 5, guide=[17], boost=50.0)
    x_b = b.draft_step([1], [1.0], 5)
    assert x_a == [17]
    za, zb = a.seqs[1].zq[0], b.seqs[1].zq[0]
    assert za[17] == zb.max() + 50.0
    assert np.array_equal(np.delete(za, 17), np.delete(zb, 17))
    c = Session(Decoder(cfg.target, tw), Decoder(cfg.draft, dw), 64, 64)
    c.prefill([1], [prompt])
    assert c.draft_step([1], [1.0], 5, guide=[-1], boost=50.0) == x_b


def test_draft_loop_takes_pages_first_in_list_order():
    """A draft loop call takes every step's pages before any step runs, one
    sequence after the other; per-step calls interleave them.  The drafts and
    lengths are the same either way."""
    sh = ModelShape("pg", 1, 16, 2, 2, 8, 16, 20, 1e4, dtype="f32", init_std=0.3)
    dec = Decoder(sh, model_weights(sh, 53))
    a = Session(dec, dec, 64, 64, page_size=4)
    b = Session(dec, dec, 64, 64, page_size=4)
    # draft caches of 6 and 4 positions: sequence 1 needs a new page at step 3
    # (position 8), sequence 2 at step 1 (position 4)
    prompts = [[1, 2, 3, 4, 5, 6, 7], [8, 9, 10, 11, 12]]
    for s in (a, b):
        s.prefill([1, 2], prompts)
    a.draft_loop([1, 2], [0.7, 0.7], 3, [4, 4])
    for _ in range(4):
        b.draft_step([1, 2], [0.7, 0.7], seed=3)
    assert a.seqs[1].drafts == b.seqs[1].drafts and a.seqs[2].drafts == b.seqs[2].drafts
    assert a.lengths(1) == b.lengths(1) and a.lengths(2) == b.lengths(2)
    assert a.pages(1)[1] == [0, 1, 3] and a.pages(2)[1] == [2, 4]
    assert b.pages(1)[1] == [0, 1, 4] and b.pages(2)[1] == [2, 3]
