"""GPU parity of the decision pass (draft sampler, acceptance scan, residual
and bonus draws, greedy mode) against the oracle rule on seeded logits.

Both sides read the same fp32 logits and key their random streams the same
way, so accepted counts and emitted tokens must be bit-exact, except where the
oracle (float64) marks a decision as within its margin: |u - min(1, p/q)| <
1e-4 for acceptance, or a Gumbel-max winner that a relative error of 1e-4 on
the probabilities (1e-5 on the noise) could overturn.  Excluded sequences are
counted and must stay rare.
"""

import numpy as np
import pytest

from oracle import rule
from tests.gpu_util import device, say, torch
from workloads import base_positions, seq_ids_for, vocab_logits

pytestmark = pytest.mark.gpu

MARGINS = rule.Margins(accept=1e-4, rel=1e-4, gumbel=1e-5, greedy=0.0)


def B():
    from paper_2607_20507_amd import binding
    return binding


def _gen(seed, ks, V, check):
    """Per-sequence logits for the sequences in ``check`` (others: any values)."""
    p_rows, q_rows = [], []
    for s, k in enumerate(ks):
        p, q = vocab_logits(seed, [s], int(k), V)
        p_rows.append(p[0])
        q_rows.append(q[0])
    return p_rows, q_rows


def run_decision_case(seed, ks, temps, V, check=None, pos_range=(512, 4096)):
    dev = device()
    b = B()
    Bn = len(ks)
    ks = np.asarray(ks, dtype=np.int32)
    temps = np.asarray(temps, dtype=np.float32)
    ids = seq_ids_for(seed, Bn)
    base = base_positions(seed, Bn, *pos_range)
    p_rows, q_rows = _gen(seed, ks, V, check)
    P = torch.from_numpy(np.concatenate(p_rows, axis=0)).to(dev)
    qcat = [q for q in q_rows if q.shape[0]]
    Q = torch.from_numpy(np.concatenate(qcat, axis=0)).to(dev) if qcat else torch.zeros(1, V, device=dev)
    nq = int(ks.sum())
    # GPU drafts from q (DRAFT stream at positions n+1..n+k)
    drow_T = np.repeat(temps, ks)
    drow_id = np.repeat(ids, ks)
    drow_pos = np.concatenate([base[s] + 1 + np.arange(ks[s]) for s in range(Bn)]).astype(np.int32) if nq else np.zeros(0, np.int32)
    drafts = torch.zeros(max(nq, 1), dtype=torch.int32, device=dev)
    if nq:
        wsd = torch.empty(8 << 20, dtype=torch.uint8, device=dev)
        say("sample_draft", seed, Bn, V)
        b.spec_sample_draft(Q, V, drow_T, drow_id, drow_pos, seed, drafts, wsd)
    n_acc = torch.full((Bn,), -7, dtype=torch.int32, device=dev)
    kmax = int(ks.max())
    out = torch.full((Bn, kmax + 1), -7, dtype=torch.int32, device=dev)
    ws = torch.empty(b.spec_sample_workspace_bytes(Bn, int((ks + 1).sum() + nq), V), dtype=torch.uint8, device=dev)
    say("sample_verify", seed, Bn, V, kmax)
    b.spec_sample_verify(ks, temps, ids, base, P, Q, drafts, V, seed, n_acc, out, ws)
    torch.cuda.synchronize()
    g_drafts = drafts.cpu().numpy()
    g_acc = n_acc.cpu().numpy()
    g_out = out.cpu().numpy()
    checked = excluded = 0
    qo = 0
    for s in range(Bn):
        k = int(ks[s])
        if check is not None and s not in check:
            qo += k
            continue
        T = float(temps[s])
        od = []
        bad = False
        for j in range(k):
            t, ex = rule.sample_draft(q_rows[s][j], T, seed, int(ids[s]), int(base[s]) + j + 1, MARGINS)
            od.append(t)
            bad |= ex
        if bad:
            excluded += 1
            qo += k
            continue
        assert od == [int(x) for x in g_drafts[qo:qo + k]], f"draft tokens differ at seq {s}"
        res = rule.verify(p_rows[s], q_rows[s], od, T, seed, int(ids[s]), int(base[s]), MARGINS)
        qo += k
        if res.excluded:
            excluded += 1
            continue
        checked += 1
        assert int(g_acc[s]) == res.n_accepted, f"seq {s}: accepted {g_acc[s]} vs {res.n_accepted}"
        want = res.tokens + [-1] * (kmax + 1 - len(res.tokens))
        assert [int(x) for x in g_out[s]] == want, f"seq {s}: tokens {g_out[s]} vs {want}"
    return checked, excluded


@pytest.mark.parametrize("V", [1000, 1001, 32000])
def test_decision_pass_small(V):
    ks = [0, 1, 3, 5, 7, 15, 2, 4]
    temps = [1.0, 0.7, 0.3, 1.5, 0.0, 1.0, 0.0, 2.0]
    checked, excluded = run_decision_case(11 + V, ks, temps, V)
    assert checked >= len(ks) - 2 and excluded <= 2


def test_decision_pass_greedy_ties_lowest_index():
    """Exactly tied maxima resolve to the lowest token id on both paths."""
    dev = device()
    b = B()
    V = 4096
    p = np.zeros((3, V), dtype=np.float32)
    p[:, [7, 900, 4000]] = 5.0
    q = np.zeros((2, V), dtype=np.float32)
    P = torch.from_numpy(p).to(dev)
    Q = torch.from_numpy(q).to(dev)
    drafts = torch.tensor([7, 900], dtype=torch.int32, device=dev)
    n_acc = torch.zeros(1, dtype=torch.int32, device=dev)
    out = torch.zeros(1, 3, dtype=torch.int32, device=dev)
    ws = torch.empty(b.spec_sample_workspace_bytes(1, 5, V), dtype=torch.uint8, device=dev)
    b.spec_sample_verify([2], [0.0], [1], [10], P, Q, drafts, V, 0, n_acc, out, ws)
    torch.cuda.synchronize()
    assert int(n_acc.item()) == 1 and out.cpu().numpy().tolist() == [[7, 7, -1]]


def test_decision_pass_vocab_stress_full_size():
    """256 sequences x (7 + 1) target rows x 128256, temperatures cycling
    {0.3, 1.0, 1.5}; the oracle checks a seeded sample of 24 sequences."""
    Bn, k, V = 256, 7, 128256
    temps = [(0.3, 1.0, 1.5)[s % 3] for s in range(Bn)]
    check = set(np.random.default_rng(5).choice(Bn, size=24, replace=False).tolist())
    checked, excluded = run_decision_case(1234, [k] * Bn, temps, V, check=check)
    assert checked >= 20


def test_decision_pass_vocab_stress_greedy_full_size():
    Bn, k, V = 256, 7, 128256
    check = set(range(0, Bn, 16))
    checked, excluded = run_decision_case(77, [k] * Bn, [0.0] * Bn, V, check=check)
    assert checked == len(check)


@pytest.mark.parametrize("V,T", [(1000, 0.0), (1001, 0.5), (128256, 1.5), (32000, 1.0)])
def test_draft_sampler(V, T):
    dev = device()
    b = B()
    n = 16
    rng = np.random.default_rng(V)
    z = (rng.standard_normal((n, V)) * 2).astype(np.float32)
    ids = seq_ids_for(V, n)
    pos = rng.integers(0, 5000, size=n).astype(np.int32)
    tok = torch.full((n,), -1, dtype=torch.int32, device=dev)
    ws = torch.empty(8 << 20, dtype=torch.uint8, device=dev)
    say("draft sampler", V, T)
    b.spec_sample_draft(torch.from_numpy(z).to(dev), V, [T] * n, ids, pos, 99, tok, ws)
    torch.cuda.synchronize()
    got = tok.cpu().numpy()
    agree = 0
    for i in range(n):
        t, ex = rule.sample_draft(z[i], T, 99, int(ids[i]), int(pos[i]), MARGINS)
        if ex:
            continue
        assert int(got[i]) == t
        agree += 1
    assert agree >= n - 1


@pytest.mark.parametrize("T", [0.9, 0.0])
def test_out_of_range_draft_is_rejected(T):
    """A draft id outside the vocabulary is never accepted, and the draw at
    that position is the ordinary one: from norm(max(0, p_j - q_j)) with the
    RESAMPLE stream (argmax p_j when greedy), with the q row normalised as
    usual.  Draft 0 has q = p (always accepted); draft 1 is out of range."""
    from oracle import philox
    dev = device()
    b = B()
    V, k, seed, sid, base = 1000, 3, 5, 123456789012, 700
    g = np.random.default_rng(8)
    p = (g.standard_normal((k + 1, V)) * 2).astype(np.float32)
    q = (g.standard_normal((k, V)) * 2).astype(np.float32)
    q[0] = p[0]
    drafts = np.array([int(np.argmax(p[0])), V + 5, 3], dtype=np.int32)
    n_acc = torch.full((1,), -7, dtype=torch.int32, device=dev)
    out = torch.full((1, k + 1), -7, dtype=torch.int32, device=dev)
    ws = torch.empty(b.spec_sample_workspace_bytes(1, 2 * k + 1, V), dtype=torch.uint8, device=dev)
    b.spec_sample_verify([k], [T], [sid], [base], torch.from_numpy(p).to(dev), torch.from_numpy(q).to(dev),
                         torch.from_numpy(drafts).to(dev), V, seed, n_acc, out, ws)
    torch.cuda.synchronize()
    assert int(n_acc.item()) == 1
    if T == 0.0:
        want = int(np.argmax(p[1]))
    else:
        pp, qq = rule.softmax_t(p[1], T), rule.softmax_t(q[1], T)
        want, ex = rule.draw_residual(pp, qq, philox.gumbel(seed, sid, base + 2, philox.RESAMPLE, V), MARGINS)
        assert not ex
    assert out.cpu().numpy().tolist() == [[int(drafts[0]), want, -1, -1]]
