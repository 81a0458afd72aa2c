"""spec_sample_verify_noalloc against spec_sample_verify.

The allocation-free entry point takes its per-sequence inputs on the device
and keeps its tables in a library-held device array; given k_max = max k it
must return exactly what spec_sample_verify returns on the same logits.  Two
calls in a row, the second smaller, check that the array's leftover contents
from the first call do not leak into the second.
"""

import numpy as np
import pytest

from tests.gpu_util import device, say, torch
from workloads import base_positions, seq_ids_for, vocab_logits

pytestmark = pytest.mark.gpu


def B():
    from paper_2607_20507_amd import binding
    return binding


def _case(seed, ks, temps, V):
    """Device logits, drafts (sampled from q by the library's draft sampler)
    and the host per-sequence arrays of one decision-pass call."""
    dev = device()
    b = B()
    ks = np.asarray(ks, dtype=np.int32)
    temps = np.asarray(temps, dtype=np.float32)
    n = len(ks)
    ids = seq_ids_for(seed, n)
    base = base_positions(seed, n, 512, 4096)
    p_rows, q_rows = [], []
    for s, k in enumerate(ks):
        p, q = vocab_logits(seed, [s], int(k), V)
        p_rows.append(p[0])
        q_rows.append(q[0])
    P = torch.from_numpy(np.concatenate(p_rows, axis=0)).to(dev)
    nq = int(ks.sum())
    qcat = [q for q in q_rows if q.shape[0]]
    Q = torch.from_numpy(np.concatenate(qcat, axis=0)).to(dev) if qcat else torch.zeros(1, V, device=dev)
    drafts = torch.zeros(max(nq, 1), dtype=torch.int32, device=dev)
    if nq:
        pos = np.concatenate([base[s] + 1 + np.arange(ks[s]) for s in range(n)]).astype(np.int32)
        wsd = torch.empty(8 << 20, dtype=torch.uint8, device=dev)
        b.spec_sample_draft(Q, V, np.repeat(temps, ks), np.repeat(ids, ks), pos, seed, drafts, wsd)
    return ks, temps, ids, base, P, Q, drafts


def _run_both(seed, ks, temps, V):
    dev = device()
    b = B()
    ks, temps, ids, base, P, Q, drafts = _case(seed, ks, temps, V)
    n, kmax = len(ks), int(ks.max())
    # existing entry point (host per-sequence arrays, caller's workspace)
    acc_a = torch.full((n,), -7, dtype=torch.int32, device=dev)
    out_a = torch.full((n, kmax + 1), -7, dtype=torch.int32, device=dev)
    ws = torch.empty(b.spec_sample_workspace_bytes(n, int((2 * ks + 1).sum()), V), dtype=torch.uint8, device=dev)
    say("sample_verify", seed, n, V, kmax)
    b.spec_sample_verify(ks, temps, ids, base, P, Q, drafts, V, seed, acc_a, out_a, ws)
    # allocation-free entry point (device per-sequence arrays)
    acc_b = torch.full((n,), -9, dtype=torch.int32, device=dev)
    out_b = torch.full((n, kmax + 1), -9, dtype=torch.int32, device=dev)
    dk = torch.from_numpy(ks).to(dev)
    dt = torch.from_numpy(temps).to(dev)
    di = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(dev)
    db = torch.from_numpy(np.asarray(base, dtype=np.int32)).to(dev)
    torch.cuda.synchronize()
    say("sample_verify_noalloc", seed, n, V, kmax)
    b.spec_sample_verify_noalloc(kmax, dk, dt, di, db, P, Q, drafts, V, seed, acc_b, out_b)
    torch.cuda.synchronize()
    return acc_a.cpu().numpy(), out_a.cpu().numpy(), acc_b.cpu().numpy(), out_b.cpu().numpy()


def _check_same(seed, ks, temps, V):
    acc_a, out_a, acc_b, out_b = _run_both(seed, ks, temps, V)
    assert (acc_a >= 0).all()
    np.testing.assert_array_equal(acc_b, acc_a)
    np.testing.assert_array_equal(out_b, out_a)
    return acc_a


def test_noalloc_matches_sample_verify_twice_second_smaller():
    rng = np.random.default_rng(71)
    ks1 = rng.integers(0, 8, size=40).astype(np.int32)
    ks1[3] = 7
    t1 = np.array([0.0, 0.3, 1.0, 1.5], dtype=np.float32)[np.arange(40) % 4]
    acc1 = _check_same(71, ks1, t1, 32000)
    # the first call must have taken both branches of the rule
    assert (acc1 < ks1).any() and (acc1[ks1 > 0] > 0).any()
    ks2 = np.array([3, 0, 5], dtype=np.int32)
    t2 = np.array([1.0, 0.7, 0.0], dtype=np.float32)
    _check_same(72, ks2, t2, 1001)  # V % 4 != 0: scalar path


def test_noalloc_vocab_stress_rows():
    """Full-vocabulary rows at the stress shape's per-sequence depth (k = 7)."""
    n = 32
    ks = np.full(n, 7, dtype=np.int32)
    temps = np.array([0.3, 1.0, 1.5], dtype=np.float32)[np.arange(n) % 3]
    _check_same(73, ks, temps, 128256)


def test_noalloc_invalid_device_inputs_mark_every_sequence():
    """A k above k_max (or a negative temperature) is found on the device:
    nothing is decided and every count and token is -1; a later valid call
    on the same array is unaffected."""
    dev = device()
    b = B()
    V = 2048
    ks, temps, ids, base, P, Q, drafts = _case(74, [2, 3], [1.0, 1.0], V)
    for bad_k, bad_t in (([2, 4], [1.0, 1.0]), ([2, 3], [1.0, -1.0])):
        acc = torch.full((2,), 5, dtype=torch.int32, device=dev)
        out = torch.full((2, 4), 5, dtype=torch.int32, device=dev)
        dk = torch.tensor(bad_k, dtype=torch.int32, device=dev)
        dt = torch.tensor(bad_t, dtype=torch.float32, device=dev)
        di = torch.from_numpy(np.asarray(ids, dtype=np.int64)).to(dev)
        db = torch.from_numpy(np.asarray(base, dtype=np.int32)).to(dev)
        say("sample_verify_noalloc invalid", bad_k, bad_t)
        b.spec_sample_verify_noalloc(3, dk, dt, di, db, P, Q, drafts, V, 74, acc, out)
        torch.cuda.synchronize()
        assert (acc.cpu().numpy() == -1).all()
        assert (out.cpu().numpy() == -1).all()
    _check_same(75, [2, 3, 1], [1.0, 0.0, 0.5], V)


def test_noalloc_rejects_oversize_on_the_host():
    dev = device()
    b = B()
    z = torch.zeros(1, dtype=torch.int32, device=dev)
    f = torch.zeros(1, device=dev)
    with pytest.raises(b.SpecError):  # B above 256
        b.check(b.lib().spec_sample_verify_noalloc(257, 1, b.dptr(z), b.dptr(f), b.dptr(z), b.dptr(z), b.dptr(f),
                                                   b.dptr(f), b.dptr(z), 16, 1, b.dptr(z), b.dptr(z), None))
    with pytest.raises(b.SpecError):  # k_max above 15
        b.check(b.lib().spec_sample_verify_noalloc(1, 16, b.dptr(z), b.dptr(f), b.dptr(z), b.dptr(z), b.dptr(f),
                                                   b.dptr(f), b.dptr(z), 16, 1, b.dptr(z), b.dptr(z), None))
