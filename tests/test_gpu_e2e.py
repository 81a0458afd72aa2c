"""End-to-end parity of prefill -> draft x k -> verify -> commit / rollback
between the HIP library (through the C ABI) and the float64 oracle session.

* tiny fp32 pair (2-layer d=256 target, 1-layer drafter, vocab 1024, prompt
  128, k = 4, 32 steps, T = 1.0 and greedy), through the separate calls and
  through the calls the bench times: accepted counts, emitted tokens, cache
  lengths and page tables bit-exact; verify logits within 1e-4 (normwise per
  row).  A decision the oracle marks as within its margin ends the comparison
  of that sequence; at least 90% of (sequence, round) decisions are compared.
* small bf16 pair shape (12-layer d=1024 target, 2-layer drafter, vocab 32000)
  with seeded external drafts: verify logits within 2e-2 normwise per row.
"""

import numpy as np
import pytest

from oracle import rule
from oracle.decoder import Decoder
from oracle.session import Session
from tests.gpu_util import device, rel_err, say, torch
from workloads import (SMALL_BF16, TINY_FP32, model_weights, prompt_lengths_uniform,
                       seq_ids_for, uniform_prompts)

pytestmark = pytest.mark.gpu


def _sessions(cfg, max_seqs, pages, max_rows=512, n_layers_t=None, n_layers_d=None):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    tw = model_weights(cfg.target, cfg.seed, n_layers_t)
    dw = model_weights(cfg.draft, cfg.seed, n_layers_d)
    gpu = SpecSession(DeviceModel(cfg.target, tw, dev), DeviceModel(cfg.draft, dw, dev), max_seqs=max_seqs,
                      k_max=max(cfg.k), max_pages_per_seq=pages, num_pages_target=max_seqs * pages,
                      num_pages_draft=max_seqs * pages, max_rows=max_rows)
    ora = Session(Decoder(cfg.target, tw), Decoder(cfg.draft, dw), max_seqs * pages, max_seqs * pages)
    return gpu, ora


def _row_rel_errs(zg, zo):
    return [rel_err(zg[r], zo[r]) for r in range(zo.shape[0])]


def _compare_state(gpu, ora, sid):
    info = gpu.seq_info(sid)
    lt, ld = ora.lengths(sid)
    pt, pd = ora.pages(sid)
    assert (info["target_len"], info["draft_len"]) == (lt, ld)
    assert info["pages_target"] == pt and info["pages_draft"] == pd
    assert info["pending_pos"] == len(ora.seqs[sid].history) - 1


# Margins of the fp32 end-to-end comparison.  Acceptance decisions use the
# given 1e-4; the others are sized to the fp32 path's own error (logits within
# ~1e-6 of the float64 oracle, Gumbel noise within ~1e-6), an order of
# magnitude below each margin, which the test checks as it goes.
E2E_MARGINS = rule.Margins(accept=1e-4, rel=1e-4, gumbel=1e-5, greedy=2e-5)


def run_tiny(temps, steps, seed, n_seqs=4, rollback_at=None, guided=False, timed=False):
    """Drive the tiny fp32 pair through ``steps`` rounds on both sides.

    Each round the oracle drafts and decides first, so a sequence with a
    decision inside its margin is known before the GPU verifies it.  That
    sequence is released on both sides (same state, so the page allocators
    stay in step) and, after the round's commit, a fresh sequence (new id and
    prompt) is prefilled on both sides in its place, so every round compares
    a full batch.  timed = True drives the GPU through the calls the bench
    times (spec_draft_loop, then spec_verify_commit_draft per round, which
    drafts the next round itself); otherwise through spec_draft_step /
    spec_verify / spec_kv_commit.  Returns the counts of compared and total
    (sequence, round) decisions."""
    cfg = TINY_FP32
    k = cfg.k[0]
    gpu, ora = _sessions(cfg, max_seqs=n_seqs, pages=40)
    fresh_ids = iter(int(x) for x in seq_ids_for(cfg.seed + 1000 + n_seqs, 64))
    fresh_lens = iter(int(x) for x in prompt_lengths_uniform(seed + 1, 64, 20, 128))
    fresh = iter(range(1, 65))
    ids = [int(x) for x in seq_ids_for(cfg.seed + n_seqs, n_seqs)]
    lens = [128] + [int(x) for x in prompt_lengths_uniform(seed, n_seqs - 1, 20, 128)] if n_seqs > 1 else [128]
    prompts = uniform_prompts(cfg.seed, lens, cfg.target.vocab)
    say("tiny e2e prefill", ids, lens, temps, "timed" if timed else "calls")
    gpu.prefill(ids, prompts)
    ora.prefill(ids, prompts)
    for sid in ids:
        _compare_state(gpu, ora, sid)
    m = E2E_MARGINS
    T = {sid: temps[i % len(temps)] for i, sid in enumerate(ids)}
    live = list(ids)
    stats = {"compared": 0, "total": n_seqs * steps, "excluded": 0, "accepted": 0, "max_logit_err": 0.0}

    def drafts(seqs, rnd, gpu_too):
        if timed:  # the GPU drafts through spec_draft_loop
            ora.draft_loop(seqs, [T[x] for x in seqs], seed + rnd, [k] * len(seqs), m)
            return
        for j in range(k):
            if guided:
                # seeded guide tokens, half of the drafts guided
                g = np.random.default_rng([seed, rnd, j]).integers(0, cfg.target.vocab, size=len(seqs))
                g[::2] = -1
                ora.draft_step(seqs, [T[x] for x in seqs], seed + rnd, m, guide=g, boost=2.0)
                gpu.draft_step_guided(seqs, [T[x] for x in seqs], seed + rnd, g, 2.0)
            else:
                ora.draft_step(seqs, [T[x] for x in seqs], seed + rnd, m)
                if gpu_too:
                    gpu.draft_step(seqs, [T[x] for x in seqs], seed + rnd)

    if timed:
        gpu.draft_loop(live, [T[x] for x in live], seed, [k] * len(live))
    drafts(live, 0, not timed)
    for rnd in range(steps):
        outs = dict(zip(live, ora.verify(live, [T[x] for x in live], seed + rnd, m)))
        excl = [x for x in live if outs[x][0].excluded]
        if excl:
            # verify pages are taken in list order: verify again without the
            # excluded sequences, as the GPU will
            ora.undo_verify(live)
            for sid in excl:
                stats["excluded"] += 1
                gpu.release(sid)
                ora.release(sid)
                live.remove(sid)
            outs = dict(zip(live, ora.verify(live, [T[x] for x in live], seed + rnd, m)))
            assert not any(outs[x][0].excluded for x in live)
        tl = [T[x] for x in live]
        if guided:
            gpu.target_forward(live)
            z_pre = gpu.last_logits().cpu().numpy()
        more = rnd + 1 < steps
        if timed:
            na, ot = gpu.verify_commit_draft(live, tl, seed + rnd, seed + rnd + 1, [k if more else 0] * len(live))
        else:
            na, ot = gpu.verify(live, tl, seed + rnd)
        zg = gpu.last_logits().cpu().numpy()
        if guided:
            assert np.array_equal(z_pre, zg), "target_forward != verify logits"
        r0 = 0
        for i, sid in enumerate(live):
            res, zp = outs[sid]
            zrow = zg[r0:r0 + zp.shape[0]]
            r0 += zp.shape[0]
            err = float(np.max(np.abs(zrow - zp)))
            stats["max_logit_err"] = max(stats["max_logit_err"], err)
            assert max(_row_rel_errs(zrow, zp)) < 1e-4, f"round {rnd} seq {sid}: logits"
            # the greedy margin must stay well above the logits' own error
            assert err < m.greedy / 4, f"round {rnd} seq {sid}: logit error {err} too close to the margin"
            assert int(na[i]) == res.n_accepted, f"round {rnd} seq {sid}"
            assert [int(x) for x in ot[i, :res.n_accepted + 1]] == res.tokens, f"round {rnd} seq {sid}"
            stats["accepted"] += res.n_accepted
            stats["compared"] += 1
        if not timed:
            gpu.commit(live, na)
        ora.commit(live, [outs[x][0] for x in live])
        if rollback_at is not None and rnd == rollback_at:
            for sid in live:
                new_len = max(0, ora.lengths(sid)[0] - 7)
                gpu.rollback(sid, new_len)
                ora.rollback(sid, new_len)
                _compare_state(gpu, ora, sid)
        if more:
            if timed:
                drafts(live, rnd + 1, False)  # the GPU drafted these in verify_commit_draft
            new = []
            for sid in excl:  # replacements, in the same order on both sides
                nid = next(fresh_ids)
                p = uniform_prompts(cfg.seed + next(fresh), [next(fresh_lens)], cfg.target.vocab)
                gpu.prefill([nid], p)
                ora.prefill([nid], p)
                T[nid] = T[sid]
                new.append(nid)
            if timed:
                if new:
                    gpu.draft_loop(new, [T[x] for x in new], seed + rnd + 1, [k] * len(new))
                    drafts(new, rnd + 1, False)
                live += new
            else:
                live += new
                drafts(live, rnd + 1, True)
        for sid in live:
            _compare_state(gpu, ora, sid)
    gpu.close()
    say("tiny e2e", stats)
    return stats


def _check(st, frac=0.9):
    assert st["compared"] >= frac * st["total"], st


@pytest.mark.parametrize("T", [1.0, 0.0])
def test_tiny_fp32_end_to_end(T):
    """4 sequences x 32 rounds through the separate calls."""
    _check(run_tiny([T], TINY_FP32.steps, seed=2024))


@pytest.mark.parametrize("T", [1.0, 0.0])
def test_tiny_fp32_end_to_end_timed_calls(T):
    """The calls the bench times (spec_draft_loop, spec_verify_commit_draft),
    4 sequences x 32 rounds: accepted counts, tokens, lengths and page tables
    bit-exact with the oracle session."""
    _check(run_tiny([T], TINY_FP32.steps, seed=2025, timed=True))


def test_tiny_fp32_timed_calls_mixed_temperatures():
    _check(run_tiny([1.0, 0.0, 0.6], 16, seed=31, n_seqs=6, timed=True))


def test_tiny_fp32_guided_drafts():
    """Draft guidance (guide token raised to max + 2 before the draw) on a mixed
    batch: accepted counts and tokens bit-exact with the oracle, and the target
    forward alone gives the verify's logits bit for bit."""
    _check(run_tiny([1.0, 0.0, 0.7], 10, seed=99, n_seqs=3, guided=True))


def test_tiny_fp32_batch_mixed_with_rollback():
    _check(run_tiny([1.0, 0.0, 0.6], 12, seed=7, n_seqs=3, rollback_at=4))


def test_tiny_fp32_identical_draft_accepts_all():
    """Drafter == target: every draft is accepted (p/q = 1) on the GPU too."""
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    cfg = TINY_FP32
    w = model_weights(cfg.target, cfg.seed)
    gpu = SpecSession(DeviceModel(cfg.target, w, dev), DeviceModel(cfg.target, w, dev), max_seqs=1, k_max=4,
                      max_pages_per_seq=40, max_rows=256)
    gpu.prefill([5], [uniform_prompts(1, [30], cfg.target.vocab)[0]])
    for step in range(5):
        for _ in range(4):
            gpu.draft_step([5], [0.8], step)
        na, ot = gpu.verify([5], [0.8], step)
        assert int(na[0]) == 4
        gpu.commit([5], na)
    assert gpu.seq_info(5)["target_len"] == 29 + 25
    gpu.close()


def test_small_bf16_verify_logits():
    """Small bf16 pair shape, full depth and width, 2 sequences with short
    prompts and seeded external drafts: verify logits within 2e-2."""
    cfg = SMALL_BF16
    k = cfg.k[0]
    gpu, ora = _sessions(cfg, max_seqs=2, pages=16, max_rows=256)
    dev = device()
    ids = [11, 1 << 33]
    prompts = uniform_prompts(cfg.seed, [70, 41], cfg.target.vocab)
    say("small bf16 prefill")
    gpu.prefill(ids, prompts)
    ora.prefill(ids, prompts)
    rng = np.random.default_rng(3)
    for sid in ids:
        drafts = rng.integers(0, cfg.target.vocab, size=k).astype(np.int32)
        zq = (rng.standard_normal((k, cfg.target.vocab)) * 0.5).astype(np.float32)
        zq_dev = torch.from_numpy(zq).to(dev)
        gpu.set_drafts(sid, drafts, zq_dev)
        ora.set_drafts(sid, drafts, zq)
        setattr(gpu, f"_keep_{sid}", zq_dev)
    na, ot = gpu.verify(ids, [0.7, 0.7], 5)
    outs = ora.verify(ids, [0.7, 0.7], 5)
    zg = gpu.last_logits().cpu().numpy()
    r0 = 0
    for i, (res, zp) in enumerate(outs):
        errs = _row_rel_errs(zg[r0:r0 + k + 1], zp)
        r0 += k + 1
        assert max(errs) < 2e-2, errs
        assert 0 <= int(na[i]) <= k
    gpu.commit(ids, na)
    gpu.close()


def _bf16_pair_hd128(vocab=1024):
    """A small bf16 pair with the 8B-shaped head layout (head_dim 128, GQA 2:1)."""
    from dataclasses import replace
    from workloads.configs import ModelShape
    t = ModelShape(f"tiny-bf16-hd128-v{vocab}", n_layers=2, d_model=256, n_heads=2, n_kv_heads=1, head_dim=128,
                   ffn_dim=512, vocab=vocab, rope_theta=5e5, dtype="bf16")
    return replace(SMALL_BF16, name=t.name, target=t, draft=replace(t, n_layers=1), k=(4,))


@pytest.mark.parametrize("which", ["hd128", "small-2L", "hd128-v1000"])
def test_fused_small_rows_teacher_forced(which):
    """Batch-1 rows (<= 8: RMSNorm and RoPE / KV append fused into the GEMMs):
    every draft logits row and every verify logits row of three rounds against
    the oracle's no-cache forward over the same tokens, within 2e-2."""
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    if which == "hd128":
        cfg, lt, ld = _bf16_pair_hd128(), None, None
    elif which == "hd128-v1000":  # a vocabulary that is not a multiple of 16: unfused LM head
        cfg, lt, ld = _bf16_pair_hd128(1000), None, None
    else:
        cfg, lt, ld = SMALL_BF16, 2, 1
    k = cfg.k[0]
    dev = device()
    tw = model_weights(cfg.target, cfg.seed, lt)
    dw = model_weights(cfg.draft, cfg.seed + 1, ld)
    gpu = SpecSession(DeviceModel(cfg.target, tw, dev, n_layers=lt), DeviceModel(cfg.draft, dw, dev, n_layers=ld),
                      max_seqs=1, k_max=k, max_pages_per_seq=16, max_rows=256)
    tgt, drf = Decoder(cfg.target, tw), Decoder(cfg.draft, dw)
    sid = 77
    hist = [int(x) for x in uniform_prompts(cfg.seed, [45], cfg.target.vocab)[0]]
    say("fused rows teacher-forced", which)
    gpu.prefill([sid], [np.array(hist, dtype=np.int32)])
    for rnd in range(3):
        for _ in range(k):
            gpu.draft_step([sid], [0.8], 31 + rnd)
        drafts = gpu.draft_tokens(sid)
        na, ot = gpu.verify([sid], [0.8], 31 + rnd)
        zp_gpu = gpu.last_logits().cpu().numpy()
        zq_gpu = np.stack([gpu.draft_logits(sid, j).cpu().numpy() for j in range(k)])
        fed = hist + drafts
        zt = tgt.full_logits(fed)
        zd = drf.full_logits(fed[:-1])
        n = len(hist) - 1
        for j in range(k):
            e = rel_err(zq_gpu[j], zd[n + j])
            assert e < 2e-2, f"round {rnd} draft row {j}: {e}"
        for r in range(k + 1):
            e = rel_err(zp_gpu[r], zt[n + r])
            assert e < 2e-2, f"round {rnd} verify row {r}: {e}"
        a = int(na[0])
        gpu.commit([sid], na)
        hist += [int(x) for x in ot[0, :a + 1]]
    gpu.close()



def _wide_pair(d, hd):
    """One-layer bf16 target of width d (32 query / 8 kv heads of hd), small
    FFN and vocabulary, with a one-layer drafter: the residual-add GEMMs of a
    48-row verify split K and fold the RMSNorm into the split-K reduction at
    this row width."""
    from workloads.configs import ModelShape, PairConfig
    t = ModelShape(f"w{d}-target", 1, d, 32, 8, hd, 1024, 2048, 5e5)
    dr = ModelShape(f"w{d}-draft", 1, 512, 8, 8, 64, 512, 2048, 5e5)
    return PairConfig(f"w{d}", t, dr, batch=8, context=("uniform", 40, 90), k=(5,), temperatures=(0.7,),
                      steps=1)


@pytest.mark.parametrize("which", ["small-2L", "d2048", "d4096"])
def test_split_k_rows_teacher_forced(which):
    """A verify of 8 sequences (48 rows): every projection runs on the MFMA
    kernel with split-K, the residual-add GEMMs' split-K reduction also
    applies the next RMSNorm (rows of 1024, 2048 and 4096 columns: one, two
    and four 4-column chunks per thread), and rope_kv does RoPE / KV append.
    Every verify logits row against the oracle's no-cache forward over the
    same tokens, within 2e-2."""
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    if which == "small-2L":
        cfg, lt, ld = SMALL_BF16, 2, 1
    else:
        cfg, lt, ld = (_wide_pair(2048, 64) if which == "d2048" else _wide_pair(4096, 128)), 1, 1
    k = cfg.k[0]
    dev = device()
    tw = model_weights(cfg.target, cfg.seed, lt)
    dw = model_weights(cfg.draft, cfg.seed + 1, ld)
    gpu = SpecSession(DeviceModel(cfg.target, tw, dev, n_layers=lt), DeviceModel(cfg.draft, dw, dev, n_layers=ld),
                      max_seqs=8, k_max=k, max_pages_per_seq=16, max_rows=512)
    tgt = Decoder(cfg.target, tw)
    ids = list(range(100, 108))
    prompts = uniform_prompts(cfg.seed + 5, [40 + 7 * i for i in range(8)], cfg.target.vocab)
    say("split-K rows teacher-forced", which, ": prefill 8 sequences")
    gpu.prefill(ids, prompts)
    rng = np.random.default_rng(9)
    keep, drafts = [], {}
    for sid in ids:
        drafts[sid] = rng.integers(0, cfg.target.vocab, size=k).astype(np.int32)
        zq = torch.from_numpy((rng.standard_normal((k, cfg.target.vocab)) * 0.5).astype(np.float32)).to(dev)
        gpu.set_drafts(sid, drafts[sid], zq)
        keep.append(zq)
    na, ot = gpu.verify(ids, [0.7] * len(ids), 5)
    zg = gpu.last_logits().cpu().numpy()
    r0 = 0
    for sid, p in zip(ids, prompts):
        fed = [int(x) for x in p] + [int(x) for x in drafts[sid]]
        zt = tgt.full_logits(fed)
        n = len(p) - 1
        for r in range(k + 1):
            e = rel_err(zg[r0 + r], zt[n + r])
            assert e < 2e-2, f"seq {sid} verify row {r}: {e}"
        r0 += k + 1
    gpu.commit(ids, na)
    gpu.close()
