"""Parity at the configured shapes, through the calls the bench times.

Every test drives the GPU with spec_draft_loop once and then
spec_verify_commit_draft per round (verify, commit, next round's drafts in
one call), and checks the draft logits rows and verify logits rows of the
checked sequences against the float64 oracle decoders within 2e-2 (normwise
per row; bf16 weights and KV).  The comparison is teacher-forced: the tokens
the GPU drafted and committed become the input sequence, and the oracle
computes every expected row from that sequence alone (its own KV cache, its
own forward).  A 2e-2 logit tolerance moves p / q by far more than the rule's
1e-4 exclusion, so bf16 decisions are compared on shared logits instead
(tests/test_gpu_vocab.py).

* batch 1 at the 8B / 1B widths (d 4096, 32 q / 8 kv heads of 128, ffn 14336;
  drafter d 2048, heads of 64, ffn 8192; vocab 128256) with one layer each:
  the fused small-row kernels (GEMV half tiles, skinny MFMA GEMMs with
  RMSNorm folded in, the QKV epilogue's RoPE and paged KV append) at their
  real shapes, k = 5, T = 0.8 and 0;
* the small bf16 pair as configured: 12-layer target, 2-layer drafter, batch
  8, prompt lengths uniform in [256, 512], k = 5, T = 0.7;
* a serving-shaped batch: 64 sequences with contexts log-uniform in
  [512, 4096], k drawn from {3, 5, 7}, full width with one layer each, a
  rollback in the middle; four sequences checked.
"""

import numpy as np
import pytest

from oracle.decoder import Decoder, matmul_wt
from tests.gpu_util import device, rel_err, say, torch
from workloads.configs import L1B_DRAFT, L8B_TARGET
from workloads import (SMALL_BF16, context_lengths_loguniform, draft_lengths,
                       model_weights, prompt_lengths_uniform, seq_ids_for, uniform_prompts)

pytestmark = pytest.mark.gpu

TOL = 2e-2


class _OracleSeq:
    """The oracle's caches of one checked sequence, following the committed
    history: the target cache holds positions < n, the draft cache < len_d."""

    def __init__(self, tgt, drf, prompt):
        self.hist = [int(t) for t in prompt]
        self.kv_t, self.kv_d = tgt.new_kv(), drf.new_kv()
        P = len(self.hist)
        if P > 1:
            tgt.forward(self.kv_t, self.hist[:-1], np.arange(P - 1), logits=False)
            drf.forward(self.kv_d, self.hist[:-1], np.arange(P - 1), logits=False)


def _rounds(gpu, tgt, drf, ids, prompts, temps, ks, rounds, seed, check, rollback=None):
    """Run ``rounds`` speculative rounds of the listed sequences on the GPU and
    compare the checked ones with the oracle; returns the number of rows
    compared.  rollback = (round, seq_id, tokens to drop) rolls one sequence
    back after that round (both sides) and drafts it again."""
    say("prefill", len(ids), "sequences; oracle prefill of", len(check))
    gpu.prefill(ids, prompts)
    ora = {sid: _OracleSeq(tgt, drf, prompts[ids.index(sid)]) for sid in check}
    T = dict(zip(ids, temps))
    K = dict(zip(ids, ks))
    gpu.draft_loop(ids, temps, seed, ks)
    compared = 0
    for rnd in range(rounds):
        # the GPU's drafts of this round (made by the previous call)
        drafts = {sid: gpu.draft_tokens(sid) for sid in check}
        zq_gpu = {sid: np.stack([gpu.draft_logits(sid, j).cpu().numpy() for j in range(K[sid])]) for sid in check}
        nxt = ks if rnd + 1 < rounds else [0] * len(ids)
        na, ot = gpu.verify_commit_draft(ids, temps, seed + rnd, seed + rnd + 1, nxt)
        zp_gpu = gpu.last_logits().cpu().numpy()
        row0, r0 = {}, 0
        for sid in ids:
            row0[sid] = r0
            r0 += K[sid] + 1
        # oracle: hidden states of every checked row, then one LM-head product per model
        hy_t, hy_d, spans = [], [], []
        for sid in check:
            o = ora[sid]
            n, d = len(o.hist) - 1, drafts[sid]
            yt = tgt.forward(o.kv_t, [o.hist[n]] + d, n + np.arange(len(d) + 1), logits=False)
            ld = o.kv_d.length
            feed = o.hist[ld:] + d[:-1]
            yd = drf.forward(o.kv_d, feed, ld + np.arange(len(feed)), logits=False)
            hy_t.append(yt)
            hy_d.append(yd[n - ld:])  # rows at positions n .. n + k - 1 give drafts 1 .. k
            spans.append((sid, n, d))
        zt = matmul_wt(np.concatenate(hy_t), tgt.w["lm_head"])
        zd = matmul_wt(np.concatenate(hy_d), drf.w["lm_head"])
        it = id_ = 0
        for sid, n, d in spans:
            k = len(d)
            for j in range(k):
                e = rel_err(zq_gpu[sid][j], zd[id_ + j])
                assert e < TOL, f"round {rnd} seq {sid} draft row {j}: {e}"
            for r in range(k + 1):
                e = rel_err(zp_gpu[row0[sid] + r], zt[it + r])
                assert e < TOL, f"round {rnd} seq {sid} verify row {r}: {e}"
            compared += 2 * k + 1
            it += k + 1
            id_ += k
            # commit the GPU's outcome on the oracle's caches
            i = ids.index(sid)
            a = int(na[i])
            o = ora[sid]
            o.hist += [int(x) for x in ot[i, :a + 1]]
            o.kv_t.truncate(n + a + 1)
            o.kv_d.truncate(min(o.kv_d.length, n + a + 1))
        say("round", rnd, "accepted", [int(x) for x in na[:8]], "rows compared", compared)
        if rollback is not None and rollback[0] == rnd:
            _, sid, drop = rollback
            info = gpu.seq_info(sid)
            new_len = info["target_len"] - drop
            gpu.rollback(sid, new_len)
            if sid in ora:
                o = ora[sid]
                del o.hist[new_len + 1:]
                o.kv_t.truncate(new_len)
                o.kv_d.truncate(min(o.kv_d.length, new_len))
            if rnd + 1 < rounds:
                gpu.draft_loop([sid], [T[sid]], seed + rnd + 1, [K[sid]])
    return compared


@pytest.fixture(scope="module")
def wide_pair():
    say("generating one-layer 8B / 1B-shaped weights (host)")
    tw = model_weights(L8B_TARGET, 1234, 1)
    dw = model_weights(L1B_DRAFT, 1235, 1)
    return tw, dw


def _wide_session(wide_pair, max_seqs, k_max, pages, max_rows):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    tw, dw = wide_pair
    dev = device()
    gpu = SpecSession(DeviceModel(L8B_TARGET, tw, dev, n_layers=1), DeviceModel(L1B_DRAFT, dw, dev, n_layers=1),
                      max_seqs=max_seqs, k_max=k_max, max_pages_per_seq=pages, max_rows=max_rows)
    return gpu, Decoder(L8B_TARGET, tw), Decoder(L1B_DRAFT, dw)


@pytest.mark.parametrize("T", [0.8, 0.0])
def test_batch1_full_width_timed_calls(wide_pair, T):
    gpu, tgt, drf = _wide_session(wide_pair, 1, 5, 32, 512)
    sid = 987654321
    prompt = uniform_prompts(77, [320], L8B_TARGET.vocab)
    say("batch-1 full width, T", T)
    n = _rounds(gpu, tgt, drf, [sid], prompt, [T], [5], 3, 40 + int(10 * T), [sid])
    assert n == 3 * 11
    gpu.close()


def test_small_pair_as_configured_timed_calls():
    """12-layer target / 2-layer drafter, 8 sequences, prompts U[256, 512]."""
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    cfg = SMALL_BF16
    dev = device()
    say("small pair weights")
    tw = model_weights(cfg.target, cfg.seed)
    dw = model_weights(cfg.draft, cfg.seed + 1)
    gpu = SpecSession(DeviceModel(cfg.target, tw, dev), DeviceModel(cfg.draft, dw, dev), max_seqs=cfg.batch,
                      k_max=5, max_pages_per_seq=40, max_rows=1024)
    lens = prompt_lengths_uniform(cfg.seed, cfg.batch, 256, 512)
    ids = [int(x) for x in seq_ids_for(cfg.seed, cfg.batch)]
    prompts = uniform_prompts(cfg.seed, lens, cfg.target.vocab)
    n = _rounds(gpu, Decoder(cfg.target, tw), Decoder(cfg.draft, dw), ids, prompts, [0.7] * cfg.batch,
                [5] * cfg.batch, 3, 17, ids)
    assert n == 3 * cfg.batch * 11
    gpu.close()


def test_serving_shape_full_width_timed_calls(wide_pair):
    """64 sequences, contexts log-uniform in [512, 4096], k from {3, 5, 7}:
    364-row verify GEMMs on the MFMA kernel with split K, the split-K
    reduction with RMSNorm, the serving attention planner; the shortest
    sequence of each k and one more are checked, one of them rolled back."""
    B_, seed = 64, 4321
    ctx = context_lengths_loguniform(seed, B_, 512, 4096)
    ks = [int(x) for x in draft_lengths(seed, B_, (3, 5, 7))]
    ids = [int(x) for x in seq_ids_for(seed, B_)]
    prompts = uniform_prompts(seed, ctx, L8B_TARGET.vocab)
    order = np.argsort(ctx)
    check = []
    for kk in (3, 5, 7):
        i = next(int(i) for i in order if ks[i] == kk)
        check.append(ids[i])
    check.append(ids[int(next(i for i in order[1:] if ids[int(i)] not in check))])
    gpu, tgt, drf = _wide_session(wide_pair, B_, 7, 4096 // 16 + 8, 4096)
    say("serving shape: contexts", int(ctx.min()), "..", int(ctx.max()), "checked", check)
    n = _rounds(gpu, tgt, drf, ids, prompts, [0.8] * B_, ks, 3, 23, check, rollback=(0, check[1], 9))
    assert n == 3 * sum(2 * ks[ids.index(s)] + 1 for s in check)
    gpu.close()
