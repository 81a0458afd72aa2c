"""spec_draft_loop (several draft steps in one call, run as one graph) against
the same steps made one spec_draft_step call at a time, in a second context
over the same weights: draft tokens, kept draft logits rows, the verify's
decisions and the committed lengths must agree bit for bit, over rounds whose
repeated shapes replay the captured graphs.  Three paths: bf16 rows fused
into the GEMMs (at most 8 rows per step), bf16 with more than 8 rows (MFMA /
skinny GEMMs, separate RMSNorm and RoPE kernels), and fp32."""

import numpy as np
import pytest

from tests.gpu_util import device, say, torch
from workloads import SMALL_BF16, TINY_FP32, model_weights, seq_ids_for, uniform_prompts

pytestmark = pytest.mark.gpu


def _pair(cfg, lt, ld, max_seqs, pages):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    tw = model_weights(cfg.target, cfg.seed, lt)
    dw = model_weights(cfg.draft, cfg.seed + 1, ld)
    k = max(cfg.k)

    def make():
        return SpecSession(DeviceModel(cfg.target, tw, dev, n_layers=lt), DeviceModel(cfg.draft, dw, dev, n_layers=ld),
                           max_seqs=max_seqs, k_max=k, max_pages_per_seq=pages, max_rows=256)
    return make(), make(), k


def _steps_one_by_one(sess, ids, temps, seed, steps):
    for j in range(max(steps)):
        sub = [i for i, s in enumerate(steps) if s > j]
        sess.draft_step([ids[i] for i in sub], [temps[i] for i in sub], seed)


def _run(cfg, lt, ld, n_seqs, rounds, seed0):
    loop, ref, k = _pair(cfg, lt, ld, max_seqs=n_seqs, pages=24)
    ids = [int(x) for x in seq_ids_for(cfg.seed + 77, n_seqs)]
    prompts = uniform_prompts(cfg.seed + 3, [20 + 9 * i for i in range(n_seqs)], cfg.target.vocab)
    temps = [[0.0, 0.8, 1.0, 0.5][i % 4] for i in range(n_seqs)]
    say("draft loop: prefill", n_seqs, "sequences, k_max", k)
    loop.prefill(ids, prompts)
    ref.prefill(ids, prompts)
    rng = np.random.default_rng(seed0)
    for r in range(rounds):
        # every other round repeats the first round's pattern (graph replay)
        steps = [int(x) for x in (rng.integers(0, k + 1, size=n_seqs) if r % 2 else
                                  [(k - i) % (k + 1) for i in range(n_seqs)])]
        seed = seed0 + r
        say("round", r, "steps", steps)
        loop.draft_loop(ids, temps, seed, steps)
        _steps_one_by_one(ref, ids, temps, seed, steps)
        for sid, s in zip(ids, steps):
            a, b = loop.draft_tokens(sid), ref.draft_tokens(sid)
            assert a == b and len(a) == s, f"round {r} seq {sid}: drafts {a} vs {b}"
            for j in range(s):
                za, zb = loop.draft_logits(sid, j), ref.draft_logits(sid, j)
                assert torch.equal(za, zb), f"round {r} seq {sid} draft {j}: logits differ"
        na, oa = loop.verify(ids, temps, seed)
        nb, ob = ref.verify(ids, temps, seed)
        assert np.array_equal(na, nb) and np.array_equal(oa, ob), f"round {r}: verify differs"
        loop.commit(ids, na)
        ref.commit(ids, nb)
        for sid in ids:
            ia, ib = loop.seq_info(sid), ref.seq_info(sid)
            for key in ("target_len", "draft_len", "pending_pos"):
                assert ia[key] == ib[key], f"round {r} seq {sid}: {key} {ia[key]} vs {ib[key]}"
    loop.close()
    ref.close()


def test_draft_loop_bf16_fused_rows():
    _run(SMALL_BF16, 2, 2, n_seqs=4, rounds=5, seed0=11)


def test_draft_loop_bf16_many_rows():
    _run(SMALL_BF16, 2, 1, n_seqs=12, rounds=3, seed0=21)


def test_draft_loop_fp32():
    _run(TINY_FP32, None, None, n_seqs=3, rounds=3, seed0=31)


def test_draft_loop_rejects_bad_steps():
    from paper_2607_20507_amd import binding as B
    loop, _, k = _pair(TINY_FP32, None, None, max_seqs=2, pages=24)
    ids = [5, 6]
    loop.prefill(ids, uniform_prompts(4, [10, 12], TINY_FP32.target.vocab))
    with pytest.raises(B.SpecError):
        loop.draft_loop(ids, [1.0, 1.0], 1, [k + 1, 1])
    with pytest.raises(B.SpecError):
        loop.draft_loop(ids, [1.0, 1.0], 1, [-1, 1])
    # nothing ran: a full loop still fits
    loop.draft_loop(ids, [1.0, 1.0], 1, [k, k])
    assert [len(loop.draft_tokens(s)) for s in ids] == [k, k]
    with pytest.raises(B.SpecError):
        loop.draft_loop(ids, [1.0, 1.0], 1, [1, 0])
    loop.close()


@pytest.mark.parametrize("which", ["bf16", "fp32"])
def test_verify_commit_draft_matches_separate_calls(which):
    """spec_verify_commit_draft against spec_verify + spec_kv_commit +
    spec_draft_loop made one by one in a second context: decisions, emitted
    tokens, the next round's drafts and their logits rows, and the lengths,
    bit for bit over 4 rounds."""
    cfg, lt, ld, n_seqs = (SMALL_BF16, 2, 2, 3) if which == "bf16" else (TINY_FP32, None, None, 2)
    fused, ref, k = _pair(cfg, lt, ld, max_seqs=n_seqs, pages=24)
    ids = [int(x) for x in seq_ids_for(cfg.seed + 5, n_seqs)]
    prompts = uniform_prompts(cfg.seed + 4, [30 + 11 * i for i in range(n_seqs)], cfg.target.vocab)
    temps = [[0.8, 0.0, 1.0][i % 3] for i in range(n_seqs)]
    fused.prefill(ids, prompts)
    ref.prefill(ids, prompts)
    steps = [k - (i % 2) for i in range(n_seqs)]
    fused.draft_loop(ids, temps, 50, steps)
    ref.draft_loop(ids, temps, 50, steps)
    for r in range(4):
        say("verify+commit+draft round", r)
        na, oa = fused.verify_commit_draft(ids, temps, 60 + r, 51 + r, steps)
        nb, ob = ref.verify(ids, temps, 60 + r)
        ref.commit(ids, nb)
        ref.draft_loop(ids, temps, 51 + r, steps)
        assert np.array_equal(na, nb) and np.array_equal(oa, ob), f"round {r}: verify differs"
        for sid, s in zip(ids, steps):
            assert fused.draft_tokens(sid) == ref.draft_tokens(sid), f"round {r} seq {sid}: drafts differ"
            for j in range(s):
                assert torch.equal(fused.draft_logits(sid, j), ref.draft_logits(sid, j))
            ia, ib = fused.seq_info(sid), ref.seq_info(sid)
            for key in ("target_len", "draft_len", "pending_pos"):
                assert ia[key] == ib[key]
    fused.close()
    ref.close()
