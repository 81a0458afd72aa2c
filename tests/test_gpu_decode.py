"""Plain batched decoding (spec_decode) against the oracle's decode.

* tiny fp32 model in a decode-only context (no draft model): 4 sequences,
  T in {1.0, 0, 0.7, 1.3}, three calls of 8 steps.  Tokens bit-exact up to
  a sequence's first decision the oracle marks as within its margin (at
  least 90% of the decisions compared), lengths and page tables bit-exact,
  the last step's logits within 1e-4 (normwise per row).
* 1B-shaped bf16 model at full width (2 of its 16 layers), decode-only,
  batch 8: each step's logits teacher-forced against the oracle's cached
  forward on the GPU's own tokens, within 2e-2; greedy tokens equal the
  oracle's argmax where its top-2 gap clears the tolerance.
* the same decode in a target/draft context, and the state errors.
"""

import numpy as np
import pytest

from oracle import rule
from oracle.decoder import Decoder, widen
from oracle.session import Session
from tests.gpu_util import device, rel_err, say, torch
from workloads import (LLAMA8B_SHAPED, TINY_FP32, model_weights, prompt_lengths_uniform, seq_ids_for,
                       uniform_prompts)

pytestmark = pytest.mark.gpu

MARGINS = rule.Margins(accept=1e-4, rel=1e-4, gumbel=1e-5, greedy=2e-5)


def B():
    from paper_2607_20507_amd import binding
    return binding


def _decode_only(shape, weights, max_seqs, pages, max_rows=512):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    gpu = SpecSession(DeviceModel(shape, weights, dev, n_layers=len(weights["layers"])), None, max_seqs=max_seqs, k_max=0,
                      max_pages_per_seq=pages, num_pages_target=max_seqs * pages, max_rows=max_rows)
    return gpu


def test_tiny_fp32_decode_only_bit_exact():
    shape = TINY_FP32.target
    w = model_weights(shape, TINY_FP32.seed)
    n, pages = 4, 16
    gpu = _decode_only(shape, w, n, pages)
    ora = Session(Decoder(shape, w), None, n * pages, 0)
    ids = [int(x) for x in seq_ids_for(TINY_FP32.seed + 77, n)]
    lens = [int(x) for x in prompt_lengths_uniform(5, n, 20, 128)]
    prompts = uniform_prompts(TINY_FP32.seed + 1, lens, shape.vocab)
    temps = [1.0, 0.0, 0.7, 1.3]
    say("decode tiny fp32 prefill", ids, lens)
    gpu.prefill(ids, prompts)
    ora.prefill(ids, prompts)
    in_sync = {sid: True for sid in ids}
    compared = total = 0
    for call in range(3):
        seed = 900 + call
        say("decode tiny fp32 call", call)
        gt = gpu.decode(ids, temps, seed, 8)
        ot, ex, zl = ora.decode(ids, temps, seed, 8, MARGINS)
        zg = gpu.last_logits().cpu().numpy()
        for i, sid in enumerate(ids):
            for j in range(8):
                total += 1
                if not in_sync[sid]:
                    continue
                if ex[i][j]:
                    in_sync[sid] = False  # the GPU may take the other side of the margin
                    continue
                assert gt[i, j] == ot[i][j], (sid, call, j)
                compared += 1
            if in_sync[sid]:
                assert rel_err(zg[i], zl[-1][i]) < 1e-4
            info = gpu.seq_info(sid)
            lt, ld = ora.lengths(sid)
            pt, pd = ora.pages(sid)
            assert (info["target_len"], info["draft_len"]) == (lt, 0)
            assert info["pages_target"] == pt and info["pages_draft"] == []
    say("decode tiny fp32", {"compared": compared, "total": total})
    assert compared >= 0.9 * total


def test_bf16_1b_width_decode_teacher_forced():
    shape = LLAMA8B_SHAPED.draft
    L = 2
    w = model_weights(shape, LLAMA8B_SHAPED.seed + 1, L)
    n, pages = 8, 32
    gpu = _decode_only(shape, w, n, pages)
    dec = Decoder(shape, w)
    ids = [int(x) for x in seq_ids_for(31, n)]
    lens = [int(x) for x in prompt_lengths_uniform(31, n, 100, 300)]
    prompts = uniform_prompts(31, lens, shape.vocab)
    say("decode bf16 1b-width prefill", lens)
    gpu.prefill(ids, prompts)
    kvs, pending = [], []
    for p in prompts:
        kv = dec.new_kv()
        dec.forward(kv, p[:-1], np.arange(len(p) - 1), logits=False)
        kvs.append(kv)
        pending.append(int(p[-1]))
    temps = [0.0, 0.8] * (n // 2)
    wlm = widen(w["lm_head"])  # the LM head in float64, widened once for all steps
    worst, greedy_checked = 0.0, 0
    for step in range(4):
        say("decode bf16 1b-width step", step)
        toks = gpu.decode(ids, temps, 40 + step, 1)
        zg = gpu.last_logits().cpu().numpy()
        for i in range(n):
            pos = kvs[i].length
            zo = dec.forward(kvs[i], [pending[i]], [pos], logits=False)[0] @ wlm.T
            e = rel_err(zg[i], zo)
            worst = max(worst, e)
            assert e < 2e-2, (i, step, e)
            if temps[i] == 0.0:
                top2 = np.sort(zo)[-2:]
                if top2[1] - top2[0] > 2 * 2e-2 * np.abs(zo).max():
                    assert toks[i, 0] == int(np.argmax(zo))
                    greedy_checked += 1
            pending[i] = int(toks[i, 0])
    say("decode bf16 1b-width", {"max_rel_err": worst, "greedy_checked": greedy_checked})


def test_decode_in_a_pair_context_and_state_errors():
    """spec_decode on the target of a target/draft context equals the
    decode-only context's result; drafts pending, or drafting in a
    decode-only context, are state errors."""
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    b = B()
    cfg = TINY_FP32
    tw = model_weights(cfg.target, cfg.seed)
    dw = model_weights(cfg.draft, cfg.seed)
    pair = SpecSession(DeviceModel(cfg.target, tw, dev), DeviceModel(cfg.draft, dw, dev), max_seqs=2,
                       k_max=4, max_pages_per_seq=16, max_rows=256)
    alone = _decode_only(cfg.target, tw, 2, 16)
    ids = [5, 9]
    prompts = uniform_prompts(3, [40, 17], cfg.target.vocab)
    pair.prefill(ids, prompts)
    alone.prefill(ids, prompts)
    say("decode pair vs decode-only")
    a = pair.decode(ids, [1.0, 0.0], 7, 6)
    c = alone.decode(ids, [1.0, 0.0], 7, 6)
    np.testing.assert_array_equal(a, c)
    # drafting then decoding is a state error; nothing runs
    pair.draft_step(ids, [1.0, 1.0], 1)
    with pytest.raises(b.SpecError) as e:
        pair.decode(ids, [1.0, 1.0], 7, 1)
    assert e.value.status == b.SPEC_E_STATE
    with pytest.raises(b.SpecError) as e:
        alone.draft_step(ids, [1.0, 1.0], 1)
    assert e.value.status == b.SPEC_E_STATE
    # the decode-only context still decodes after the refused call
    alone.decode(ids, [1.0, 0.0], 8, 2)
    torch.cuda.synchronize()
