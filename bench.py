#!/usr/bin/env python3
"""Verified tokens/s and verify-step latency of draft-and-verify on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one pass of the whole hot path on one batch: k draft steps, the
verify (target forward over the k+1 rows of every sequence, logits, decision
pass) and the KV commit / rollback.  Inputs (random-init weights, prompts)
are synthetic, seeded and resident in HBM before the timed region.

Workloads:
  all (default) the 8b-shaped line below, with sub-objects: the same sequence
                at T = 0 ("greedy"), plain target decode with k = 0
                ("plain_decode"), the serving batch ("serving"), the 1b-shaped
                model decoding 64 sequences by itself ("small_decode"), a
                15-node draft tree against the 5-draft chain ("tree_verify"),
                long-context prefill of 2048 to 8192 tokens ("prefill") and
                the decision pass alone ("vocab_stress"), each with its own
                timing (and roofline and oracle baseline where one is timed).
  8b-shaped     32-layer d=4096 target (32/8 heads, ffn 14336, vocab 128256),
                16-layer d=2048 drafter, batch 1, 2048-token context, k = 5,
                T = 0.8 (default) or --temperature 0 for greedy.
  8b-serving    the same pair serving 64 sequences (contexts log-uniform in
                [512, 4096], k in {3, 5, 7}, drafts mixed toward the target's
                top-1 off the clock), greedy by default.
  vocab-stress  the decision pass alone: 256 sequences x (7 + 1) rows x 128256.

Prints one JSON line: metric, value (verified tokens/s, whole job), latency,
roofline of the dominant kernel (live HIP-event timing through the library's
kernel timer), and one whole float64 oracle step timed on the host.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def pmc_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` measured by the profiler's FETCH_SIZE and
    WRITE_SIZE counters (scaled by a copy of known size), from the committed
    summaries under profiles/; None unless the kernel's source is unchanged
    since the counters were taken."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", "pmc_*.txt")):
        fields = {}
        with open(path) as f:
            for line in f:
                if ": " in line and not line.startswith((" ", "#")):
                    key, val = line.rstrip("\n").split(": ", 1)
                    fields[key] = val
        if fields.get("kernel") != kernel or fields.get("workload") != workload:
            continue
        try:
            with open(os.path.join(ROOT, fields["source"]), "rb") as f:
                if hashlib.sha256(f.read()).hexdigest() != fields["source_sha256"]:
                    return None
            return float(fields["traffic_bytes_per_launch"])
        except (OSError, KeyError, ValueError):
            return None
    return None


def cpu_info():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    threads = None
    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"), default=None)
    except Exception:
        pass
    aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return model, threads or aff, aff


def roofline_pass(B, sess, kernel, step, args):
    """Per-kernel timing: the timed steps replay captured graphs, in which a
    single launch cannot be bracketed by events, so `roof_steps` further steps
    of the same workload run with the library's kernel timer on (eager
    launches), which records kernel-level start / end events on every launch
    of `kernel`."""
    B.spec_timing_enable(sess.ctx, kernel)
    for s in range(args.roof_steps):
        step(args.warmup + args.steps + s, False)
    out = B.spec_timing_read(sess.ctx)
    B.spec_timing_enable(sess.ctx, None)
    return out


# ---------------------------------------------------------------------------
# 8B-shaped pair, batch 1

def device_models(cfg):
    import torch
    from paper_2607_20507_amd.session import DeviceModel
    log("drawing weights on device")
    dev = torch.device("cuda:0")
    return (DeviceModel(cfg.target, None, dev, seed=cfg.seed),
            DeviceModel(cfg.draft, None, dev, seed=cfg.seed + 1))


def timed_rounds(stream, n, fn):
    """Run fn(i) for i < n between a host clock and HIP events; fn returns
    (tokens emitted, accepted drafts).  Returns (tokens, wall s, event ms,
    accepted list)."""
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    tokens, acc = 0, []
    for i in range(n):
        t, a = fn(i)
        tokens += t
        acc.append(a)
    ev1.record(stream)
    torch.cuda.synchronize()
    return tokens, time.perf_counter() - t0, ev0.elapsed_time(ev1), acc


def bench_8b(args, target, draft, extras=False):
    import torch
    from paper_2607_20507_amd import binding as B
    from paper_2607_20507_amd.session import SpecSession
    from workloads import LLAMA8B_SHAPED, seq_ids_for, uniform_prompts

    cfg = LLAMA8B_SHAPED
    k = cfg.k[0]
    T = args.temperature
    ctx_len = cfg.context[1]
    total_steps = args.warmup + 2 * args.steps + args.roof_steps + 1  # + the latency rounds and round 0
    if extras:  # greedy rounds and plain-decode steps on the same sequence
        total_steps += 2 * (args.warmup + args.steps) + 1
    max_len = ctx_len + total_steps * (k + 1) + 64
    pages = (max_len + 15) // 16
    sess = SpecSession(target, draft, max_seqs=1, k_max=k, max_pages_per_seq=pages, max_rows=2048)
    sid = int(seq_ids_for(cfg.seed, 1)[0])
    stream = torch.cuda.current_stream()
    prompt = uniform_prompts(cfg.seed, [ctx_len], cfg.target.vocab)[0]
    log("prefill", ctx_len)
    sess.prefill([sid], [prompt])
    acc_hist = []
    lat = []

    # A step is one round: verify the pending k drafts, commit, and draft the
    # next round's k, in one library call (the host round trip between the
    # verify's outputs and the next drafts stays inside the library).  Round
    # 0's drafts are made before the warm-up.
    def step(s, record):
        na, _ = sess.verify_commit_draft([sid], [T], cfg.seed + s, cfg.seed + s + 1, [k])
        if record:
            acc_hist.append(int(na[0]))
        return int(na[0]) + 1

    sess.draft_loop([sid], [T], cfg.seed, [k])
    for s in range(args.warmup):
        step(s, False)
    kernel = args.kernel or "gemm_skinny_bf16<1, 2, true>"
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    tokens = 0
    for s in range(args.steps):
        tokens += step(args.warmup + s, True)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = ev0.elapsed_time(ev1)
    k_ms, k_n, k_bytes, k_flops = roofline_pass(B, sess, kernel, step, args)
    # verify-step latency (spec_verify + spec_kv_commit between HIP events),
    # from rounds made with the separate calls after the timed region
    for s in range(args.steps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        na, _ = sess.verify([sid], [T], cfg.seed + 1000 + s)
        sess.commit([sid], na)
        e1.record(stream)
        lat.append((e0, e1))
        sess.draft_loop([sid], [T], cfg.seed + 1001 + s, [k])
    torch.cuda.synchronize()
    lats = sorted(a.elapsed_time(b) for a, b in lat)
    info = {
        "tokens": tokens, "wall_s": wall, "event_ms": ev_ms, "acc_hist": acc_hist,
        "verify_ms_median": float(np.median(lats)), "verify_ms_p90": float(np.percentile(lats, 90)),
        "verify_latency": (f"HIP events around spec_verify + spec_kv_commit, {args.steps} rounds made with "
                           "separate calls after the timed region (the timed steps use spec_verify_commit_draft)"),
        "kernel": kernel, "k_ms": k_ms, "k_n": k_n, "k_bytes": k_bytes, "k_flops": k_flops,
        "weights_gb_per_step": (cfg.target.weight_bytes_per_forward() + k * cfg.draft.weight_bytes_per_forward()) / 1e9,
    }
    if extras:
        base = cfg.seed + 5000

        # greedy (T = 0) rounds of the same sequence, one call per round
        def greedy(i):
            na, _ = sess.verify_commit_draft([sid], [0.0], base + 2 * i, base + 2 * i + 1, [k])
            return int(na[0]) + 1, int(na[0])

        for i in range(args.warmup):
            greedy(i)
        g_tok, g_wall, g_ev, g_acc = timed_rounds(stream, args.steps, lambda i: greedy(args.warmup + i))
        info["greedy"] = {"value": g_tok / g_wall, "unit": "tokens/s", "ms_per_step": g_wall * 1e3 / args.steps,
                          "event_ms_per_step": g_ev / args.steps, "steps": args.steps, "temperature": 0.0,
                          "mean_accepted": float(np.mean(g_acc))}
        # plain target decode (k = 0): each step is a one-row verify, which
        # emits the target's own next token, and its commit; no drafting.
        # The first call verifies the pending drafts and drafts none.
        base += 1000
        sess.verify_commit_draft([sid], [T], base, base + 1, [0])

        def plain(i):
            sess.verify_commit_draft([sid], [T], base + 2 + i, base + 3 + i, [0])
            return 1, 0

        for i in range(args.warmup):
            plain(i)
        p_tok, p_wall, p_ev, _ = timed_rounds(stream, args.steps, lambda i: plain(args.warmup + i))
        info["plain_decode"] = {"value": p_tok / p_wall, "unit": "tokens/s", "ms_per_step": p_wall * 1e3 / args.steps,
                                "event_ms_per_step": p_ev / args.steps, "steps": args.steps, "temperature": T,
                                "what": "target alone, one token per step: spec_verify_commit_draft with k = 0 "
                                        "(a one-row target forward, the decision pass's bonus draw, the commit)"}
    sess.close()
    return info


def oracle_models():
    """The float64 oracle decoders of the 8B-shaped pair for the CPU timing.
    Every layer of a model is the same layer, drawn from its seed (the cost of
    a forward does not depend on the weight values, and drawing 32 distinct
    layers would take minutes of host time); the embedding is the LM head."""
    from oracle import decoder as OD
    from workloads import LLAMA8B_SHAPED
    from workloads.gen import layer_weights, _normal, _ones

    cfg = LLAMA8B_SHAPED
    log("oracle: drawing one layer + LM head of each model")

    def model(shape, seed):
        lm = _normal(seed, shape, "lm_head", 0, (shape.vocab, shape.d_model))
        lw = layer_weights(shape, seed, 0)
        return OD.Decoder(shape, {"embed": lm, "final_norm": _ones(shape, shape.d_model), "lm_head": lm,
                                  "layers": [lw] * shape.n_layers})

    return model(cfg.target, cfg.seed), model(cfg.draft, cfg.seed + 1)


def cpu_full_step(tdec, ddec, ctx, k, T, seed):
    """One whole oracle step of one sequence, timed on the host: k drafter
    forwards of one row each over a cache of ctx positions (with LM head and
    draft draw), the target forward over the k + 1 verify rows, its LM head,
    and the rule.  The caches hold ctx positions of random keys and values
    (set up before the clock starts)."""
    from oracle import rule

    rng = np.random.default_rng(seed)

    def filled(dec):
        kv = dec.new_kv()
        sh = dec.shape
        for l in range(dec.n_layers):
            kv.append(l, rng.standard_normal((ctx, sh.n_kv_heads, sh.head_dim)),
                      rng.standard_normal((ctx, sh.n_kv_heads, sh.head_dim)))
        return kv

    tkv, dkv = filled(tdec), filled(ddec)
    pending = int(rng.integers(0, tdec.shape.vocab))
    t0 = time.perf_counter()
    tok, drafts, zq = pending, [], []
    for j in range(k):
        z = ddec.forward(dkv, [tok], [ctx + j])[0]
        tok = rule.sample_draft(z, T, seed, 1, ctx + j + 1)[0]
        drafts.append(int(tok))
        zq.append(z)
    t1 = time.perf_counter()
    zp = tdec.forward(tkv, [pending] + drafts, ctx + np.arange(k + 1))
    t2 = time.perf_counter()
    res = rule.verify(zp, np.array(zq), drafts, T, seed, 1, ctx)
    t3 = time.perf_counter()
    return {"step_s": t3 - t0, "draft_s": t1 - t0, "target_forward_s": t2 - t1, "rule_s": t3 - t2,
            "accepted": int(res.n_accepted)}


def cpu_baseline_8b(mean_tokens_per_step, models):
    from workloads import LLAMA8B_SHAPED
    cfg = LLAMA8B_SHAPED
    log("oracle: one full batch-1 step")
    r = cpu_full_step(*models, cfg.context[1], cfg.k[0], 0.8, cfg.seed)
    return {"value": mean_tokens_per_step / r["step_s"], "step_s": r["step_s"], "sample_s": r["step_s"],
            "parts_s": {x: r[x] for x in ("draft_s", "target_forward_s", "rule_s")},
            "sample": ("one whole oracle step (float64): 5 drafter steps of 16 layers + LM head + draw, the "
                       "32-layer target forward over the 6 verify rows + LM head, and the rule, over caches of "
                       "2048 random positions; each model's layers share one seeded layer's weights")}


# ---------------------------------------------------------------------------
# 8B-shaped pair, serving batch of 64 sequences

def bench_serving(args, target, draft, T):
    import torch
    from paper_2607_20507_amd import binding as B
    from paper_2607_20507_amd.session import SpecSession
    from workloads import (SERVING_8B, context_lengths_loguniform, draft_lengths, mix_draws, seq_ids_for,
                           uniform_prompts)

    cfg = SERVING_8B
    n = cfg.batch
    ctx = context_lengths_loguniform(cfg.seed, n, cfg.context[1], cfg.context[2])
    ks = draft_lengths(cfg.seed, n, cfg.k)
    kmax = int(max(cfg.k))
    ids = [int(x) for x in seq_ids_for(cfg.seed, n)]
    total_steps = args.warmup + args.steps + args.roof_steps
    max_len = int(ctx.max()) + total_steps * (kmax + 1) + 64
    pages = (max_len + 15) // 16
    need = int(sum((int(c) + total_steps * (kmax + 1) + 64 + 15) // 16 for c in ctx))
    sess = SpecSession(target, draft, max_seqs=n, k_max=kmax, max_pages_per_seq=pages,
                       num_pages_target=need, num_pages_draft=need, max_rows=4096)
    prompts = uniform_prompts(cfg.seed, [int(c) for c in ctx], cfg.target.vocab)
    log("prefill", int(ctx.sum()), "tokens")
    sess.prefill(ids, prompts)
    stream = torch.cuda.current_stream()
    temps = [T] * n
    acc_hist, lat, on_clock = [], [], []
    roof = {"kernel": None, "acc": []}  # per-kernel timing of the verify only (roofline steps)
    pend = {ids[i]: int(ctx[i]) - 1 for i in range(n)}  # pending-token position n of each sequence
    mix = cfg.mix_rate > 0 and not args.no_mix
    V = cfg.target.vocab

    def step(s, record):
        # Draft mixing (off the clock): before drafting position n + j the
        # target's top-1 token there comes from the target forward over the
        # pending token and the drafts so far; with probability mix_rate
        # (seeded per sequence and position) the draft is guided to it.  Only
        # the draft steps, the verify and the commit are timed, on the GPU
        # clock between events.
        spans = []
        for j in range(1, kmax + 1):
            live = [ids[i] for i in range(n) if ks[i] >= j]
            if mix:
                sess.target_forward(live)
                z = sess.last_logits()
                top1 = torch.argmax(z.view(len(live), j, V)[:, j - 1, :], dim=1).to(torch.int32).cpu().numpy()
                pos = [pend[sid] + j for sid in live]
                guide = np.where(mix_draws(cfg.seed + s, live, pos, cfg.mix_rate), top1, -1).astype(np.int32)
                torch.cuda.synchronize()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(stream)
            if mix:
                sess.draft_step_guided(live, [T] * len(live), cfg.seed + s, guide, cfg.mix_boost)
            else:
                sess.draft_step(live, [T] * len(live), cfg.seed + s)
            b.record(stream)
            spans.append((a, b))
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        if roof["kernel"]:
            B.spec_timing_enable(sess.ctx, roof["kernel"])
        na, _ = sess.verify(ids, temps, cfg.seed + s)
        if roof["kernel"]:
            roof["acc"].append(B.spec_timing_read(sess.ctx))
            B.spec_timing_enable(sess.ctx, None)
        sess.commit(ids, na)
        e1.record(stream)
        spans.append((e0, e1))
        for i, sid in enumerate(ids):
            pend[sid] += int(na[i]) + 1
        if record:
            acc_hist.extend(int(x) for x in na)
            lat.append((e0, e1))
            on_clock.append(spans)
        return int(na.sum()) + n

    for s in range(args.warmup):
        step(s, False)
    kernel = args.kernel or "gemm_mfma3_bf16<2, 12, 4, 4>"
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    tokens = 0
    for s in range(args.steps):
        tokens += step(args.warmup + s, True)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    event_ms = ev0.elapsed_time(ev1)
    clock_ms = sum(a.elapsed_time(b) for spans in on_clock for a, b in spans)
    # roofline steps: the verify's launches of `kernel` only (the drafter's
    # 64-row gate/up and the off-clock target forwards use the same kernel)
    roof["kernel"] = kernel
    for s in range(args.roof_steps):
        step(args.warmup + args.steps + s, False)
    k_ms, k_n, k_bytes, k_flops = (sum(x[i] for x in roof["acc"]) for i in range(4))
    lats = sorted(a.elapsed_time(b) for a, b in lat)
    sess.close()
    # with mixing, the timed work is the on-clock spans only
    return {"tokens": tokens, "wall_s": (clock_ms / 1e3) if mix else wall, "event_ms": event_ms,
            "acc_hist": acc_hist, "mix": mix, "offclock_ms": event_ms - clock_ms if mix else 0.0,
            "verify_ms_median": float(np.median(lats)), "verify_ms_p90": float(np.percentile(lats, 90)),
            "kernel": kernel, "k_ms": k_ms, "k_n": k_n, "k_bytes": k_bytes, "k_flops": k_flops,
            "mean_ctx": float(ctx.mean()), "rows_per_verify": int((ks + 1).sum()),
            "ctx": ctx, "ks": ks}


# ---------------------------------------------------------------------------
# long-context prefill

def bench_prefill(args, target):
    """Prefill of one prompt of 2048, 4096 and 8192 tokens through the 32-layer
    8B-shaped target (a decode-only context over the same weights; chunks of
    up to 8192 rows), the paper's length range.  Each length is prefilled
    `warmup` times untimed, then timed `reps` times (host clock around the
    call, which returns when the work is done); the large-M gate/up GEMM and
    the causal prefill attention are timed at kernel level on one more
    prefill of 8192 tokens."""
    import torch
    from paper_2607_20507_amd import binding as B
    from paper_2607_20507_amd.session import SpecSession
    from workloads import LLAMA8B_SHAPED, uniform_prompts

    cfg = LLAMA8B_SHAPED
    V = cfg.target.vocab
    reps = max(2, min(args.steps, 5))
    sess = SpecSession(target, None, max_seqs=1, k_max=0, max_pages_per_seq=8192 // 16 + 2, max_rows=8192)
    out = {}
    for P in (2048, 4096, 8192):
        prompt = uniform_prompts(cfg.seed + P, [P + 1], V)[0]
        times = []
        for r in range(max(1, args.warmup) + reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            sess.prefill([1], [prompt])
            t = time.perf_counter() - t0
            sess.release(1)
            if r >= max(1, args.warmup):
                times.append(t)
        ms = float(np.median(times)) * 1e3
        out[str(P)] = {"ms": ms, "tokens_per_s": P / (ms / 1e3),
                       "tflops": 2.0 * P * cfg.target.layer_params() * cfg.target.n_layers / (ms / 1e3) / 1e12}
    prompt = uniform_prompts(cfg.seed + 8192, [8193], V)[0]
    roof = {}
    for kernel, bound in (("gemm_mfma3_bf16<2, 12, 4, 4>", "mfma"), ("attn_prefill_bf16_kernel<128>", "mfma")):
        B.spec_timing_enable(sess.ctx, kernel)
        sess.prefill([1], [prompt])
        sess.release(1)
        k_ms, k_n, k_bytes, k_flops = B.spec_timing_read(sess.ctx)
        B.spec_timing_enable(sess.ctx, None)
        info = {"kernel": kernel, "k_ms": k_ms, "k_n": k_n, "k_bytes": k_bytes, "k_flops": k_flops}
        roof[kernel] = roofline_of(info, bound, "prefill-8192", 1, " (one 8192-token prefill)")
    sess.close()
    out["roofline"] = roof["gemm_mfma3_bf16<2, 12, 4, 4>"]
    out["attention"] = roof["attn_prefill_bf16_kernel<128>"]
    out["config"] = {"workload": "8b-shaped target prefill of one prompt (2048, 4096, 8192 tokens; positions "
                                 "0..P-1 into the paged cache, no LM head), chunks of up to 8192 rows",
                     "tflops_counts": "2 x parameters of the 32 layers per token (attention excluded)"}
    return out


# ---------------------------------------------------------------------------
# tree verification at batch 1

def bench_tree(args, target, draft):
    """Verify rounds of a 15-node draft tree (3 candidates, 2 under each, one
    under each of those: depth 3) against the 5-draft chain, on the 8B-shaped
    target at context 2048.  Drafts are external (seeded tokens and draft
    logits): the measured cost is the target's forward over the tree rows and
    the tree decision, whatever proposer made the tree."""
    import torch
    from paper_2607_20507_amd import binding as B
    from paper_2607_20507_amd.session import SpecSession
    from workloads import LLAMA8B_SHAPED, uniform_prompts

    cfg = LLAMA8B_SHAPED
    V = cfg.target.vocab
    parents, level = [], [-1]
    for b in (3, 2, 1):
        nxt = []
        for u in level:
            for _ in range(b):
                parents.append(u)
                nxt.append(len(parents) - 1)
        level = nxt
    m = len(parents)
    rounds = args.warmup + args.steps + args.roof_steps
    ctx_len = cfg.context[1]
    pages = (ctx_len + rounds * (m + 1) + 64 + 15) // 16
    sess = SpecSession(target, draft, max_seqs=1, k_max=m, max_pages_per_seq=pages, max_rows=2048)
    sid = 77
    sess.prefill([sid], [uniform_prompts(cfg.seed + 3, [ctx_len], V)[0]])
    g = torch.Generator(device="cuda:0")
    g.manual_seed(cfg.seed)
    zq = torch.randn(m + 1, V, generator=g, device="cuda:0")
    rng = np.random.default_rng(cfg.seed)
    stream = torch.cuda.current_stream()
    out = {}
    for name, shape in (("tree", parents), ("chain", list(range(-1, 4)))):
        lat, acc = [], []
        for r in range(args.warmup + args.steps):
            toks = [int(x) for x in rng.integers(0, V, size=len(shape))]
            sess.set_draft_tree(sid, shape, toks, zq)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            na, _ = sess.verify([sid], [0.8], cfg.seed + r)
            sess.commit([sid], na)
            e1.record(stream)
            if r >= args.warmup:
                lat.append((e0, e1))
                acc.append(int(na[0]))
        torch.cuda.synchronize()
        ls = sorted(a.elapsed_time(b) for a, b in lat)
        out[name] = {"nodes": len(shape), "verify_ms_median": float(np.median(ls)),
                     "verify_ms_p90": float(np.percentile(ls, 90)), "mean_accepted": float(np.mean(acc))}
    # the tree decision after the statistics pass alone (residual-mass passes,
    # draws and walk; kernel-level events around them)
    B.spec_timing_enable(sess.ctx, "tree_decision")
    for r in range(args.roof_steps):
        sess.set_draft_tree(sid, parents, [int(x) for x in rng.integers(0, V, size=m)], zq)
        na, _ = sess.verify([sid], [0.8], cfg.seed + 500 + r)
        sess.commit([sid], na)
    k_ms, k_n, _, _ = B.spec_timing_read(sess.ctx)
    B.spec_timing_enable(sess.ctx, None)
    sess.close()
    out["tree"]["decide_us"] = k_ms * 1e3 / max(1, k_n)
    out["config"] = {"workload": "8b-shaped target, batch 1, context 2048, T = 0.8: a 15-node draft tree "
                                 "(branching 3, 2, 1) against a 5-draft chain, external seeded drafts",
                     "parents": parents}
    return out


# ---------------------------------------------------------------------------
# the small model decoding by itself, batched

def bench_small_decode(args, small):
    """Plain batched decoding of the 1B-shaped model in a decode-only context
    that shares its weights: 64 sequences with the serving workload's
    contexts, T = 0.8, one token per sequence per step (spec_decode)."""
    import torch
    from paper_2607_20507_amd import binding as B
    from paper_2607_20507_amd.session import SpecSession
    from workloads import SERVING_8B, context_lengths_loguniform, seq_ids_for, uniform_prompts

    cfg = SERVING_8B
    n = cfg.batch
    ctx = context_lengths_loguniform(cfg.seed, n, cfg.context[1], cfg.context[2])
    ids = [int(x) for x in seq_ids_for(cfg.seed + 7, n)]
    total = args.warmup + args.steps + args.roof_steps
    pages = (int(ctx.max()) + total + 16 + 15) // 16
    need = int(sum((int(c) + total + 16 + 15) // 16 for c in ctx))
    sess = SpecSession(small, None, max_seqs=n, k_max=0, max_pages_per_seq=pages, num_pages_target=need,
                       max_rows=4096)
    prompts = uniform_prompts(cfg.seed + 7, [int(c) for c in ctx], cfg.draft.vocab)
    log("small-model decode: prefill", int(ctx.sum()), "tokens")
    sess.prefill(ids, prompts)
    stream = torch.cuda.current_stream()
    temps = [0.8] * n
    sess.decode(ids, temps, cfg.seed, args.warmup)
    # one call decodes every timed step (the library loops over the steps)
    tok, wall, ev, _ = timed_rounds(stream, 1, lambda i: (sess.decode(ids, temps, cfg.seed + 1, args.steps).size, 0))
    kernel = args.kernel or "attn_bf16_kernel<64, 1, 4>"
    B.spec_timing_enable(sess.ctx, kernel)
    sess.decode(ids, temps, cfg.seed + 2, args.roof_steps)
    k_ms, k_n, k_bytes, k_flops = B.spec_timing_read(sess.ctx)
    B.spec_timing_enable(sess.ctx, None)
    sess.close()
    return {"tokens": tok, "wall_s": wall, "event_ms": ev, "kernel": kernel, "k_ms": k_ms, "k_n": k_n,
            "k_bytes": k_bytes, "k_flops": k_flops, "mean_ctx": float(ctx.mean())}


# ---------------------------------------------------------------------------
# decision pass alone

def bench_vocab(args):
    import torch
    from paper_2607_20507_amd import binding as B
    from workloads import VOCAB_STRESS, base_positions, seq_ids_for, vocab_temperatures

    cfg = VOCAB_STRESS
    dev = torch.device("cuda:0")
    Bn, k, V = cfg.batch, cfg.k, cfg.vocab
    g = torch.Generator(device=dev)
    g.manual_seed(cfg.seed)
    P = torch.randn(Bn * (k + 1), V, generator=g, device=dev) * cfg.p_std
    Q = P.view(Bn, k + 1, V)[:, :k].reshape(Bn * k, V) + torch.randn(Bn * k, V, generator=g, device=dev) * cfg.q_noise_std
    temps = vocab_temperatures(Bn, cfg.temperatures)
    ids = seq_ids_for(cfg.seed, Bn)
    base = base_positions(cfg.seed, Bn, *cfg.base_pos_range)
    drafts = torch.zeros(Bn * k, dtype=torch.int32, device=dev)
    wsd = torch.empty(16 << 20, dtype=torch.uint8, device=dev)
    B.spec_sample_draft(Q, V, np.repeat(temps, k), np.repeat(ids, k),
                        np.concatenate([base[s] + 1 + np.arange(k) for s in range(Bn)]), cfg.seed, drafts, wsd)
    # every call writes its own outputs, so the timed calls go back to back
    # (each one's host work overlaps the previous one's kernels); the per-call
    # latency is measured after, one synchronised call at a time
    n_out = max(1, args.warmup + 2 * args.steps + args.roof_steps)
    na = torch.zeros(n_out, Bn, dtype=torch.int32, device=dev)
    out = torch.zeros(n_out, Bn, k + 1, dtype=torch.int32, device=dev)
    ws = torch.empty(B.spec_sample_workspace_bytes(Bn, Bn * (2 * k + 1), V), dtype=torch.uint8, device=dev)
    ks = np.full(Bn, k, dtype=np.int32)  # host arrays in the C types: no per-call conversion

    def step(s):
        B.spec_sample_verify(ks, temps, ids, base, P, Q, drafts, V, cfg.seed + s, na[s], out[s], ws)

    for s in range(args.warmup):
        step(s)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for s in range(args.steps):
        step(args.warmup + s)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    acc_all = na[args.warmup:args.warmup + args.steps].cpu().numpy()
    tokens = int(acc_all.sum()) + Bn * args.steps
    # early-exit accounting: rows up to the first rejection (p rows 0..a,
    # q rows 0..min(a, k-1)); the parallel pass reads all 2k + 1 rows
    early_rows = int(np.sum(acc_all + 1 + np.minimum(acc_all + 1, k)))
    lats = []
    for s in range(args.steps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step(args.warmup + args.steps + s)
        b.record(stream)
        torch.cuda.synchronize()
        lats.append(a.elapsed_time(b))
    kernel = args.kernel or "stats_kernel<true>"
    B.spec_timing_enable(None, kernel)
    for s in range(args.roof_steps):
        step(args.warmup + 2 * args.steps + s)
    torch.cuda.synchronize()
    k_ms, k_n, k_bytes, k_flops = B.spec_timing_read(None)
    B.spec_timing_enable(None, None)
    ls = sorted(lats)
    return {"tokens": tokens, "wall_s": wall, "event_ms": ev0.elapsed_time(ev1),
            "verify_ms_median": float(np.median(ls)), "verify_ms_p90": float(np.percentile(ls, 90)),
            "verify_latency": "HIP events around one spec_sample_verify call, synchronised, from an idle GPU "
                              "(includes the host's table layout and upload)",
            "kernel": kernel, "k_ms": k_ms, "k_n": k_n, "k_bytes": k_bytes, "k_flops": k_flops,
            "acc_hist": [],
            "vocab_bytes": {"read_per_step": 4.0 * V * Bn * (2 * k + 1),
                            "early_exit_per_step": 4.0 * V * early_rows / args.steps,
                            "note": "logit rows the parallel pass reads (all k + 1 p rows and k q rows) "
                                    "vs the rows an early-exit scan would need (p rows 0..a, q rows "
                                    "0..min(a, k-1)); the rejected or bonus row's second read is not counted"}}


def cpu_baseline_vocab(mean_tokens_per_step):
    """The oracle rule (float64) on the whole batch: for each of the 256
    sequences, its k draft draws and the acceptance / resample decision, on
    the same synthetic logit law (drawn on the host, 32 sequences at a time,
    outside the clock)."""
    from oracle import rule
    from workloads import VOCAB_STRESS, vocab_logits

    cfg = VOCAB_STRESS
    dt = 0.0
    for s0 in range(0, cfg.batch, 32):
        seqs = list(range(s0, min(cfg.batch, s0 + 32)))
        p, q = vocab_logits(cfg.seed, seqs, cfg.k, cfg.vocab)
        t0 = time.perf_counter()
        for i, s in enumerate(seqs):
            T = cfg.temperatures[s % 3]
            drafts = [rule.sample_draft(q[i, j], T, 1, s, 100 + j + 1)[0] for j in range(cfg.k)]
            rule.verify(p[i], q[i], drafts, T, 1, s, 100)
        dt += time.perf_counter() - t0
    return {"value": mean_tokens_per_step / dt, "step_s": dt, "sample_s": dt,
            "sample": "draft draws + rule on all 256 sequences (one whole step)"}


def roofline_of(info, bound, workload, roof_steps, note=""):
    """Roofline object of a workload's dominant kernel from its kernel-level
    event timing: algorithmic bytes (or flops) per launch / average launch."""
    n = info["k_n"]
    per_launch_ms = info["k_ms"] / max(1, n)
    if bound == "mfma":
        achieved = (info["k_flops"] / n) / (per_launch_ms / 1e3) / 1e12 if n else None
        peak, unit = BF16_PEAK_TFLOPS, "TFLOP/s"
    else:
        achieved = (info["k_bytes"] / n) / (per_launch_ms / 1e3) / 1e9 if n else None
        peak, unit = HBM_PEAK_GBS, "GB/s"
    r = {"bound": bound, "kernel": info["kernel"], "achieved": achieved, "peak": peak, "unit": unit,
         "frac": (achieved / peak) if achieved else None, "traffic": pmc_traffic(info["kernel"], workload),
         "launches": n, "avg_launch_us": per_launch_ms * 1e3,
         "timing": f"kernel-level HIP events (start and end of each launch of the kernel), "
                   f"{roof_steps} eager steps after the timed region" + note,
         "bytes_per_launch": info["k_bytes"] / max(1, n), "flops_per_launch": info["k_flops"] / max(1, n)}
    if bound == "hbm" and info["k_flops"] and n:
        r["tflops"] = info["k_flops"] / (info["k_ms"] / 1e3) / 1e12
    if bound == "mfma" and n:
        r["gbs"] = info["k_bytes"] / (info["k_ms"] / 1e3) / 1e9
    return r


def cpu_line(cb, threads, model, aff):
    out = {"value": cb["value"], "unit": "tokens/s", "cores": threads, "kind": "oracle", "sample": cb["sample"],
           "sample_s": cb["sample_s"], "est_step_s": cb["step_s"], "cpu": model, "affinity": aff}
    if "parts_s" in cb:
        out["parts_s"] = cb["parts_s"]
    return out


def serving_config(info, T):
    return {"workload": "8b-shaped target / 1b-shaped drafter serving 64 sequences, contexts log-uniform "
                        "[512, 4096] in 16-token pages, k per sequence in {3,5,7}"
                        + (", drafts mixed toward the target's top-1 at rate 0.7 (boost 2.0), off the clock"
                           if info["mix"] else ", no draft mixing"),
            "batch": 64, "mean_context": info["mean_ctx"], "rows_per_verify": info["rows_per_verify"],
            "temperature": T, "draft_mixing": info["mix"]}


def serving_cpu(info, models):
    """The oracle runs sequences one by one: one whole step of the batch's
    sequence with k = 5 nearest the median context, times the 64 sequences."""
    ctx, ks = info["ctx"], info["ks"]
    cand = [i for i in range(len(ks)) if int(ks[i]) == 5] or list(range(len(ks)))
    med = float(np.median(ctx))
    i = min(cand, key=lambda j: abs(float(ctx[j]) - med))
    log("oracle: one full step of serving sequence", i, "context", int(ctx[i]))
    r = cpu_full_step(*models, int(ctx[i]), int(ks[i]), info["T"], 1234 + i)
    step_s = r["step_s"] * len(ks)
    return {"value": info["tokens"] / info["steps"] / step_s, "step_s": step_s, "sample_s": r["step_s"],
            "parts_s": {x: r[x] for x in ("draft_s", "target_forward_s", "rule_s")},
            "sample": (f"one whole oracle step (float64) of one of the 64 sequences (context {int(ctx[i])}, "
                       f"k = {int(ks[i])}), times 64; each model's layers share one seeded layer's weights")}


def sub_line(info, steps, extra):
    out = {"value": info["tokens"] / info["wall_s"], "unit": "tokens/s", "steps": steps,
           "ms_per_step": info["wall_s"] * 1e3 / steps, "event_ms_per_step": info["event_ms"] / steps,
           "verify_ms_median": info["verify_ms_median"], "verify_ms_p90": info["verify_ms_p90"],
           "mean_accepted": float(np.mean(info["acc_hist"])) if info["acc_hist"] else None}
    if "verify_latency" in info:
        out["verify_latency"] = info["verify_latency"]
    out.update(extra)
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="all", choices=["all", "8b-shaped", "8b-serving", "vocab-stress", "prefill"],
                    help="all (default): the 8b-shaped line with greedy, plain-decode, serving and "
                         "vocab-stress sub-objects; prefill: only the long-context prefill object (for profiling)")
    ap.add_argument("--temperature", type=float, default=None,
                    help="sampling temperature (default 0.8; 0, greedy, for the serving workload, whose draft "
                         "mixing fixes top-1 agreement, i.e. the greedy acceptance test)")
    ap.add_argument("--kernel", default=None, help="kernel to time for the roofline (profiler name)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-mix", action="store_true",
                    help="serving workload without draft mixing (natural acceptance of the random-init pair)")
    ap.add_argument("--roof-steps", type=int, default=4,
                    help="steps after the timed region that run with per-kernel timing (eager launches)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-MiB device buffer --steps times (a plain copy kernel of known "
                         "size, for scaling the profiler's FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py measures one GPU only: sequences shard by data parallelism "
                                   "with no exchange, so a multi-GPU figure is N independent copies of the "
                                   "one-GPU line; run with --gpus 1"}))
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)

    if args.calibrate_copy:
        nbytes = args.calibrate_copy << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read_per_copy": nbytes,
                          "bytes_written_per_copy": nbytes, "copies": args.steps}), flush=True)
        return

    from workloads import LLAMA8B_SHAPED
    wl = args.workload
    serve_T = 0.0 if args.temperature is None or wl == "all" else args.temperature
    if args.temperature is None or wl == "all":
        args.temperature = 0.0 if wl == "8b-serving" else 0.8
    steps = args.steps
    info = info_s = info_v = info_d = info_t = info_p = None
    if wl == "prefill":
        target, _ = device_models(LLAMA8B_SHAPED)
        log("long-context prefill")
        print(json.dumps({"workload": "prefill", "prefill": bench_prefill(args, target)}), flush=True)
        return
    if wl in ("all", "8b-shaped", "8b-serving"):
        target, draft = device_models(LLAMA8B_SHAPED)
        if wl in ("all", "8b-shaped"):
            info = bench_8b(args, target, draft, extras=(wl == "all"))
        if wl in ("all", "8b-serving"):
            log("serving workload")
            info_s = bench_serving(args, target, draft, serve_T)
            info_s["T"], info_s["steps"] = serve_T, steps
        if wl == "all":
            info_d = bench_small_decode(args, draft)
            log("tree verification")
            info_t = bench_tree(args, target, draft)
            log("long-context prefill")
            info_p = bench_prefill(args, target)
        del target, draft
        torch.cuda.empty_cache()
    if wl in ("all", "vocab-stress"):
        log("vocab-stress workload")
        info_v = bench_vocab(args)

    b1_config = {"workload": "8b-shaped target / 1b-shaped drafter, batch 1, context 2048, k=5",
                 "target": "32L d4096 32q/8kv hd128 ffn14336 V128256", "draft": "16L d2048 32q/8kv hd64 ffn8192",
                 "batch": 1, "context": 2048, "k": 5, "temperature": args.temperature}
    vocab_config = {"workload": "vocab-stress: decision pass alone, 256 seqs x 8 rows x 128256",
                    "batch": 256, "k": 7, "vocab": 128256, "temperatures": [0.3, 1.0, 1.5]}
    serve_note = " (verify launches only)"
    if info is not None:  # the headline: batch 1
        head, bound, hw = info, "hbm", "8b-shaped"
        config = b1_config
    elif info_s is not None:
        head, bound, hw = info_s, "mfma", "8b-serving"
        config = serving_config(info_s, serve_T)
    else:
        head, bound, hw = info_v, "hbm", "vocab-stress"
        config = vocab_config
    line = {
        "metric": "verified tokens/sec + verify-step latency (ms) at 1 MI355X; % MFMA/HBM peak",
        "value": head["tokens"] / head["wall_s"], "unit": "tokens/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": head["wall_s"] * 1e3 / steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights and prompts)", "config": config,
        "verify_ms_median": head["verify_ms_median"], "verify_ms_p90": head["verify_ms_p90"],
        "verify_latency": head.get("verify_latency",
                                   "HIP events around spec_verify + spec_kv_commit of each timed step"),
        "event_ms_per_step": head["event_ms"] / steps,
        "mean_accepted": float(np.mean(head["acc_hist"])) if head["acc_hist"] else None,
        "offclock_ms_per_step": head.get("offclock_ms", 0.0) / steps,
        "roofline": roofline_of(head, bound, hw, args.roof_steps, serve_note if hw == "8b-serving" else ""),
    }
    if info is not None and "greedy" in info:
        line["greedy"] = info["greedy"]
        line["plain_decode"] = info["plain_decode"]
        line["speculative_gain"] = {
            "sampled": line["value"] / info["plain_decode"]["value"],
            "greedy": info["greedy"]["value"] / info["plain_decode"]["value"],
            "note": "verified tokens/s of draft-and-verify over plain target decode (k = 0) on the same box; "
                    "random-init models accept few drafts, so this is a slowdown here"}
    if info_s is not None and head is not info_s:
        line["serving"] = sub_line(info_s, steps, {
            "config": serving_config(info_s, serve_T),
            "offclock_ms_per_step": info_s.get("offclock_ms", 0.0) / steps,
            "roofline": roofline_of(info_s, "mfma", "8b-serving", args.roof_steps, serve_note)})
    if info_d is not None:
        line["small_decode"] = {
            "value": info_d["tokens"] / info_d["wall_s"], "unit": "tokens/s", "steps": steps,
            "ms_per_step": info_d["wall_s"] * 1e3 / steps, "event_ms_per_step": info_d["event_ms"] / steps,
            "config": {"workload": "1b-shaped model decoding alone (decode-only context sharing the drafter's "
                                   "weights), 64 sequences, contexts log-uniform [512, 4096], T = 0.8, "
                                   "one token per sequence per step",
                       "batch": 64, "mean_context": info_d["mean_ctx"], "temperature": 0.8},
            "roofline": roofline_of(info_d, "hbm", "small-decode", args.roof_steps)}
    if info_t is not None:
        line["tree_verify"] = info_t
    if info_p is not None:
        line["prefill"] = info_p
    if info_v is not None and head is not info_v:
        line["vocab_stress"] = sub_line(info_v, steps, {
            "config": vocab_config, "roofline": roofline_of(info_v, "hbm", "vocab-stress", args.roof_steps)})
    for obj, inf in ((line, head), (line.get("vocab_stress"), info_v)):
        if obj is not None and inf is not None and "vocab_bytes" in inf:
            vb = dict(inf["vocab_bytes"])
            ms = obj["ms_per_step"]
            vb["read_gbs"] = vb["read_per_step"] / (ms / 1e3) / 1e9
            vb["early_exit_gbs"] = vb["early_exit_per_step"] / (ms / 1e3) / 1e9
            obj["vocab_bytes"] = vb
    if not args.no_cpu_baseline:
        model, threads, aff = cpu_info()
        log("timing the oracle on a bounded sample")
        models = oracle_models() if (info is not None or info_s is not None) else None
        if info is not None:
            line["cpu_baseline"] = cpu_line(cpu_baseline_8b(info["tokens"] / steps, models), threads, model, aff)
        if info_s is not None:
            cb = cpu_line(serving_cpu(info_s, models), threads, model, aff)
            (line if head is info_s else line["serving"])["cpu_baseline"] = cb
        if info_v is not None:
            cb = cpu_line(cpu_baseline_vocab(info_v["tokens"] / steps), threads, model, aff)
            (line if head is info_v else line["vocab_stress"])["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
