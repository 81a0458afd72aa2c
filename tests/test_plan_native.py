"""CPU checks of the attention work planner (plan_attention, host C++): on
seeded random batches, every (row, key) pair a row attends is covered by
exactly one work item, items stay inside their sequence's rows with
consecutive positions, query tiles fit the kernel's 16-wide tiles, split
items map one-to-one onto partials that their groups combine, and the tile
width follows the rule for one sequence versus several."""

import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2607_20507_amd", "csrc")


@pytest.fixture(scope="module")
def plan_exe(tmp_path_factory):
    hipcc = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)
    if not hipcc:
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("plan") / "plan_driver")
    subprocess.run([hipcc, "-O1", "-std=c++17", "--offload-arch=gfx950", "-x", "hip", "-I", CSRC, "-I",
                    os.path.join(ROOT, "include"), os.path.join(HERE, "native", "plan_driver.cpp"),
                    os.path.join(CSRC, "plan.cpp"), "-o", exe], check=True, capture_output=True)
    return exe


def run_plans(exe, problems):
    text = []
    for G, Hkv, max_parts, target, allow_prefill, segs in problems:
        text.append(f"{G} {Hkv} {max_parts} {target} {int(allow_prefill)} {len(segs)}")
        text += [f"{s} {r0} {n} {p0}" for s, r0, n, p0 in segs]
    out = subprocess.run([exe], input="\n".join(text) + "\n", capture_output=True, text=True, check=True).stdout
    plans, cur = [], None
    for line in out.splitlines():
        f = line.split()
        if f[0] == "plan":
            cur = {"nt": int(f[1]), "w": int(f[2]), "prefill": bool(int(f[3])), "n_parts": int(f[4]),
                   "items": [], "groups": []}
            plans.append(cur)
        elif f[0] == "item":
            cur["items"].append(tuple(int(x) for x in f[1:]))
        else:
            cur["groups"].append(tuple(int(x) for x in f[1:]))
    assert len(plans) == len(problems)
    return plans


def expected_nt(segs, G):
    """The tile rule: 16-wide tiles for rows * G query vectors, halved once for a single sequence
    when a row's query heads still fit."""
    want = min(max(n for _, _, n, _ in segs) * G, 64)
    nt = 1 if want <= 16 else (2 if want <= 32 else 4)
    if len(segs) == 1 and nt >= 2 and G <= 8 * nt:
        nt //= 2
    return nt


def check_plan(plan, G, Hkv, max_parts, segs):
    items, groups = plan["items"], plan["groups"]
    by_seq = {s: (r0, n, p0) for s, r0, n, p0 in segs}
    cover = {}
    for row0, nrows, pos0, seq, t0, t1, part in items:
        r0, n, p0 = by_seq[seq]
        assert r0 <= row0 and row0 + nrows <= r0 + n and nrows >= 1
        assert pos0 == p0 + (row0 - r0), "rows of an item sit at consecutive positions of its sequence"
        assert 0 <= t0 < t1 <= pos0 + nrows, "keys past the item's last row are never read"
        for r in range(row0, row0 + nrows):
            cover.setdefault(r, []).append((t0, t1))
        if not plan["prefill"]:
            assert nrows * G <= 16 * plan["nt"], "query vectors fit the item's tiles"
    for s, r0, n, p0 in segs:
        for r in range(r0, r0 + n):
            pos = p0 + (r - r0)
            ranges = sorted(cover.get(r, []))
            # keys 0..pos each covered exactly once (keys past pos are masked)
            assert ranges and ranges[0][0] == 0
            for (a0, a1), (b0, b1) in zip(ranges, ranges[1:]):
                assert a1 == b0, f"row {r}: key ranges {ranges} overlap or leave a gap"
            assert ranges[-1][1] >= pos + 1
    if plan["prefill"]:
        assert not groups and all(it[6] < 0 and it[4] == 0 for it in items)
        assert all(it[1] <= 256 // G for it in items)
        t1s = [it[5] for it in items]
        assert t1s == sorted(t1s, reverse=True), "prefill blocks heaviest first"
        return
    nt, w = plan["nt"], plan["w"]
    assert nt == expected_nt(segs, G)
    assert w == (2 if nt >= 4 else 4)
    assert plan["n_parts"] <= max_parts
    parts = sorted(it[6] for it in items if it[6] >= 0)
    assert parts == list(range(plan["n_parts"])), "every partial written by exactly one item"
    part_rows = {it[6]: (it[0], it[1]) for it in items if it[6] >= 0}
    seen = []
    for row0, nrows, part0, nparts in groups:
        assert nparts >= 2
        for q in range(part0, part0 + nparts):
            assert part_rows[q] == (row0, nrows), "a group combines the partials of its own rows"
            seen.append(q)
    assert sorted(seen) == parts, "every partial combined by exactly one group"
    for it in items:
        if it[6] >= 0:
            assert it[4] % 32 == 0, "split key ranges start on 32-key chunks"
    lens = [it[5] - it[4] for it in items]
    assert lens == sorted(lens, reverse=True), "longest key ranges first"


def random_problem(g, shape):
    G = int(g.choice([1, 2, 4, 8, 16, 32]))
    Hkv = int(g.choice([1, 2, 8]))
    max_parts = int(g.choice([16, 64, 4096]))
    allow_prefill = bool(g.integers(0, 2))
    if shape == "single":
        n_seq = 1
    elif shape == "few":
        n_seq = int(g.integers(2, 6))
    else:
        n_seq = int(g.integers(8, 65))
    long_rows = shape != "many" and g.random() < 0.3
    segs, row = [], 0
    for s in range(n_seq):
        n = int(g.integers(64, 300)) if long_rows else int(g.integers(1, 17))
        p0 = int(g.integers(0, 5000))
        segs.append((s, row, n, p0))
        row += n
    return G, Hkv, max_parts, 512, allow_prefill, segs


@pytest.mark.parametrize("shape", ["single", "few", "many"])
def test_plan_invariants(plan_exe, shape):
    g = np.random.default_rng({"single": 1, "few": 2, "many": 3}[shape])
    problems = [random_problem(g, shape) for _ in range(60)]
    for prob, plan in zip(problems, run_plans(plan_exe, problems)):
        G, Hkv, max_parts, _, _, segs = prob
        check_plan(plan, G, Hkv, max_parts, segs)


def test_plan_batch1_shapes(plan_exe):
    # the 8B-shaped verify (6 rows, 4 query heads per KV head) and the
    # drafter's one-row step at context 2048, and a 15-node tree's rows
    problems = [(4, 8, 4096, 512, True, [(0, 0, 6, 2048)]),
                (4, 8, 4096, 512, True, [(0, 0, 1, 2048)]),
                (4, 8, 4096, 512, False, [(0, 0, 15, 2048)]),
                (4, 8, 4096, 512, True, [(s, 6 * s, 6, 2048) for s in range(4)])]
    plans = run_plans(plan_exe, problems)
    for prob, plan in zip(problems, plans):
        check_plan(plan, prob[0], prob[1], prob[2], prob[5])
    assert [p["nt"] for p in plans] == [1, 1, 2, 2]
    # the single 6-row verify: two 4- and 2-row tiles, 128-key ranges (17 partials each)
    assert sorted({(it[0], it[1]) for it in plans[0]["items"]}) == [(0, 4), (4, 2)]
    assert plans[0]["n_parts"] == 34
