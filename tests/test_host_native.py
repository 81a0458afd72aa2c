"""CPU checks of the native library: it loads and exports every symbol the
public headers declare, and its host page allocator assigns exactly the pages
the oracle's allocation rule fixes (bit-exact KV indices)."""

import os
import re
import shutil
import subprocess

import numpy as np
import pytest

from oracle.paging import PageOOM, PagePool

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))


def header_symbols():
    syms = []
    for h in ("spec.h", "spec_ops.h"):
        txt = open(os.path.join(ROOT, "include", h)).read()
        syms += re.findall(r"SPEC_API\s+[\w\s\*]+?\b(spec_\w+)\s*\(", txt)
    return sorted(set(syms))


def test_headers_declare_the_boundary():
    syms = header_symbols()
    for name in ("spec_prefill", "spec_draft_step", "spec_verify", "spec_kv_commit", "spec_kv_rollback",
                 "spec_sample_verify", "spec_ctx_create"):
        assert name in syms


def test_library_loads_and_exports_every_symbol():
    from paper_2607_20507_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("library not built")
    L = binding.lib()
    for s in header_symbols():
        assert hasattr(L, s), s
        assert s in binding.SIGNATURES, f"binding lacks {s}"
    # host-only calls need no GPU
    assert L.spec_sample_workspace_bytes(0, 0, 10) == 0
    assert binding.lib().spec_last_error(None) is not None


@pytest.fixture(scope="module")
def pagepool_exe(tmp_path_factory):
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("pp") / "pagepool_driver")
    subprocess.run([gxx, "-O1", "-std=c++17", "-I", os.path.join(ROOT, "paper_2607_20507_amd", "csrc"),
                    os.path.join(HERE, "native", "pagepool_driver.cpp"), "-o", exe], check=True)
    return exe


def test_page_allocator_matches_oracle_rule(pagepool_exe):
    g = np.random.default_rng(0)
    num_pages = 40
    ops = []
    lens = {}
    for _ in range(600):
        s = int(g.integers(0, 5))
        cur = lens.get(s, 0)
        if g.random() < 0.6:
            n = cur + int(g.integers(0, 40))
            ops.append(("E", s, n))
        else:
            n = int(g.integers(0, cur + 1))
            ops.append(("T", s, n))
    script = f"{num_pages}\n" + "".join(f"{o} {s} {n}\n" for o, s, n in ops)
    out = subprocess.run([pagepool_exe], input=script, capture_output=True, text=True, check=True).stdout.splitlines()
    pool = PagePool(num_pages, 16)
    tabs = {}
    for (o, s, n), line in zip(ops, out):
        tabs.setdefault(s, None)
        if o == "E":
            try:
                pool.ensure(s, n)
                status = "ok"
                lens[s] = n
            except PageOOM:
                status = "oom"
        else:
            pool.truncate(s, n)
            status = "ok"
        parts = line.split(" |")
        assert parts[0] == status
        got = {int(p.split(":")[0]): [int(x) for x in p.split(":")[1].split()] for p in parts[1:]}
        want = {k: pool.tables.get(k, []) for k in got}
        assert got == want
