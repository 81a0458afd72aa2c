"""CPU check of the decision-pass workspace bounds: a context sizes its
decision, tree and draft workspaces once, for its largest call, and every
smaller call must fit too.  A plan's chunk count grows as its rows shrink, so
the largest call's own plan is not an upper bound (a 1-sequence, 79-row call
of an 8-sequence, k = 5 context took more than it); the bound functions are
checked against every plan of every smaller call on the host."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(ROOT, "paper_2607_20507_amd", "csrc")


@pytest.fixture(scope="module")
def bound_exe(tmp_path_factory):
    hipcc = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)
    if not hipcc:
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("wsb") / "ws_bound_driver")
    subprocess.run([hipcc, "-O1", "-std=c++17", "--offload-arch=gfx950", "-x", "hip", "-I", CSRC, "-I",
                    os.path.join(ROOT, "include"), os.path.join(HERE, "native", "ws_bound_driver.cpp"),
                    os.path.join(CSRC, "vocab.hip"), "-o", exe], check=True, capture_output=True)
    return exe


def test_workspace_bounds_cover_every_smaller_call(bound_exe):
    cases = []
    for V in (1000, 4096, 32000, 128256, 151936):
        for B in (1, 2, 8, 64, 256):
            for k in (0, 5, 15):
                cases.append((V, B, B * (2 * k + 1)))
    out = subprocess.run([bound_exe], input="".join(f"{v} {b} {n}\n" for v, b, n in cases), capture_output=True,
                         text=True, check=True).stdout.split("\n")
    assert out[:len(cases)] == ["ok"] * len(cases), [(c, o) for c, o in zip(cases, out) if o != "ok"][:3]
