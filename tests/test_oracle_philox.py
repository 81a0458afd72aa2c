"""Pins of the oracle's Philox4x32-10 generator and its uniform/Gumbel maps."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import philox

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((v[0:4], v[4:6], v[6:10]))
    return rows


def test_known_answer_vectors():
    rows = _kat()
    assert len(rows) == 3
    for ctr, key, want in rows:
        got = philox.philox4x32_10(np.array(ctr, dtype=np.uint32), key)
        assert [int(x) for x in got] == want


@pytest.fixture(scope="module")
def rocrand_ref(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc) or not os.path.isdir("/opt/rocm/include/rocrand"):
        pytest.skip("hipcc / rocRAND headers not available")
    exe = str(tmp_path_factory.mktemp("rr") / "rocrand_philox_ref")
    src = os.path.join(HERE, "native", "rocrand_philox_ref.cpp")
    subprocess.run([hipcc, "-x", "hip", "--offload-arch=gfx950", "-I/opt/rocm/include",
                    "-O1", src, "-o", exe], check=True, capture_output=True)
    return exe


def test_matches_rocrand_header(rocrand_ref):
    """rocRAND's open-source Philox (seed -> key, (block, subsequence) -> counter)
    agrees with the oracle on random keys and counters, all four words."""
    g = np.random.default_rng(7)
    cases = []
    for _ in range(300):
        seed = int(g.integers(0, 1 << 63)) * 2 + int(g.integers(0, 2))
        sub = int(g.integers(0, 1 << 63)) * 2 + int(g.integers(0, 2))
        blk = int(g.integers(0, 1 << 40))
        cases.append((seed, sub, blk))
    cases += [(0, 0, 0), ((1 << 64) - 1, (1 << 64) - 1, 0), (5, 1 << 32, 3)]
    inp = "".join(f"{s} {u} {b}\n" for s, u, b in cases)
    out = subprocess.run([rocrand_ref], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    for (seed, sub, blk), line in zip(cases, out):
        ctr = np.array([blk & 0xFFFFFFFF, blk >> 32, sub & 0xFFFFFFFF, sub >> 32], dtype=np.uint32)
        got = philox.philox4x32_10(ctr, philox.seed_key(seed))
        assert " ".join("%08x" % int(x) for x in got) == line


def test_uniform_exact_and_open_interval():
    x = np.array([0, 1, 511, 512, 0x7FFFFFFF, 0xFFFFFFFF], dtype=np.uint32)
    u64 = philox.to_uniform(x)
    # the same map evaluated in fp32 is exact: every value is a 24-bit mantissa
    u32 = ((x >> 9).astype(np.float32) + np.float32(0.5)) * np.float32(2.0 ** -23)
    assert np.array_equal(u64, u32.astype(np.float64))
    assert u64.min() == 2.0 ** -24 and u64.max() == 1.0 - 2.0 ** -24
    assert np.all((u64 > 0) & (u64 < 1))


def test_uniformity_chi2():
    w = philox.raw_words(123, 99, 7, philox.RESAMPLE, 200_000)
    u = philox.to_uniform(w)
    counts, _ = np.histogram(u, bins=64, range=(0, 1))
    e = len(u) / 64
    chi2 = ((counts - e) ** 2 / e).sum()
    assert chi2 < 120  # 63 dof: mean 63, sd ~11


def test_stream_layout_and_independence():
    # word i is output lane i & 3 of block i >> 2
    w = philox.raw_words(1, 2, 3, philox.DRAFT, 10)
    b2 = philox.philox4x32_10(philox.stream_counter(2, 3, philox.DRAFT, [2])[0], philox.seed_key(1))
    assert int(w[8]) == int(b2[0]) and int(w[9]) == int(b2[1])
    # purposes, positions, sequences (including the high id bits) and seeds all change the stream
    base = philox.raw_words(1, 2, 3, philox.DRAFT, 8)
    for alt in (philox.raw_words(1, 2, 3, philox.ACCEPT, 8), philox.raw_words(1, 2, 4, philox.DRAFT, 8),
                philox.raw_words(1, 2 + (1 << 32), 3, philox.DRAFT, 8), philox.raw_words(2, 2, 3, philox.DRAFT, 8)):
        assert not np.array_equal(base, alt)


def test_gumbel_moments():
    G = philox.gumbel(5, 11, 13, philox.BONUS, 400_000)
    # Gumbel(0,1): mean = Euler-Mascheroni constant, variance = pi^2 / 6
    assert abs(G.mean() - 0.5772156649) < 4 * np.sqrt(np.pi ** 2 / 6 / len(G))
    assert abs(G.var() - np.pi ** 2 / 6) < 0.02
