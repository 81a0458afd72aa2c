"""Philox4x32-10 counter-based generator, written from its published definition.

Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3"
(SC'11), Section 3 (the Philox S-box): a 4x32 counter and a 2x32 key; each of
the 10 rounds multiplies words 0 and 2 by the constants M0 and M1, and the new
state is (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0)); the
key is bumped by the Weyl constants (W0, W1) between rounds.

Keying used by the verify step (a reading the paper leaves open; it names no
generator): key = (seed lo32, seed hi32); counter = (block, pos, seq lo32,
(seq bits 32..55) << 8 | purpose).  ``pos`` is the absolute position of the token
being decided; ``seq`` is the caller's stable sequence id.  Vocabulary noise for
token i uses block i >> 2 and output word i & 3; a scalar draw uses block 0,
word 0.

Uniform: u = ((x >> 9) + 0.5) * 2^-23, exact in both fp32 and fp64 and strictly
inside (0, 1).  Gumbel: G = -log(-log u).
"""

from __future__ import annotations

import numpy as np

M0 = 0xD2511F53
M1 = 0xCD9E8D57
W0 = 0x9E3779B9
W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF

# purposes of the random streams
DRAFT = 0
ACCEPT = 1
RESAMPLE = 2
BONUS = 3


def philox4x32_10(ctr, key):
    """Philox4x32-10 of counters ``ctr`` (array [..., 4] of uint32) under ``key``
    (k0, k1).  Returns uint32 array [..., 4]."""
    ctr = np.asarray(ctr, dtype=np.uint64)
    c0, c1, c2, c3 = (ctr[..., i].copy() for i in range(4))
    k0 = np.uint64(int(key[0]) & MASK32)
    k1 = np.uint64(int(key[1]) & MASK32)
    m0, m1, mask = np.uint64(M0), np.uint64(M1), np.uint64(MASK32)
    sh = np.uint64(32)
    for _ in range(10):
        p0 = m0 * c0            # < 2^64: both factors are below 2^32
        p1 = m1 * c2
        c0, c1, c2, c3 = ((p1 >> sh) ^ c1 ^ k0, p1 & mask,
                          (p0 >> sh) ^ c3 ^ k1, p0 & mask)
        k0 = np.uint64((int(k0) + W0) & MASK32)
        k1 = np.uint64((int(k1) + W1) & MASK32)
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def seed_key(seed: int):
    seed = int(seed) & ((1 << 64) - 1)
    return (seed & MASK32, seed >> 32)


def stream_counter(seq: int, pos: int, purpose: int, blocks) -> np.ndarray:
    """Counters (block, pos, seq lo32, seq hi24 << 8 | purpose) for ``blocks``."""
    seq = int(seq) & ((1 << 64) - 1)
    blocks = np.asarray(blocks, dtype=np.uint64)
    c = np.empty(blocks.shape + (4,), dtype=np.uint64)
    c[..., 0] = blocks
    c[..., 1] = np.uint64(int(pos) & MASK32)
    c[..., 2] = np.uint64(seq & MASK32)
    c[..., 3] = np.uint64((((seq >> 32) & 0xFFFFFF) << 8) | (int(purpose) & 0xFF))
    return c


def raw_words(seed: int, seq: int, pos: int, purpose: int, n: int) -> np.ndarray:
    """The first ``n`` 32-bit words of stream (seed, seq, pos, purpose): word i is
    output lane i & 3 of block i >> 2."""
    nb = (n + 3) // 4
    out = philox4x32_10(stream_counter(seq, pos, purpose, np.arange(nb)), seed_key(seed))
    return out.reshape(-1)[:n]


def to_uniform(x) -> np.ndarray:
    """u = ((x >> 9) + 0.5) * 2^-23 in float64 (exact)."""
    x = np.asarray(x, dtype=np.uint64)
    return ((x >> np.uint64(9)).astype(np.float64) + 0.5) * (2.0 ** -23)


def uniform(seed: int, seq: int, pos: int, purpose: int) -> float:
    """The scalar uniform of a stream (block 0, word 0)."""
    return float(to_uniform(raw_words(seed, seq, pos, purpose, 1))[0])


def uniform_block(seed: int, seq: int, pos: int, purpose: int, block: int) -> float:
    """Word 0 of block ``block`` of a stream as a uniform (block 0 is ``uniform``):
    the scalar draw of candidate ``block`` among several at one position."""
    w = philox4x32_10(stream_counter(seq, pos, purpose, [int(block)]), seed_key(seed))
    return float(to_uniform(w[0, 0]))


def gumbel(seed: int, seq: int, pos: int, purpose: int, n: int) -> np.ndarray:
    """Gumbel(0,1) noise G_i = -log(-log u_i) for i < n, float64."""
    u = to_uniform(raw_words(seed, seq, pos, purpose, n))
    return -np.log(-np.log(u))
