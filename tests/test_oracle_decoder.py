"""Pins of the oracle decoder's building blocks against independent definitions
(PyTorch CPU float64 library routines, complex arithmetic) and of its KV cache
against a no-cache forward."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decoder as D
from workloads import ModelShape, model_weights, bf16_round_u16


def test_widen_bf16_matches_torch():
    g = np.random.default_rng(0)
    x = g.standard_normal(1000).astype(np.float32) * 3
    u = bf16_round_u16(x)
    ref = torch.from_numpy(u.view(np.int16)).view(torch.bfloat16).double().numpy()
    assert np.array_equal(D.widen(u), ref)
    # round-to-nearest-even against torch's own fp32 -> bf16 conversion
    t = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(u, t)


def test_rms_norm_matches_torch():
    g = np.random.default_rng(1)
    x = g.standard_normal((7, 96))
    w = g.standard_normal(96).astype(np.float32)
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(w.astype(np.float64)), eps=1e-5).numpy()
    assert np.allclose(D.rms_norm(x, w, 1e-5), ref, rtol=1e-13, atol=1e-13)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 601)
    assert np.allclose(D.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-13, atol=1e-300)


@pytest.mark.parametrize("hq,hkv", [(4, 4), (8, 2), (6, 1)])
def test_attention_matches_sdpa_gqa_window(hq, hkv):
    """Verify-window attention: n query rows at positions T-n..T-1 over T keys."""
    g = np.random.default_rng(hq * 10 + hkv)
    T, n, hd = 37, 6, 16
    q = g.standard_normal((n, hq, hd))
    K = g.standard_normal((T, hkv, hd))
    V = g.standard_normal((T, hkv, hd))
    qpos = np.arange(T - n, T)
    got = D.attention(q, K, V, qpos)
    mask = torch.from_numpy(np.arange(T)[None, :] <= qpos[:, None])
    ref = F.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(0, 1), torch.from_numpy(K).transpose(0, 1),
        torch.from_numpy(V).transpose(0, 1), attn_mask=mask, enable_gqa=True).transpose(0, 1).numpy()
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_rope_is_complex_rotation():
    """Rotate-half RoPE on pairs (i, i+hd/2) equals multiplying the complex number
    x_i + j x_{i+hd/2} by exp(j * pos * theta^(-2i/hd))."""
    g = np.random.default_rng(3)
    hd, theta = 64, 1e4
    x = g.standard_normal((5, 3, hd))
    pos = np.array([0, 1, 17, 1000, 123456])
    got = D.rope(x, pos, theta)
    i = np.arange(hd // 2)
    zc = x[..., :hd // 2] + 1j * x[..., hd // 2:]
    rot = np.exp(1j * pos[:, None, None] * (theta ** (-(2 * i) / hd))[None, None, :])
    ref = zc * rot
    assert np.allclose(got[..., :hd // 2], ref.real, atol=1e-12)
    assert np.allclose(got[..., hd // 2:], ref.imag, atol=1e-12)
    assert np.array_equal(D.rope(x, np.zeros(5, dtype=int), theta), x)


def test_rope_relative_position_invariance():
    g = np.random.default_rng(4)
    hd = 128
    q = g.standard_normal((1, 1, hd))
    k = g.standard_normal((1, 1, hd))
    a = (D.rope(q, [50], 5e5) * D.rope(k, [20], 5e5)).sum()
    b = (D.rope(q, [1050], 5e5) * D.rope(k, [1020], 5e5)).sum()
    assert abs(a - b) < 1e-10


def _tiny(V=64, dtype="f32", hq=4, hkv=2):
    return ModelShape("pin-tiny", 2, 32, hq, hkv, 8, 48, V, 1e4, dtype=dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_kv_cache_invariance(dtype):
    """Logits computed incrementally through the cache (any chunking, with
    truncations and re-feeds) equal a no-cache forward of the whole sequence."""
    sh = _tiny(dtype=dtype)
    dec = D.Decoder(sh, model_weights(sh, 11))
    g = np.random.default_rng(5)
    toks = g.integers(0, sh.vocab, size=30)
    full = dec.full_logits(toks)
    kv = dec.new_kv()
    dec.forward(kv, toks[:10], np.arange(10), logits=False)
    # feed a wrong continuation, then roll it back
    dec.forward(kv, (toks[10:15] + 1) % sh.vocab, np.arange(10, 15), logits=False)
    kv.truncate(10)
    z1 = dec.forward(kv, toks[10:13], np.arange(10, 13))
    z2 = dec.forward(kv, toks[13:30], np.arange(13, 30))
    assert np.allclose(np.concatenate([z1, z2]), full[10:], rtol=1e-12, atol=1e-12)


def test_gqa_equals_repeated_heads():
    """A GQA model equals the MHA model whose k/v heads are the GQA heads repeated."""
    g = np.random.default_rng(6)
    n, T, hd = 3, 9, 8
    q = g.standard_normal((n, 8, hd))
    K = g.standard_normal((T, 2, hd))
    V = g.standard_normal((T, 2, hd))
    pos = np.arange(T - n, T)
    a = D.attention(q, K, V, pos)
    b = D.attention(q, np.repeat(K, 4, axis=1), np.repeat(V, 4, axis=1), pos)
    assert np.allclose(a, b, rtol=0, atol=1e-14)


@pytest.mark.parametrize("L", [1, 2, 3])
def test_kv_at_sampled_rows_equals_the_cached_forward(L):
    """Decoder.kv_at (every layer's K/V at chosen positions, computing only what
    they depend on) against the K/V that the full cached forward appends."""
    from workloads import TINY_FP32, uniform_prompts
    sh = TINY_FP32.target
    w = model_weights(sh, 5, L)
    dec = D.Decoder(sh, w)
    toks = uniform_prompts(3, [90], sh.vocab)[0]
    rows = [0, 15, 16, 44, 88]
    got = dec.kv_at(toks[:89], rows)
    kv = dec.new_kv()
    dec.forward(kv, toks[:89], np.arange(89), logits=False)
    for l in range(L):
        np.testing.assert_allclose(got[l][0], kv.K[l][rows], rtol=0, atol=1e-12)
        np.testing.assert_allclose(got[l][1], kv.V[l][rows], rtol=0, atol=1e-12)
