"""Long-context prefill (the paper's 1K-8K contexts) against the oracle.

A two-layer target at the 8B width (d 4096, 32 q / 8 kv heads of 128, ffn
14336, RoPE theta 5e5) prefills one prompt of 4096 or 8192 tokens, in one
chunk of max_rows rows or in two.  Every layer's K (after RoPE) and V are
read back from the paged pool (the documented page layout) at sampled
positions, among them the first and last of each page and chunk, and
compared with the oracle's no-cache forward restricted to those positions
(Decoder.kv_at), within 2e-2 normwise per layer.  Layer 1's K/V at a
position are the projection of layer 0's output there, so this checks the
large-M QKV, O, gate/up and down GEMMs and the causal prefill attention of
layer 0 over the whole prefix at each sampled row.
"""

import numpy as np
import pytest

from oracle.decoder import Decoder
from tests.gpu_util import device, rel_err, say, torch
from workloads import model_weights, uniform_prompts
from workloads.configs import L8B_TARGET

pytestmark = pytest.mark.gpu


def _k_off(k, d):
    """Element of token k (of 16), dim d in a bf16 (page, kv head) K block."""
    c = d >> 3
    s, g = c >> 2, c & 3
    h, j = (k >> 2) & 1, (k & 3) + 4 * (k >> 3)
    return ((((s * 2 + h) * 4 + g) * 8 + j) << 3) + (d & 7)


def _v_off(k, d):
    return ((((d >> 4) * 2 + (k >> 3)) * 16 + (d & 15)) << 3) + (k & 7)


_W = {}


def _weights():
    if "w" not in _W:
        _W["w"] = model_weights(L8B_TARGET, 4321, 2)
    return _W["w"]


@pytest.mark.parametrize("P,max_rows", [(4097, 4096), (8193, 4096), (8193, 8192)])
def test_long_prefill_kv_sampled(P, max_rows):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    sh = L8B_TARGET
    w = _weights()
    pages = (P + 15) // 16 + 2
    gpu = SpecSession(DeviceModel(sh, w, dev, n_layers=2), None, max_seqs=1, k_max=0, max_pages_per_seq=pages,
                      max_rows=max_rows)
    prompt = uniform_prompts(77 + P, [P], sh.vocab)[0]
    say("prefill", P, "tokens, chunks of", max_rows)
    gpu.prefill([5], [prompt])
    torch.cuda.synchronize()
    n = P - 1  # positions 0..P-2 are cached
    rows = sorted({0, 1, 15, 16, 17, 255, 1023, 2047, 2048, max_rows - 1, min(max_rows, n - 1), n // 2 + 3,
                   n - 17, n - 2, n - 1} | set(int(x) for x in np.random.default_rng(P).integers(0, n, size=6)))
    info = gpu.seq_info(5)
    assert info["target_len"] == n
    table = info["pages_target"]
    Hkv, hd = sh.n_kv_heads, sh.head_dim
    num_pages = gpu.cache.num_pages_target
    layer_stride = num_pages * Hkv * 16 * hd * 2
    v_off = layer_stride // 2
    pool = gpu.kv_target.view(torch.int16).cpu().numpy().view(np.uint16)
    d = np.arange(hd)
    say("oracle kv at", len(rows), "rows")
    ref = Decoder(sh, w).kv_at(prompt[:n], rows)
    for l in range(2):
        K = np.zeros((len(rows), Hkv, hd))
        V = np.zeros((len(rows), Hkv, hd))
        for i, r in enumerate(rows):
            pg, k = table[r // 16], r % 16
            for h in range(Hkv):
                blk = l * layer_stride + (pg * Hkv + h) * 16 * hd
                K[i, h] = pool[blk + _k_off(k, d)]
                V[i, h] = pool[v_off + blk + _v_off(k, d)]
        K = ((K.astype(np.uint32) << np.uint32(16)).view(np.float32)).astype(np.float64)
        V = ((V.astype(np.uint32) << np.uint32(16)).view(np.float32)).astype(np.float64)
        ek, ev = rel_err(K, ref[l][0]), rel_err(V, ref[l][1])
        say("layer", l, "K err", ek, "V err", ev)
        assert ek < 2e-2 and ev < 2e-2, (l, ek, ev)
        for i, r in enumerate(rows):  # no sampled row may hide a local error
            assert rel_err(K[i], ref[l][0][i]) < 3e-2 and rel_err(V[i], ref[l][1][i]) < 3e-2, (l, r)
    gpu.close()
