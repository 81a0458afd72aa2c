"""Graph replay of the draft step and the verify against eager launches.

The same seeded run (prefill, k draft steps, verify, commit, with a sequence
released midway so that the batch shape changes and changes back) is executed
twice through the C ABI: once replaying captured graphs, once launching every
kernel eagerly.  Every replay is checked against its eager counterpart:
accepted counts, emitted tokens and verify logits bit-exact, cache lengths and
page tables equal.  Between replays the library's own eager work (commit,
release) and the verify's synchronisation run as usual.
"""

import numpy as np
import pytest

from tests.gpu_util import device, say, torch
from workloads import SMALL_BF16, TINY_FP32, model_weights, seq_ids_for, uniform_prompts

pytestmark = pytest.mark.gpu


def _run(cfg, graphs, n_layers_t, n_layers_d, temps, steps, lens):
    from paper_2607_20507_amd.session import DeviceModel, SpecSession
    dev = device()
    tw = model_weights(cfg.target, cfg.seed, n_layers_t)
    dw = model_weights(cfg.draft, cfg.seed, n_layers_d)
    k = max(cfg.k)
    gpu = SpecSession(DeviceModel(cfg.target, tw, dev, n_layers=n_layers_t),
                      DeviceModel(cfg.draft, dw, dev, n_layers=n_layers_d), max_seqs=4,
                      k_max=k, max_pages_per_seq=48, max_rows=512, graphs=graphs)
    ids = [int(x) for x in seq_ids_for(cfg.seed + 5, len(lens))]
    gpu.prefill(ids, uniform_prompts(cfg.seed, lens, cfg.target.vocab))
    live = list(ids)
    trace = []
    for step in range(steps):
        if step == steps // 2:
            gpu.release(live[-1])  # shape change: n drops by one
            live = live[:-1]
        tl = [temps[i % len(temps)] for i in range(len(live))]
        for _ in range(k):
            gpu.draft_step(live, tl, 100 + step)
        na, ot = gpu.verify(live, tl, 100 + step)
        z = gpu.last_logits().cpu().numpy()
        gpu.commit(live, na)
        info = [gpu.seq_info(s) for s in live]
        trace.append((na.copy(), ot.copy(), z, info))
    gpu.close()
    return trace


@pytest.mark.parametrize("cfg,layers", [(SMALL_BF16, (2, 1)), (TINY_FP32, (None, None))],
                         ids=["small-bf16-2L", "tiny-fp32"])
def test_graph_replay_matches_eager(cfg, layers):
    args = dict(n_layers_t=layers[0], n_layers_d=layers[1], temps=[0.7, 0.0, 1.0], steps=8,
                lens=[70, 41, 96])
    say("graph replay vs eager", cfg.target.d_model)
    g = _run(cfg, True, **args)
    e = _run(cfg, False, **args)
    assert len(g) == len(e)
    for step, (a, b) in enumerate(zip(g, e)):
        assert np.array_equal(a[0], b[0]), f"step {step}: accepted counts differ"
        assert np.array_equal(a[1], b[1]), f"step {step}: tokens differ"
        assert np.array_equal(a[2], b[2]), f"step {step}: verify logits differ"
        assert a[3] == b[3], f"step {step}: cache state differs"
