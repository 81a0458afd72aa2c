"""Shared helpers of the GPU parity tests (not collected: no test_ prefix)."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")


def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_20507_amd import binding
    binding.lib()  # the HIP library must load: no fallback
    return torch.device("cuda:0")


def bf16_bits(t):
    """bf16 device tensor -> uint16 numpy bit patterns."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def widen_bits(u16):
    return (u16.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def rel_err(got, ref):
    """max |got - ref| / max |ref| (per-tensor normwise relative error)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-300))


def say(*a):
    """Print a progress line that names the GPU case before it runs."""
    print("[gpu]", *a, flush=True)
