"""Plain, slow CPU oracle of the speculative-decoding verify step.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(the HIP library and its Python binding) never calls it and shares no code
with it; both sides read only the seeded inputs of ``workloads``.

What it computes (CacheSpec, Section 3.4 "Cache-Miss Branch" and the
speculative-decoding paragraph of Section 2: the small model drafts candidate
tokens, the target scores them in one parallel pass and accepts, corrects or
continues; the rule is the cited speculative sampling of Leviathan et al. 2023
and Chen et al. 2023):

* ``philox``   Philox4x32-10 (Salmon et al., SC'11), uniforms, Gumbel noise.
* ``decoder``  Llama-style decoder forward in float64 with a per-sequence KV list.
* ``rule``     the draft sampler and the accept / residual-resample / bonus rule,
               greedy mode, the exact outcome law, and decision margins.
* ``paging``   the lowest-free-page allocator that fixes KV page indices.
* ``session``  prefill -> draft x k -> verify -> commit / rollback, end to end.
* ``brute``    brute-force output marginal of repeated draft-and-verify steps.

Every floating-point computation here is float64 (weights given in fp32 or
bf16 are widened exactly).  Pins: see the ``-m "not gpu"`` tests.
"""
