"""MI355X-native speculative-decoding verify step.

``binding``  ctypes wrappers of libspecverify.so (include/spec.h, spec_ops.h).
``session``  device weights, KV pools, workspace and a session object.
``build``    compiles the HIP library for gfx950.
"""

from . import binding  # noqa: F401

__all__ = ["binding"]
