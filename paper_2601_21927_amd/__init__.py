"""SONIC segment-structured attention on MI355X (gfx950).

The path: masked prefill under the hierarchical visibility mask, KV
compaction to {system, Nexus, current}, decode over the compact cache.  All
three steps run in the HIP kernels of ``libsonic.so``; ``sonic`` is its thin
ctypes binding and ``runner`` the device-memory plumbing used by tests and the
benchmark.
"""
from . import sonic  # noqa: F401

__all__ = ["sonic"]
