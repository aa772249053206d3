"""KV retention after prefill (oracle; test infrastructure only).

Once prefill over the augmented sequence is done, generation may only see the
system prompt, the Nexus tokens and the current query (Sec. 3, Fig. 2
caption; Sec. 3.2 after Eq.(4); App. C): every history body entry is dropped
from the cache.  The retained entries keep their original order (reading
A13: the order is ascending position, so the result is unique).

Cache layout produced here (the layout the HIP path must reproduce bit for bit):
request b owns cache rows [row_off[b], row_off[b] + row_cap[b]); its j-th kept
token goes to row row_off[b] + j as raw bf16 bits; ``keep_idx`` at the same row
holds the request-local source position; ``length[b]`` is the kept count.
Rows from length[b] up to the capacity are left as they were.
"""
from __future__ import annotations

import numpy as np

from .layout import HISTORY_TEXT


def kept_positions(role) -> np.ndarray:
    """Request-local positions of the retained tokens, ascending."""
    role = np.asarray(role)
    return np.array([t for t in range(len(role)) if role[t] != HISTORY_TEXT], dtype=np.int32)


def compact_batch(k_bits, v_bits, role, cu_seqlens, row_off, row_cap, k_cache, v_cache, keep_idx):
    """Fill the caller's cache arrays in place; returns per-request lengths.

    k_cache, v_cache: uint16 [rows, Hkv, d]; keep_idx: int32 [rows].
    Raises OverflowError when a request keeps more rows than its capacity.
    """
    cu = np.asarray(cu_seqlens)
    lengths = np.zeros(len(cu) - 1, dtype=np.int32)
    for b in range(len(cu) - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        keep = kept_positions(role[s:e])
        if len(keep) > int(row_cap[b]):
            raise OverflowError(f"request {b} keeps {len(keep)} rows, capacity {int(row_cap[b])}")
        base = int(row_off[b])
        for j, t in enumerate(keep.tolist()):
            k_cache[base + j] = k_bits[s + t]
            v_cache[base + j] = v_bits[s + t]
            keep_idx[base + j] = t
        lengths[b] = len(keep)
    return lengths
