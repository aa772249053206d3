"""Dense masked softmax attention in float64 (oracle; test infrastructure only).

For every query position p of a request and every query head h (Sec. 3.2 with
standard scaled dot-product attention, the Transformer block the method sits
in):

    s[p, q]  = scale * <Q[p, h], K[q, g(h)]>            for every key q (dense)
    P[p, :]  = softmax over the keys with vis[p, q]      (masked keys get 0)
    O[p, h]  = sum_q P[p, q] * V[q, g(h)]

Readings where the paper is silent: grouped-query heads map q-head h to
kv-head g(h) = floor(h / (Hq / Hkv)) (A6); scale defaults to 1/sqrt(d) (A7);
the -inf entries of M are applied as boolean exclusion, which is the same
thing because every row sees at least its own position (A11).
"""
from __future__ import annotations

import numpy as np

from .layout import Parsed, parse
from .mask import NEXUS_ALL, visibility_rows


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def kv_head(h: int, num_q_heads: int, num_kv_heads: int) -> int:
    group = num_q_heads // num_kv_heads
    return h // group


def softmax_probs(scores: np.ndarray, vis: np.ndarray) -> np.ndarray:
    """Row softmax over the visible entries; masked entries are exactly 0."""
    s = np.where(vis, scores, -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.where(vis, np.exp(s - m), 0.0)
    return e / e.sum(axis=1, keepdims=True)


def request_probs(q, k, role, turn_id, h: int, scale=None, rows=None, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """Attention probabilities P[rows, :] of q-head h of one request (float64)."""
    qf = bf16_bits_to_f64(q)
    kf = bf16_bits_to_f64(k)
    Hq, Hkv, d = qf.shape[1], kf.shape[1], qf.shape[2]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    L = qf.shape[0]
    r = np.arange(L) if rows is None else np.asarray(rows)
    vis = visibility_rows(role, turn_id, r, nexus_scope=nexus_scope)
    g = kv_head(h, Hq, Hkv)
    scores = scale * (qf[r, h, :] @ kf[:, g, :].T)
    return softmax_probs(scores, vis)


def prefill_request(q, k, v, role, turn_id, scale=None, rows=None, block=512,
                    parsed: Parsed = None, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """O[rows, Hq, d] for one request: dense scores, explicit mask, softmax, P @ V.

    Per block of query rows the mask is built over every key; key columns that no
    row of the block sees are then left out of the products.  Their entries of M
    are -inf (Sec. 3.2), so their probabilities are exactly 0 and the result is
    the same softmax over the same visible keys."""
    kf = bf16_bits_to_f64(k)
    vf = bf16_bits_to_f64(v)
    L, Hq, d = q.shape
    Hkv = kf.shape[1]
    if Hq % Hkv:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    if parsed is None:
        parsed = parse(role, turn_id)
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.zeros((len(rows), Hq, d), dtype=np.float64)
    for r0 in range(0, len(rows), block):
        rb = rows[r0:r0 + block]
        qf = bf16_bits_to_f64(q[rb])          # only the query rows of this block
        vis = visibility_rows(role, turn_id, rb, parsed=parsed, nexus_scope=nexus_scope)
        cols = np.flatnonzero(vis.any(axis=0))   # keys some row of the block sees
        vis = vis[:, cols]
        for h in range(Hq):
            g = kv_head(h, Hq, Hkv)
            scores = scale * (qf[:, h, :] @ kf[cols, g, :].T)
            probs = softmax_probs(scores, vis)
            out[r0:r0 + len(rb), h, :] = probs @ vf[cols, g, :]
    return out


def prefill_batch(q, k, v, role, turn_id, cu_seqlens, scale=None, rows_per_request=None):
    """Per-request outputs of a packed batch.  `rows_per_request[b]` optionally selects
    request-local query rows; returns a list of float64 arrays [rows, Hq, d]."""
    cu = np.asarray(cu_seqlens)
    outs = []
    for b in range(len(cu) - 1):
        s, e = int(cu[b]), int(cu[b + 1])
        rows = None if rows_per_request is None else rows_per_request[b]
        outs.append(prefill_request(q[s:e], k[s:e], v[s:e], role[s:e], turn_id[s:e], scale, rows))
    return outs
