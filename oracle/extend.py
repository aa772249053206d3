"""Next-turn Nexus generation over the compact cache (oracle; test infrastructure only).

When turn n of a session ends, its query and response become the body B_n of a
new history segment, and the K Nexus tokens N_n follow it (Eq.(1)).  At that
moment the compact cache of the request holds the system prompt, the Nexus
tokens of the earlier segments and, at its end, the rows of turn n, i.e. B_n.

By the mask of Sec. 3.2 a Nexus row of segment n sees
* the system prompt and every Nexus token of the earlier segments (causal,
  Eq.(3); reading A1 for Nexus keys of earlier segments),
* its own body B_n, because it is not after max(N_n) (Eq.(4)),
* every Nexus token of its own segment (Eq.(5)),
and nothing else exists yet.  So its keys are exactly the cache rows followed
by the new Nexus rows, all of them visible.  This holds under either reading of
Nexus visibility across segments (A3 or causal-across-segments), because only
the newest segment is computed here.

Afterwards the body is dropped (no later row may see it, Eq.(4)) and the new
Nexus rows take its place, so the cache reads [system, N_1, ..., N_n]: the
generated Nexus KV is kept for the rest of the session (efficiency section).

A turn is two segments: the user utterance and the assistant response each get
their own Nexus tokens (Sec. 3.1).  With body_len, only the first body_len rows
after keep_len are this step's segment; the rows after them (the response)
come later in the sequence, so by the causal rule (Eq.(3)) the new Nexus rows do
not see them, and they stay in the cache behind the new Nexus rows, to be the
body of the next step.  Two steps, utterance then response, give the Nexus rows
of both segments as computed in one prefill where a Nexus token sees the Nexus
tokens of its own and earlier segments (the response's Nexus rows see the
utterance's, and its body is hidden from them by Eq.(4)).
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64, kv_head


def extend_request(q_new, k_new, v_new, k_cache, v_cache, keep_len: int, scale=None, body_len=None):
    """One request.

    q_new [k, Hq, d], k_new / v_new [k, Hkv, d]: the new Nexus rows (bf16 bits);
    k_cache / v_cache [len, Hkv, d]: the request's cache rows 0..len (bf16 bits),
    of which the first keep_len (system and earlier Nexus) stay; body_len: the rows
    keep_len .. keep_len + body_len are the segment's body (default: all the rest).
    Returns (out [k, Hq, d] float64, cache_k [keep_len + k + rest, Hkv, d], cache_v),
    the new cache as bf16 bits, rest being the rows after the body.
    """
    k_cache = np.asarray(k_cache)
    v_cache = np.asarray(v_cache)
    if not 0 <= keep_len <= len(k_cache):
        raise ValueError(f"keep_len {keep_len} outside the cache's {len(k_cache)} rows")
    if body_len is None:
        body_len = len(k_cache) - keep_len
    if not 0 <= body_len <= len(k_cache) - keep_len:
        raise ValueError(f"body_len {body_len} outside the cache's tail of {len(k_cache) - keep_len} rows")
    seen = keep_len + body_len                           # the keys: kept rows, then the body
    qf = bf16_bits_to_f64(q_new)
    kf = np.concatenate([bf16_bits_to_f64(k_cache[:seen]), bf16_bits_to_f64(k_new)], axis=0)
    vf = np.concatenate([bf16_bits_to_f64(v_cache[:seen]), bf16_bits_to_f64(v_new)], axis=0)
    n, Hq, d = qf.shape
    Hkv = kf.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    out = np.zeros((n, Hq, d), dtype=np.float64)
    for h in range(Hq):
        g = kv_head(h, Hq, Hkv)
        s = scale * (qf[:, h, :] @ kf[:, g, :].T)        # every key is visible
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        out[:, h, :] = (e / e.sum(axis=1, keepdims=True)) @ vf[:, g, :]
    new_k = np.concatenate([k_cache[:keep_len], np.asarray(k_new), k_cache[seen:]], axis=0)
    new_v = np.concatenate([v_cache[:keep_len], np.asarray(v_new), v_cache[seen:]], axis=0)
    return out, new_k, new_v
