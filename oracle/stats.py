"""Attention statistics of the masked prefill (oracle; test infrastructure only).

Two quantities the paper's training objectives are built from (Sec. 4):

* Nexus attention mass (Nexus attention regularisation): how much attention a
  query row puts on Nexus tokens.  Per query row p and q-head h,
      A_nexus[p, h] = sum over Nexus keys x of P_h[p, x],
  where P_h is the masked softmax of Sec. 3.2.  The loss averages it over the
  current query's rows (and heads); the per-(row, head) mass is the building
  block (reading A19).
* Key importance (attention-guided distillation): the attention a key receives
  from the current rows, averaged over the heads,
      w(x) = (1 / Hq) * sum over q-heads h, sum over CURRENT rows p of P_h[p, x].
  The paper takes it from the teacher's attention; here it is taken from
  whatever mask the prefill runs with (reading A20).

Both come straight from the explicit probabilities of oracle.attention.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64, kv_head, softmax_probs
from .layout import CURRENT, NEXUS, parse
from .mask import NEXUS_ALL, visibility_rows


def _probs(qf, kf, h, g, vis, scale):
    return softmax_probs(scale * (qf[:, h, :] @ kf[:, g, :].T), vis)


def nexus_mass(q, k, role, turn_id, scale=None, rows=None, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """A_nexus[rows, Hq] of one request (float64)."""
    role = np.asarray(role)
    L, Hq, d = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    parsed = parse(role, turn_id)
    vis = visibility_rows(role, turn_id, rows, parsed=parsed, nexus_scope=nexus_scope)
    qf = bf16_bits_to_f64(q[rows])
    kf = bf16_bits_to_f64(k)
    is_nexus = role == NEXUS
    out = np.zeros((len(rows), Hq), dtype=np.float64)
    for h in range(Hq):
        P = _probs(qf, kf, h, kv_head(h, Hq, Hkv), vis, scale)
        out[:, h] = P[:, is_nexus].sum(axis=1)
    return out


def key_weight(q, k, role, turn_id, scale=None, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """w[L] of one request (float64): head-averaged attention received from CURRENT rows."""
    role = np.asarray(role)
    L, Hq, d = q.shape
    Hkv = k.shape[1]
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    cur = np.nonzero(role == CURRENT)[0]
    w = np.zeros(L, dtype=np.float64)
    if len(cur) == 0:
        return w
    parsed = parse(role, turn_id)
    vis = visibility_rows(role, turn_id, cur, parsed=parsed, nexus_scope=nexus_scope)
    qf = bf16_bits_to_f64(q[cur])
    kf = bf16_bits_to_f64(k)
    for h in range(Hq):
        w += _probs(qf, kf, h, kv_head(h, Hq, Hkv), vis, scale).sum(axis=0)
    return w / Hq
