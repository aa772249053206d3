"""Reconstruction targets of the information bottleneck (oracle; test infrastructure only).

Sec. 4 ("Information Bottleneck and Reconstruction"): the body B_i of history
segment i is cut into K sub-intervals B_i^1 .. B_i^K, one per Nexus token of
the segment.  For the j-th Nexus token, with h() the model's hidden state,

    alpha(x)   = exp(cos(h(N_j), h(x))) / sum over y in B_i^j of exp(cos(h(N_j), h(y)))
    target_j   = sum over x in B_i^j of alpha(x) h(x)

and the loss uses cos(h(N_j), target_j) and the entropy H(alpha) normalised by
log |B_i^j|.  Readings where the paper is silent:

* A21: K is the segment's own Nexus count (the budget is per segment).  Interval
  j is [floor(j b / K), max(floor((j + 1) b / K), floor(j b / K) + 1)) of the
  body's b tokens: K near-equal consecutive pieces when b >= K; when b < K
  ("padding"), single tokens, every body token used, in order.
* A22: the entropy ratio H(alpha) / log |B| is 1 for a one-token interval (a
  single weight is as spread as it can be).
* A23: cos(a, b) = 0 when a or b is the zero vector.

Outputs are per Nexus token of the request, in position order.
"""
from __future__ import annotations

import numpy as np

from .attention import bf16_bits_to_f64
from .layout import parse


def interval(j: int, b: int, K: int):
    """[start, end) of sub-interval j of a body of b tokens cut for K Nexus tokens (A21)."""
    s = (j * b) // K
    e = max(((j + 1) * b) // K, s + 1)
    return s, e


def _cos(a, B):
    na = np.linalg.norm(a)
    nb = np.linalg.norm(B, axis=-1)
    den = na * nb
    dots = B @ a
    return np.where(den > 0, dots / np.where(den > 0, den, 1.0), 0.0)


def recon_request(h, role, turn_id):
    """For one request: (target [n, Dm], cos_target [n], entropy_ratio [n]) float64, one
    row per Nexus token in position order; h is bf16 bits [L, Dm]."""
    hf = bf16_bits_to_f64(h)
    parsed = parse(np.asarray(role), np.asarray(turn_id))
    targets, coss, ratios = [], [], []
    for seg in parsed.segments:
        K = seg.nexus_len
        for j in range(K):
            s, e = interval(j, seg.body_len, K)
            rows = hf[seg.body_start + s:seg.body_start + e]
            hn = hf[seg.nexus_start + j]
            c = _cos(hn, rows)
            w = np.exp(c)
            alpha = w / w.sum()
            t = alpha @ rows
            targets.append(t)
            coss.append(float(_cos(t, hn[None, :])[0]))
            n = len(rows)
            H = float(-(alpha * np.log(alpha)).sum())
            ratios.append(H / np.log(n) if n > 1 else 1.0)
    Dm = hf.shape[1]
    return (np.array(targets).reshape(-1, Dm), np.array(coss), np.array(ratios))
