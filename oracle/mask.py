"""Explicit hierarchical visibility mask (oracle; test infrastructure only).

Sec. 3.2 defines an additive mask M in R^{L x L} with M[p, q] = 0 when key q is
visible to query p and -inf otherwise.  The oracle stores the boolean
``vis[p, q] = (M[p, q] == 0)`` and builds it from the three rules in the order
the section states them:

* Basic causal rule, Eq.(3): for non-Nexus pairs, visible iff q <= p.
  Reading A1/A2: the section applies causal masking globally, so a pair with
  exactly one Nexus token is also causal.
* Historical body removal, Eq.(4): once p lies after the last Nexus token of
  segment i (p > max(N_i)), every body key of B_i is masked.  Reading A4: a
  segment without Nexus tokens ends at its last body token.
* Bidirectional Nexus visibility, Eq.(5): every Nexus token sees every Nexus
  token, within and across segments (the literal "fully connected" reading,
  scope NEXUS_ALL).  Reading A3' (scope NEXUS_UP_TO_OWN): a Nexus token sees
  the Nexus tokens of its own segment and of the earlier ones, not of later
  segments.  That is what a session computes when each segment's Nexus tokens
  are generated as its turn ends, over the Nexus KV kept from the earlier
  turns (the efficiency discussion of the paper keeps that KV across turns).

Large requests are handled one block of query rows at a time; every block is
still an explicit boolean matrix.
"""
from __future__ import annotations

import numpy as np

from .layout import NEXUS, HISTORY_TEXT, Parsed, parse

NEXUS_ALL = "all"              # Eq.(5) as written
NEXUS_UP_TO_OWN = "up_to_own"  # reading A3': own and earlier segments only


def _last_of_key(parsed: Parsed) -> np.ndarray:
    """For a body key of segment i: max(N_i) (A4 fallback); +inf-like for other keys."""
    L = parsed.length
    last = np.full(L, np.iinfo(np.int64).max, dtype=np.int64)
    for s in parsed.segments:
        last[s.body_start:s.body_start + s.body_len] = s.last
    return last


def _nexus_segment(parsed: Parsed) -> np.ndarray:
    """Segment index (0, 1, ...) of each Nexus position; -1 elsewhere."""
    seg = np.full(parsed.length, -1, dtype=np.int64)
    for i, s in enumerate(parsed.segments):
        seg[s.nexus_start:s.nexus_start + s.nexus_len] = i
    return seg


def visibility_rows(role, turn_id, rows=None, parsed: Parsed = None, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """Boolean visibility of all L keys for the query positions `rows` (default: all)."""
    role = np.asarray(role)
    if parsed is None:
        parsed = parse(role, turn_id)
    L = parsed.length
    p = np.arange(L, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    P = p[:, None]
    Q = np.arange(L, dtype=np.int64)[None, :]
    nexus_p = (role[p] == NEXUS)[:, None]
    nexus_q = (role == NEXUS)[None, :]
    body_q = (role == HISTORY_TEXT)[None, :]

    # start from "everything masked" (M = -inf)
    vis = np.zeros((len(p), L), dtype=bool)
    # Eq.(3) and readings A1/A2: causal for every pair that is not Nexus-Nexus
    not_nexus_pair = ~(nexus_p & nexus_q)
    vis |= not_nexus_pair & (Q <= P)
    # Eq.(4): p > max(N_i) masks the body B_i
    last = _last_of_key(parsed)[None, :]
    vis &= ~(body_q & (P > last))
    # Eq.(5): Nexus <-> Nexus fully visible, within and across segments (A3' limits
    # the keys to the query's own and earlier segments)
    if nexus_scope == NEXUS_ALL:
        vis |= nexus_p & nexus_q
    elif nexus_scope == NEXUS_UP_TO_OWN:
        seg = _nexus_segment(parsed)
        vis |= nexus_p & nexus_q & (seg[None, :] <= seg[p][:, None])
    else:
        raise ValueError(f"unknown Nexus scope {nexus_scope!r}")
    return vis


def visibility(role, turn_id, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """The full explicit L x L boolean mask of one request."""
    return visibility_rows(role, turn_id, nexus_scope=nexus_scope)


def additive_mask(role, turn_id, nexus_scope: str = NEXUS_ALL) -> np.ndarray:
    """M itself: 0 where visible, -inf where masked (float64)."""
    vis = visibility(role, turn_id, nexus_scope)
    return np.where(vis, 0.0, -np.inf)
