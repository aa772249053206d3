"""Augmented-sequence grammar and segment index sets (oracle; test infrastructure only).

Sec. 3.1, Eq.(1): a request is laid out as
    { I_sys, m_1, N^(1), m_2, N^(2), ..., m_h, N^(h), Q_curr }
with the Nexus tokens N^(i) appended after the body of history segment m_i.
Sec. 3.2 names, per segment i, the body index set B_i and the Nexus index set
N_i.  This module checks a per-token (role, segment id) description against
that grammar and returns those sets.

Readings where the paper is silent:
* A segment may carry zero Nexus tokens (the budget can drop below the body
  length, Sec. 4.2 and 4.3); a body must hold at least one token.
* The segment id only separates adjacent segments; it must be constant within
  a segment (body and its Nexus) and strictly increase from one history
  segment to the next.  Ids of system and current tokens are ignored.
"""
from __future__ import annotations

import dataclasses
from typing import List

import numpy as np

SYSTEM = 0
HISTORY_TEXT = 1
NEXUS = 2
CURRENT = 3


class LayoutError(ValueError):
    """The role/segment sequence does not follow the augmented-sequence grammar."""


@dataclasses.dataclass
class Segment:
    body_start: int
    body_len: int
    nexus_start: int
    nexus_len: int
    turn: int

    @property
    def body(self) -> range:          # B_i
        return range(self.body_start, self.body_start + self.body_len)

    @property
    def nexus(self) -> range:         # N_i
        return range(self.nexus_start, self.nexus_start + self.nexus_len)

    @property
    def last(self) -> int:
        """max(N_i); for a segment without Nexus tokens, its last body position."""
        if self.nexus_len > 0:
            return self.nexus_start + self.nexus_len - 1
        return self.body_start + self.body_len - 1


@dataclasses.dataclass
class Parsed:
    length: int
    system: int                 # |I_sys|
    segments: List[Segment]
    current_start: int
    current: int                # |Q_curr|


def parse(role, turn_id) -> Parsed:
    """Walk one request's tokens left to right and split them per Eq.(1)."""
    role = np.asarray(role)
    turn_id = np.asarray(turn_id)
    L = len(role)
    if len(turn_id) != L:
        raise LayoutError("role and turn_id lengths differ")
    for r in role.tolist():
        if r not in (SYSTEM, HISTORY_TEXT, NEXUS, CURRENT):
            raise LayoutError(f"unknown role code {r}")
    p = 0
    while p < L and role[p] == SYSTEM:
        p += 1
    system = p
    segments: List[Segment] = []
    while p < L and role[p] == HISTORY_TEXT:
        t = int(turn_id[p])
        if segments and t <= segments[-1].turn:
            raise LayoutError(f"segment id {t} at {p} does not increase")
        b0 = p
        while p < L and role[p] == HISTORY_TEXT and int(turn_id[p]) == t:
            p += 1
        n0 = p
        while p < L and role[p] == NEXUS:
            if int(turn_id[p]) != t:
                raise LayoutError(f"Nexus token at {p} has segment id {turn_id[p]} != {t}")
            p += 1
        segments.append(Segment(b0, n0 - b0, n0, p - n0, t))
    c0 = p
    while p < L and role[p] == CURRENT:
        p += 1
    if p != L:
        raise LayoutError(f"token {p} (role {int(role[p])}) breaks the augmented-sequence order")
    return Parsed(L, system, segments, c0, L - c0)


def parse_batch(role, turn_id, cu_seqlens) -> List[Parsed]:
    cu = np.asarray(cu_seqlens)
    if len(cu) == 0 or cu[0] != 0 or np.any(np.diff(cu) < 0):
        raise LayoutError("cu_seqlens must start at 0 and not decrease")
    return [parse(role[cu[b]:cu[b + 1]], turn_id[cu[b]:cu[b + 1]]) for b in range(len(cu) - 1)]


def segment_of_token(parsed: Parsed) -> np.ndarray:
    """Index (0-based) of the history segment owning each token, -1 for system/current."""
    seg = np.full(parsed.length, -1, dtype=np.int64)
    for i, s in enumerate(parsed.segments):
        seg[s.body_start:s.nexus_start + s.nexus_len] = i
    return seg
