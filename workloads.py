"""Seeded synthetic inputs for the SONIC segment-attention path.

This module is shared, as *input only*, by the fp64 oracle (``oracle/``) and by
the HIP path (``paper_2601_21927_amd``).  It holds none of the method's
arithmetic: it draws token layouts (roles and segment ids in the order of the
augmented sequence of Eq.(1), Sec. 3.1) and bf16 Q/K/V bit patterns, nothing
else.  Neither the mask rules nor attention nor compaction appear here.

Role codes follow the token classes named in Sec. 3.1-3.2: system prompt,
history body text, Nexus token, current query.

Recipe: the structure (and per-head scales) is drawn first from
numpy PCG64 seeded with the workload number; then each tensor (Q, K, V, per-step
decode q, k, v) is drawn as N(0,1) float32 in blocks of 2^22 values, block j of
tensor t from PCG64(SeedSequence([seed, t, j])).  fp32 samples are rounded to
bf16 by round-to-nearest-even and handed over as raw uint16 bit patterns, so
both sides read identical bits.
"""
from __future__ import annotations

import dataclasses
import os
from typing import List, Optional, Sequence

import numpy as np

ROLE_SYSTEM = 0
ROLE_HISTORY_TEXT = 1
ROLE_NEXUS = 2
ROLE_CURRENT = 3


# ---------------------------------------------------------------------------
# bf16 encoding (input encoding only)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even), return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # finite inputs only (the generators draw normals): the sum cannot wrap in 32 bits
    r = (u >> 16) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= 16
    return r.astype(np.uint16)


# ---------------------------------------------------------------------------
# layouts
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class RequestLayout:
    """One request of the augmented sequence {I_sys, m_1, N^(1), ..., m_h, N^(h), Q_curr}."""
    system: int
    bodies: List[int]
    nexus: List[int]
    current: int

    @property
    def length(self) -> int:
        return self.system + sum(self.bodies) + sum(self.nexus) + self.current

    def roles_and_turns(self, first_turn: int = 1):
        """Per-token role codes and segment ids (segment i of the history gets id first_turn+i)."""
        role = np.empty(self.length, dtype=np.uint8)
        turn = np.empty(self.length, dtype=np.int32)
        p = 0
        role[p:p + self.system] = ROLE_SYSTEM
        turn[p:p + self.system] = 0
        p += self.system
        for i, (b, k) in enumerate(zip(self.bodies, self.nexus)):
            role[p:p + b] = ROLE_HISTORY_TEXT
            turn[p:p + b] = first_turn + i
            p += b
            role[p:p + k] = ROLE_NEXUS
            turn[p:p + k] = first_turn + i
            p += k
        role[p:p + self.current] = ROLE_CURRENT
        turn[p:p + self.current] = first_turn + len(self.bodies)
        p += self.current
        assert p == self.length
        return role, turn


@dataclasses.dataclass
class Batch:
    """A packed (varlen) batch: token-major tensors, request b at rows cu[b]:cu[b+1]."""
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    layouts: List[RequestLayout]
    role: np.ndarray            # uint8 [T]
    turn_id: np.ndarray         # int32 [T]
    cu_seqlens: np.ndarray      # int32 [B+1]
    q: Optional[np.ndarray] = None   # uint16 bf16 bits [T, Hq, d]
    k: Optional[np.ndarray] = None   # uint16 bf16 bits [T, Hkv, d]
    v: Optional[np.ndarray] = None   # uint16 bf16 bits [T, Hkv, d]
    decode_steps: int = 0
    dec_q: Optional[np.ndarray] = None   # uint16 [steps, B, Hq, d]
    dec_k: Optional[np.ndarray] = None   # uint16 [steps, B, Hkv, d]
    dec_v: Optional[np.ndarray] = None   # uint16 [steps, B, Hkv, d]
    scale_q: Optional[np.ndarray] = None
    scale_k: Optional[np.ndarray] = None
    scale_v: Optional[np.ndarray] = None

    @property
    def batch(self) -> int:
        return len(self.layouts)

    @property
    def total_tokens(self) -> int:
        return int(self.cu_seqlens[-1])

    @property
    def max_seqlen(self) -> int:
        if self.batch == 0:
            return 0
        return int(np.max(np.diff(self.cu_seqlens)))


def pack_layouts(layouts: Sequence[RequestLayout]):
    roles, turns, cu = [], [], [0]
    for lay in layouts:
        r, t = lay.roles_and_turns()
        roles.append(r)
        turns.append(t)
        cu.append(cu[-1] + lay.length)
    role = np.concatenate(roles) if roles else np.zeros(0, np.uint8)
    turn = np.concatenate(turns) if turns else np.zeros(0, np.int32)
    return role.astype(np.uint8), turn.astype(np.int32), np.asarray(cu, dtype=np.int32)


_BLOCK = 1 << 22   # values per independent generator block


def _normal_bf16(seed, tensor_id: int, shape, scale=None) -> np.ndarray:
    """N(0,1) (times an optional broadcast scale) rounded to bf16, drawn block by block:
    block j of tensor `tensor_id` comes from PCG64(SeedSequence([seed, tensor_id, j])), so the
    bytes do not depend on how many threads fill the blocks."""
    shape = tuple(int(x) for x in shape)
    n = int(np.prod(shape)) if shape else 1
    out = np.empty(n, dtype=np.uint16)
    sc = None if scale is None else np.broadcast_to(np.asarray(scale, np.float32), shape).reshape(-1)

    def fill(j):
        a, e = j * _BLOCK, min(n, (j + 1) * _BLOCK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed), int(tensor_id), j])))
        x = g.standard_normal(e - a, dtype=np.float32)
        if sc is not None:
            x *= sc[a:e]
        out[a:e] = f32_to_bf16_bits(x)

    nblocks = (n + _BLOCK - 1) // _BLOCK
    if nblocks <= 1:
        for j in range(nblocks):
            fill(j)
    else:
        import concurrent.futures
        workers = min(nblocks, max(1, min(16, os.cpu_count() or 1)))
        with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(fill, range(nblocks)))
    return out.reshape(shape)


def _draw_tensors(rng, batch: Batch, scales: bool, decode_steps: int, seed: int, with_q: bool = True):
    """Per-head scales come from the structure stream `rng`; the tensors from per-block streams
    keyed by `seed` and a fixed tensor id (1 Q, 2 K, 3 V, 4 decode q, 5 decode k, 6 decode v)."""
    T, Hq, Hkv, d = batch.total_tokens, batch.num_q_heads, batch.num_kv_heads, batch.head_dim
    sq = sk = sv = None
    if scales:
        sq = rng.uniform(0.5, 2.0, size=Hq)
        sk = rng.uniform(0.5, 2.0, size=Hkv)
        sv = rng.uniform(0.5, 2.0, size=Hkv)
        batch.scale_q, batch.scale_k, batch.scale_v = sq, sk, sv
    hs = lambda s: None if s is None else s[:, None]
    if with_q:
        batch.q = _normal_bf16(seed, 1, (T, Hq, d), hs(sq))
    batch.k = _normal_bf16(seed, 2, (T, Hkv, d), hs(sk))
    batch.v = _normal_bf16(seed, 3, (T, Hkv, d), hs(sv))
    B = batch.batch
    batch.decode_steps = decode_steps
    if decode_steps:
        batch.dec_q = _normal_bf16(seed, 4, (decode_steps, B, Hq, d), hs(sq))
        batch.dec_k = _normal_bf16(seed, 5, (decode_steps, B, Hkv, d), hs(sk))
        batch.dec_v = _normal_bf16(seed, 6, (decode_steps, B, Hkv, d), hs(sv))


def make_batch(name, layouts, Hq, Hkv, d, seed, decode_steps=0, scales=False, tensors=True) -> Batch:
    role, turn, cu = pack_layouts(layouts)
    b = Batch(name=name, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d, layouts=list(layouts),
              role=role, turn_id=turn, cu_seqlens=cu)
    if tensors:
        rng = np.random.default_rng(seed)
        _draw_tensors(rng, b, scales, decode_steps, seed)
    return b


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------
WORKLOADS = {
    1: "tiny: B=1, 4/2 heads, d=64, S=32, 3 x (128 text + 8 Nexus), C=64, 16 decode steps",
    2: "llama3-8b-shape: B=8, 32/8 heads, d=128, S=256, 8 x (512 text + 102 Nexus), C=256, 256 decode steps",
    3: "ragged-50pct: B=16, 32/8 heads, d=128, h~U{2..12}, b~U{64..1024}, k=b/2, S~U{128..512}, "
       "C~U{32..512}, per-head scales U[0.5,2], 256 decode steps",
    4: "long-dialogue: B=4, 28/4 heads, d=128, S=512, 32 x (1024 text + 204 Nexus), C=512, 512 decode steps",
    5: "dynamic-budget decode: B=64, 32/8 heads, d=128, full context U{1024..8192}, budget {10,20,50}%, "
       "1024 decode steps",
}


def _uniform_layouts(n, S, b, k, h, C):
    return [RequestLayout(S, [b] * h, [k] * h, C) for _ in range(n)]


def workload_structure(index: int) -> dict:
    """Layouts and head shapes of a workload, drawn first from its seeded generator."""
    rng = np.random.default_rng(index)
    if index == 1:
        return dict(layouts=_uniform_layouts(1, 32, 128, 8, 3, 64), Hq=4, Hkv=2, d=64, steps=16, scales=False)
    if index == 2:
        return dict(layouts=_uniform_layouts(8, 256, 512, 102, 8, 256), Hq=32, Hkv=8, d=128, steps=256,
                    scales=False)
    if index == 3:
        lays = []
        for _ in range(16):
            h = int(rng.integers(2, 13))
            S = int(rng.integers(128, 513))
            bodies = [int(x) for x in rng.integers(64, 1025, size=h)]
            nexus = [b // 2 for b in bodies]
            C = int(rng.integers(32, 513))
            lays.append(RequestLayout(S, bodies, nexus, C))
        return dict(layouts=lays, Hq=32, Hkv=8, d=128, steps=256, scales=True, rng=rng)
    if index == 4:
        return dict(layouts=_uniform_layouts(4, 512, 1024, 204, 32, 512), Hq=28, Hkv=4, d=128, steps=512,
                    scales=False)
    if index == 5:
        lays, ratios, full = [], [], []
        for _ in range(64):
            L_full = int(rng.integers(1024, 8193))
            r = float(rng.choice([0.1, 0.2, 0.5]))
            S = int(rng.integers(64, 257))
            C = int(rng.integers(32, 257))
            hist = L_full - S - C
            bodies = []
            while hist > 0:
                b = int(rng.integers(64, 1025))
                if b >= hist:
                    b = hist
                bodies.append(b)
                hist -= b
            if len(bodies) > 1 and bodies[-1] < 64:
                tail = bodies.pop()
                bodies[-1] += tail
            nexus = [max(1, int(np.floor(r * b))) for b in bodies]
            lays.append(RequestLayout(S, bodies, nexus, C))
            ratios.append(r)
            full.append(L_full)
        return dict(layouts=lays, Hq=32, Hkv=8, d=128, steps=1024, scales=False, ratios=ratios,
                    full_lengths=full, rng=rng)
    raise ValueError(f"unknown workload {index}")


def workload(index: int, tensors: bool = True, decode_steps: Optional[int] = None) -> Batch:
    """Build workload `index` (1..5).  The structure draw precedes the tensor draws on one stream."""
    st = workload_structure(index)
    # structures drawn from the stream continue on it; uniform ones draw nothing first
    rng = st["rng"] if "rng" in st else np.random.default_rng(index)
    role, turn, cu = pack_layouts(st["layouts"])
    b = Batch(name=f"workload{index}", num_q_heads=st["Hq"], num_kv_heads=st["Hkv"], head_dim=st["d"],
              layouts=st["layouts"], role=role, turn_id=turn, cu_seqlens=cu)
    steps = st["steps"] if decode_steps is None else decode_steps
    b.decode_steps = steps
    if tensors:
        # the dynamic-budget workload is decode-only: its caches come from K/V, it needs no prefill Q
        _draw_tensors(rng, b, st["scales"], steps, index, with_q=(index != 5))
    if index == 5:
        b.ratios = st["ratios"]
        b.full_lengths = st["full_lengths"]
    return b


def random_layout(rng: np.random.Generator, max_h=4, max_b=80, max_k=40, max_s=70, max_c=70,
                  allow_empty_body=False) -> RequestLayout:
    """A random well-formed layout for property tests (any part may be empty except bodies)."""
    h = int(rng.integers(0, max_h + 1))
    lo = 0 if allow_empty_body else 1
    bodies = [int(x) for x in rng.integers(lo if lo else 1, max_b + 1, size=h)]
    nexus = [int(x) for x in rng.integers(0, max_k + 1, size=h)]
    return RequestLayout(int(rng.integers(0, max_s + 1)), bodies, nexus, int(rng.integers(0, max_c + 1)))


def extend_positions(lay: RequestLayout):
    """Positions (in the layout) of a next-turn Nexus step for the layout's last segment:
    (cache rows in order: system, earlier segments' Nexus, the last body; rows kept
    afterwards; positions of the last segment's Nexus rows).  The layout must have at
    least one segment and no current-query tokens."""
    if not lay.bodies or lay.current:
        raise ValueError("needs a history segment last and no current query")
    p = lay.system
    cache = list(range(lay.system))
    for i, (b, k) in enumerate(zip(lay.bodies, lay.nexus)):
        last = i == len(lay.bodies) - 1
        if last:
            cache += list(range(p, p + b))
            nexus = list(range(p + b, p + b + k))
        else:
            cache += list(range(p + b, p + b + k))
        p += b + k
    keep = lay.system + sum(lay.nexus[:-1])
    return np.array(cache, np.int64), keep, np.array(nexus, np.int64)


def turn_positions(lay: RequestLayout):
    """Positions (in the layout) of a turn of two segments, the layout's last two (an
    utterance U, then a response R): (cache rows in order: system, the earlier segments'
    Nexus, U's body, R's body; rows kept; U's body length; positions of U's Nexus rows;
    positions of R's Nexus rows).  The layout must have at least two segments and no
    current-query tokens."""
    h = len(lay.bodies)
    if h < 2 or lay.current:
        raise ValueError("needs two history segments last and no current query")
    p = lay.system
    cache = list(range(lay.system))
    starts = []
    for i, (b, k) in enumerate(zip(lay.bodies, lay.nexus)):
        starts.append(p)
        if i < h - 2:
            cache += list(range(p + b, p + b + k))
        p += b + k
    u0, r0 = starts[h - 2], starts[h - 1]
    ub, rb = lay.bodies[h - 2], lay.bodies[h - 1]
    cache += list(range(u0, u0 + ub)) + list(range(r0, r0 + rb))
    keep = lay.system + sum(lay.nexus[:h - 2])
    nu = np.arange(u0 + ub, u0 + ub + lay.nexus[h - 2])
    nr = np.arange(r0 + rb, r0 + rb + lay.nexus[h - 1])
    return np.array(cache, np.int64), keep, ub, nu, nr


def text_only_layout(lay: RequestLayout) -> RequestLayout:
    """The same conversation without Nexus tokens: what a full-context model keeps."""
    return RequestLayout(lay.system, list(lay.bodies), [0] * len(lay.bodies), lay.current)
