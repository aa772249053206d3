"""Shared pieces of the GPU parity tests: tolerances, row sampling, device plumbing."""
import sys

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attention as OA
from oracle import compaction as OC
from oracle import decode as OD
from oracle import layout as OL
from oracle import mask as OM

# Attention tolerance for bf16 inputs with fp32 accumulation, against the fp64 oracle.
MAX_ABS = 1e-2
MEAN_ABS = 1e-3


def need_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    from paper_2601_21927_amd import sonic
    sonic.lib()   # raises if libsonic.so is not built: no fallback


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def assert_close(got, want, what):
    err = np.abs(np.asarray(got, np.float64) - np.asarray(want, np.float64))
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    note(f"  {what}: max_abs={mx:.3e} mean_abs={mean:.3e} n={err.size}")
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert mx <= MAX_ABS, f"{what}: max abs error {mx:.3e} > {MAX_ABS}"
    assert mean <= MEAN_ABS, f"{what}: mean abs error {mean:.3e} > {MEAN_ABS}"
    return mx, mean


def run_starts(lay: W.RequestLayout):
    """Request-local starts of the runs (maximal ranges of one role and one segment)."""
    role, turn = lay.roles_and_turns()
    return [0] + [i for i in range(1, lay.length) if role[i] != role[i - 1] or turn[i] != turn[i - 1]]


def sample_rows(lay: W.RequestLayout, rng, every=None, extra=16):
    """Request-local rows to check: the first and last row of every run, rows around every
    32-row block edge inside runs, the last row of every 32-row block of the request, and a
    few random rows."""
    L = lay.length
    if L == 0:
        return np.zeros(0, np.int64)
    rows = set([0, L - 1])
    for s in run_starts(lay):
        for r in (s - 1, s, s + 1, s + 31, s + 32, s + 33):
            if 0 <= r < L:
                rows.add(r)
    rows.update(range(31, L, 32))
    rows.update(int(x) for x in rng.integers(0, L, size=extra))
    if every:
        rows.update(range(0, L, every))
    return np.array(sorted(rows), np.int64)


def subset_rows(lay: W.RequestLayout, margin=64, every=16):
    """The deterministic row subset of a long request: every system, Nexus and current row;
    the `margin` rows on either side of every run boundary; every `every`-th body row; and the
    last row of every 32-row block."""
    role, _ = lay.roles_and_turns()
    L = lay.length
    keep = role != W.ROLE_HISTORY_TEXT
    for s in run_starts(lay):
        keep[max(0, s - margin):min(L, s + margin)] = True
    body = np.flatnonzero(role == W.ROLE_HISTORY_TEXT)
    keep[body[body % every == 0]] = True
    keep[31::32] = True
    if L:
        keep[L - 1] = True
    return np.flatnonzero(keep).astype(np.int64)


def oracle_prefill_rows(batch: W.Batch, rows_per_req, nexus_scope=OM.NEXUS_ALL):
    outs = []
    cu = batch.cu_seqlens
    for b, rows in enumerate(rows_per_req):
        s, e = int(cu[b]), int(cu[b + 1])
        if len(rows) == 0:
            outs.append(np.zeros((0, batch.num_q_heads, batch.head_dim)))
            continue
        outs.append(OA.prefill_request(batch.q[s:e], batch.k[s:e], batch.v[s:e], batch.role[s:e],
                                       batch.turn_id[s:e], rows=rows, nexus_scope=nexus_scope))
    return outs


def device_batch(batch: W.Batch):
    from paper_2601_21927_amd.runner import SonicBatch
    return SonicBatch(batch.role, batch.turn_id, batch.cu_seqlens, batch.q, batch.k, batch.v)


def oracle_compact(batch: W.Batch, caps, fill=0xFFFF):
    cu = batch.cu_seqlens
    caps = np.asarray(caps, np.int64)
    off = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    rows = int(caps.sum())
    kc = np.full((max(rows, 1), batch.num_kv_heads, batch.head_dim), fill, np.uint16)
    vc = np.full_like(kc, fill)
    ki = np.full(max(rows, 1), -1, np.int32)
    n = OC.compact_batch(batch.k, batch.v, batch.role, cu, off, caps, kc, vc, ki)
    return kc, vc, ki, n, off


def kept_counts(batch: W.Batch):
    return np.array([lay.system + sum(lay.nexus) + lay.current for lay in batch.layouts], np.int64)
