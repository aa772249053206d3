"""Oracle prefill rows of the seeded workloads, computed in worker processes.

Test infrastructure: the workers regenerate a workload from its seed (the same
bits the GPU receives) and run the fp64 oracle on groups of rows.  They import
only numpy, `workloads` and `oracle`; nothing here touches the GPU, and the
pool is started with the "spawn" method so that no worker inherits the parent's
GPU state.
"""
from __future__ import annotations

import concurrent.futures
import multiprocessing
import os

import numpy as np

import workloads as W
from oracle import attention as OA

MAX_WORKERS = 16            # the host-CPU share of one GPU
ROWS_PER_JOB = 512

_batches = {}


def _workload(idx: int) -> W.Batch:
    if idx not in _batches:
        _batches.clear()
        _batches[idx] = W.workload(idx, decode_steps=0)
    return _batches[idx]


def _job(args):
    idx, b, rows, scope = args
    batch = _workload(idx)
    s, e = int(batch.cu_seqlens[b]), int(batch.cu_seqlens[b + 1])
    return OA.prefill_request(batch.q[s:e], batch.k[s:e], batch.v[s:e], batch.role[s:e], batch.turn_id[s:e],
                              rows=rows, nexus_scope=scope)


def run_ids(lay: W.RequestLayout) -> np.ndarray:
    """Index of the run (maximal range of one role and one segment) of every position."""
    role, turn = lay.roles_and_turns()
    change = np.ones(len(role), bool)
    change[1:] = (role[1:] != role[:-1]) | (turn[1:] != turn[:-1])
    return np.cumsum(change) - 1


def workload_rows(idx: int, rows_per_req: dict, scope=None, workers: int = None) -> dict:
    """{request: oracle output [len(rows), Hq, d]} for request-local rows of workload `idx`.
    Rows are grouped by run (so a group's visible keys are few) and split into jobs."""
    from oracle import mask as OM
    scope = OM.NEXUS_ALL if scope is None else scope
    lays = W.workload_structure(idx)["layouts"]
    jobs, where = [], []
    for b, rows in rows_per_req.items():
        rows = np.asarray(rows, np.int64)
        rid = run_ids(lays[b])[rows]
        for r in np.unique(rid):
            sel = np.flatnonzero(rid == r)
            for j in range(0, len(sel), ROWS_PER_JOB):
                part = sel[j:j + ROWS_PER_JOB]
                jobs.append((idx, b, rows[part], scope))
                where.append((b, part))
    n = workers or min(MAX_WORKERS, len(os.sched_getaffinity(0)), max(1, len(jobs)))
    # one BLAS thread per worker; set before the workers start (they read it at import)
    saved = {k: os.environ.get(k) for k in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS")}
    os.environ["OPENBLAS_NUM_THREADS"] = "1"
    os.environ["OMP_NUM_THREADS"] = "1"
    try:
        ctx = multiprocessing.get_context("spawn")
        with concurrent.futures.ProcessPoolExecutor(max_workers=n, mp_context=ctx) as ex:
            results = list(ex.map(_job, jobs))
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    st = W.workload_structure(idx)
    Hq, d = st["Hq"], st["d"]
    out = {b: np.zeros((len(rows), Hq, d)) for b, rows in rows_per_req.items()}
    for (b, part), res in zip(where, results):
        out[b][part] = res
    return out
