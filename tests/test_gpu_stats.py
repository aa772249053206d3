"""Attention statistics of the prefill on the GPU against the fp64 oracle.

nexus_mass (per row and q-head) and key_weight (per key) are sums of fp32
probabilities computed from fp32 scores of bf16 inputs (exact products, fp32
accumulation), so they are checked to |got - want| <= 1e-5 + 1e-4 |want|: a
score carries a relative error of about 1e-7 (|s| below 20 here), a probability
about 2e-6 after exp2 and the normaliser, and the sums add at most a few
thousand such terms in fp32.  The attention output of the statistics variant must equal the plain
prefill's bit for bit (the extra sums do not touch its arithmetic), and the key
weights must not change from run to run.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import layout as OL
from oracle import mask as OM
from oracle import stats as OS
from paper_2601_21927_amd import sonic
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu

ATOL, RTOL = 1e-5, 1e-4


def close(got, want, what):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    err = np.abs(got - want)
    H.note(f"  {what}: max_abs={err.max() if err.size else 0:.3e} n={err.size}")
    assert np.all(np.isfinite(got)), what
    assert np.all(err <= ATOL + RTOL * np.abs(want)), f"{what}: max error {err.max():.3e}"


def run_stats(batch, scope=sonic.NEXUS_ALL, mass=True, weight=True):
    H.need_gpu()
    db = H.device_batch(batch)
    T, Hq = batch.total_tokens, batch.num_q_heads
    nm = torch.full((max(T, 1), Hq), float("nan"), dtype=torch.float32, device="cuda") if mass else None
    kw = torch.full((max(T, 1),), float("nan"), dtype=torch.float32, device="cuda") if weight else None
    st = db.prefill(nexus_scope=scope, nexus_mass=nm, key_weight=kw)
    assert st == sonic.OK, sonic.status_string(st)
    torch.cuda.synchronize()
    assert db.read_status() == 0, sonic.status_string(db.read_status())
    return db, (nm.cpu().numpy()[:T] if mass else None), (kw.cpu().numpy()[:T] if weight else None)


def oracle_scope(scope):
    return OM.NEXUS_ALL if scope == sonic.NEXUS_ALL else OM.NEXUS_UP_TO_OWN


def check_batch(batch, scope, mass, weight):
    cu = batch.cu_seqlens
    for b in range(batch.batch):
        s, e = int(cu[b]), int(cu[b + 1])
        if e == s:
            continue
        args = (batch.q[s:e], batch.k[s:e], batch.role[s:e], batch.turn_id[s:e])
        close(mass[s:e], OS.nexus_mass(*args, nexus_scope=oracle_scope(scope)), f"{batch.name} A_nexus req {b}")
        close(weight[s:e], OS.key_weight(*args, nexus_scope=oracle_scope(scope)), f"{batch.name} w(x) req {b}")


@pytest.mark.parametrize("Hq,Hkv,d,scope", [(4, 2, 64, sonic.NEXUS_ALL), (8, 2, 128, sonic.NEXUS_ALL),
                                             (32, 8, 128, sonic.NEXUS_UP_TO_OWN), (7, 1, 128, sonic.NEXUS_ALL),
                                             (6, 2, 64, sonic.NEXUS_UP_TO_OWN)])
def test_stats_random_layouts(Hq, Hkv, d, scope):
    rng = np.random.default_rng(700 + Hq + Hkv + d + scope)
    lays = [W.random_layout(rng, max_h=4, max_b=90, max_k=45, max_s=70, max_c=100) for _ in range(3)]
    H.note(f"stats random Hq={Hq} Hkv={Hkv} d={d} scope={scope}: {[l.length for l in lays]}")
    batch = W.make_batch("stats", lays, Hq, Hkv, d, seed=int(rng.integers(1 << 30)))
    _, mass, weight = run_stats(batch, scope)
    check_batch(batch, scope, mass, weight)


def test_stats_edge_layouts():
    """No current rows (all weights 0), no Nexus (all masses 0), an empty request, one token,
    current rows only, and blocks of exactly 64 kept keys."""
    lays = [W.RequestLayout(5, [9, 4], [3, 2], 0), W.RequestLayout(4, [10, 7], [0, 0], 6),
            W.RequestLayout(0, [], [], 0), W.RequestLayout(1, [], [], 0), W.RequestLayout(0, [], [], 70),
            W.RequestLayout(32, [40], [32], 64)]
    batch = W.make_batch("stats-edge", lays, 8, 2, 128, seed=17)
    _, mass, weight = run_stats(batch)
    check_batch(batch, sonic.NEXUS_ALL, mass, weight)
    cu = batch.cu_seqlens
    assert np.all(weight[cu[0]:cu[1]] == 0)
    assert np.all(mass[cu[1]:cu[2]] == 0)


def test_stats_leave_attention_output_unchanged_and_are_reproducible():
    rng = np.random.default_rng(711)
    lays = [W.random_layout(rng, max_h=4, max_b=200, max_k=60, max_s=100, max_c=150) for _ in range(4)]
    batch = W.make_batch("stats-same", lays, 16, 4, 128, seed=712)
    db0 = H.device_batch(batch)
    assert db0.prefill() == sonic.OK
    torch.cuda.synchronize()
    plain = db0.out.cpu().numpy()
    db1, _, w1 = run_stats(batch)
    assert np.array_equal(db1.out.cpu().numpy(), plain)
    _, _, w2 = run_stats(batch, mass=False)
    assert np.array_equal(w1, w2)
    db3, m3, _ = run_stats(batch, weight=False)
    assert np.array_equal(db3.out.cpu().numpy(), plain)
    cu = batch.cu_seqlens
    for b, lay in enumerate(lays):   # the weights of a request sum to its current row count
        assert abs(float(w1[cu[b]:cu[b + 1]].astype(np.float64).sum()) - lay.current) <= 1e-3 * max(lay.current, 1)


def test_stats_workload_rows():
    """The 8B-shaped workload: A_nexus of sampled rows and w(x) of every key, two requests."""
    H.need_gpu()
    batch = W.workload(2, decode_steps=0)
    _, mass, weight = run_stats(batch)
    rng = np.random.default_rng(9)
    cu = batch.cu_seqlens
    for b in (0, 6):
        s, e = int(cu[b]), int(cu[b + 1])
        args = (batch.q[s:e], batch.k[s:e], batch.role[s:e], batch.turn_id[s:e])
        rows = np.unique(np.concatenate([rng.integers(0, e - s, 40), np.arange(e - s - 256, e - s, 17)]))
        close(mass[s + rows], OS.nexus_mass(*args, rows=rows), f"workload 2 A_nexus req {b}")
        close(weight[s:e], OS.key_weight(*args), f"workload 2 w(x) req {b}")
        assert np.all(weight[s:e][batch.role[s:e] == OL.HISTORY_TEXT] == 0)
