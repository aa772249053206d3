"""Masked prefill on the GPU against the fp64 oracle (max-abs <= 1e-2, mean-abs <= 1e-3)."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import mask as OM
from paper_2601_21927_amd import sonic
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu


def run_prefill(batch, nexus_scope=sonic.NEXUS_ALL):
    H.need_gpu()
    db = H.device_batch(batch)
    db.out.fill_(float("nan"))
    st = db.prefill(nexus_scope=nexus_scope)
    assert st == sonic.OK, sonic.status_string(st)
    torch.cuda.synchronize()
    assert db.read_status() == 0, sonic.status_string(db.read_status())
    return db


def check_all_rows(batch, db, nexus_scope=OM.NEXUS_ALL):
    out = db.out.cpu().numpy()
    cu = batch.cu_seqlens
    for b, lay in enumerate(batch.layouts):
        s, e = int(cu[b]), int(cu[b + 1])
        if e == s:
            continue
        want = H.oracle_prefill_rows(batch, [np.arange(e - s) if i == b else np.zeros(0, np.int64)
                                             for i in range(batch.batch)], nexus_scope)[b]
        H.assert_close(out[s:e], want, f"{batch.name} request {b} (L={e - s})")


SMALL_SHAPES = [(4, 2, 64), (8, 2, 128), (7, 1, 128), (2, 2, 128), (8, 1, 64), (32, 8, 128), (6, 2, 64)]


@pytest.mark.parametrize("Hq,Hkv,d", SMALL_SHAPES)
def test_prefill_random_layouts_all_rows(Hq, Hkv, d):
    rng = np.random.default_rng(100 + Hq * 7 + Hkv + d)
    lays = [W.random_layout(rng, max_h=4, max_b=90, max_k=45, max_s=70, max_c=70) for _ in range(3)]
    H.note(f"prefill random layouts Hq={Hq} Hkv={Hkv} d={d}: {[l.length for l in lays]}")
    batch = W.make_batch("random", lays, Hq, Hkv, d, seed=int(rng.integers(1 << 30)))
    db = run_prefill(batch)
    check_all_rows(batch, db)


EDGE_LAYOUTS = {
    "single_token": [W.RequestLayout(1, [], [], 0)],
    "only_current": [W.RequestLayout(0, [], [], 45)],
    "no_system": [W.RequestLayout(0, [33, 40], [5, 31], 9)],
    "zero_nexus": [W.RequestLayout(10, [20, 20, 20], [0, 0, 0], 5)],
    "no_current": [W.RequestLayout(12, [70], [33], 0)],
    "empty_request_in_batch": [W.RequestLayout(5, [9], [3], 4), W.RequestLayout(0, [], [], 0),
                               W.RequestLayout(3, [2], [1], 1)],
    "long_system_only": [W.RequestLayout(300, [], [], 0)],
    "nexus_exact_tiles": [W.RequestLayout(32, [64, 32], [32, 64], 32)],
    "many_tiny_segments": [W.RequestLayout(2, [1] * 40, [1, 0] * 20, 3)],
}


@pytest.mark.parametrize("name", sorted(EDGE_LAYOUTS))
def test_prefill_edge_layouts(name):
    lays = EDGE_LAYOUTS[name]
    H.note(f"prefill edge layout {name}")
    batch = W.make_batch(name, lays, 8, 2, 128, seed=7)
    db = run_prefill(batch)
    check_all_rows(batch, db)


@pytest.mark.parametrize("Hq,Hkv,d", [(4, 2, 64), (32, 8, 128), (7, 1, 128)])
def test_prefill_up_to_own_scope_random_layouts_all_rows(Hq, Hkv, d):
    """Nexus rows see the Nexus tokens of their own and earlier segments only."""
    rng = np.random.default_rng(500 + Hq * 7 + Hkv + d)
    lays = [W.random_layout(rng, max_h=5, max_b=90, max_k=45, max_s=70, max_c=70) for _ in range(3)]
    lays.append(W.RequestLayout(3, [40, 2, 33], [33, 1, 64], 5))
    H.note(f"prefill up-to-own scope Hq={Hq} Hkv={Hkv} d={d}: {[l.length for l in lays]}")
    batch = W.make_batch("scope", lays, Hq, Hkv, d, seed=int(rng.integers(1 << 30)))
    db = run_prefill(batch, sonic.NEXUS_UP_TO_OWN)
    check_all_rows(batch, db, OM.NEXUS_UP_TO_OWN)


def test_prefill_up_to_own_scope_workload_rows():
    """The 8B-shaped workload: every Nexus row of segments 1, 4 and 8 and sampled other rows."""
    H.need_gpu()
    batch = W.workload(2, decode_steps=0)
    db = run_prefill(batch, sonic.NEXUS_UP_TO_OWN)
    out = db.out.cpu().numpy()
    rng = np.random.default_rng(5)
    lay = batch.layouts[0]
    nexus_rows = []
    p = lay.system
    for i, (bl, k) in enumerate(zip(lay.bodies, lay.nexus)):
        if i in (0, 3, 7):
            nexus_rows.append(np.arange(p + bl, p + bl + k))
        p += bl + k
    rows = [np.unique(np.concatenate(nexus_rows + [rng.integers(0, lay.length, 24)])) if b in (0, 5) else
            np.zeros(0, np.int64) for b in range(batch.batch)]
    want = H.oracle_prefill_rows(batch, rows, OM.NEXUS_UP_TO_OWN)
    for b in (0, 5):
        s = int(batch.cu_seqlens[b])
        H.assert_close(out[s + rows[b]], want[b], f"workload 2 up-to-own request {b}")


def test_prefill_unknown_scope_is_rejected():
    H.need_gpu()
    batch = W.make_batch("scope-arg", [W.RequestLayout(3, [5], [2], 2)], 4, 2, 64, seed=1)
    db = H.device_batch(batch)
    assert db.prefill(nexus_scope=2) == sonic.ERR_INVALID_ARG


@pytest.mark.parametrize("scope", [OM.NEXUS_ALL, OM.NEXUS_UP_TO_OWN])
def test_prefill_mask_revealed_by_one_hot_values(scope):
    """Q = 0 and V[q] = e_q make output row p equal 1/|vis(p)| on exactly the visible keys."""
    H.need_gpu()
    lays = [W.RequestLayout(5, [20, 17, 9], [7, 0, 12], 17), W.RequestLayout(0, [40], [3], 30)]
    d = 128
    batch = W.make_batch("onehot", lays, 4, 2, d, seed=3)
    T = batch.total_tokens
    batch.q = np.zeros_like(batch.q)
    v = np.zeros((T, 2, d), np.uint16)
    for b, lay in enumerate(lays):
        s = int(batch.cu_seqlens[b])
        for i in range(lay.length):
            v[s + i, :, i] = 0x3F80   # 1.0
    batch.v = v
    db = run_prefill(batch, sonic.NEXUS_ALL if scope == OM.NEXUS_ALL else sonic.NEXUS_UP_TO_OWN)
    out = db.out.cpu().numpy()
    for b, lay in enumerate(lays):
        s, e = int(batch.cu_seqlens[b]), int(batch.cu_seqlens[b + 1])
        role, turn = lay.roles_and_turns()
        vis = OM.visibility(role, turn, scope)
        L = e - s
        for p in range(L):
            n = int(vis[p].sum())
            want = np.where(vis[p], np.float32(1.0) / np.float32(n), 0.0).astype(np.float32)
            for h in range(4):
                got = out[s + p, h, :L]
                assert np.array_equal(got != 0, vis[p]), (b, p, h)
                assert np.allclose(got, want, rtol=1e-6, atol=0), (b, p, h)
            assert np.all(out[s + p, :, L:] == 0)


def test_prefill_bad_layout_reports_and_leaves_output():
    H.need_gpu()
    lay = W.RequestLayout(3, [5], [2], 2)
    batch = W.make_batch("bad", [lay], 4, 2, 64, seed=1)
    batch.role = batch.role.copy()
    batch.role[1] = sonic.ROLE_NEXUS     # a Nexus token inside the system prompt
    db = H.device_batch(batch)
    db.out.fill_(7.0)
    assert db.prefill() == sonic.OK
    torch.cuda.synchronize()
    assert db.read_status() == sonic.ERR_BAD_LAYOUT
    assert torch.all(db.out == 7.0)


def test_prefill_argument_errors():
    H.need_gpu()
    batch = W.make_batch("args", [W.RequestLayout(2, [3], [1], 2)], 4, 2, 64, seed=1)
    db = H.device_batch(batch)
    small_ws = db.prefill_ws[:16]
    st = sonic.segment_attn_prefill(db.cu, db.role, db.turn_id, db.q, db.k, db.v, db.out, small_ws, db.status)
    assert st == sonic.ERR_WORKSPACE
    q96 = torch.zeros((db.T, 4, 96), dtype=torch.bfloat16, device="cuda")
    k96 = torch.zeros((db.T, 2, 96), dtype=torch.bfloat16, device="cuda")
    st = sonic.segment_attn_prefill(db.cu, db.role, db.turn_id, q96, k96, k96, db.out, db.prefill_ws, db.status)
    assert st == sonic.ERR_UNSUPPORTED


# Rows checked per workload: the tiny one in full; for the long ones, the deterministic subset
# (every system, Nexus and current row, +-64 rows around every run boundary, every 16th body
# row, the last row of every 32-row block) of the requests listed here, and sampled rows
# (every run edge and block edge, the last row of every block, random rows) of every other one.
SUBSET_REQUESTS = {2: (0,), 3: (), 4: (0,)}


@pytest.mark.parametrize("idx", [1, 2, 3, 4])
def test_prefill_workloads(idx):
    from tests import oracle_pool as P
    H.need_gpu()
    batch = W.workload(idx, decode_steps=0)
    H.note(f"prefill workload {idx}: B={batch.batch} T={batch.total_tokens} Hq={batch.num_q_heads} "
           f"Hkv={batch.num_kv_heads} d={batch.head_dim}")
    db = run_prefill(batch)
    out = db.out
    assert torch.isfinite(out).all()
    if idx == 1:
        check_all_rows(batch, db)
        return
    rng = np.random.default_rng(idx)
    rows = {b: (H.subset_rows(lay) if b in SUBSET_REQUESTS[idx] else H.sample_rows(lay, rng))
            for b, lay in enumerate(batch.layouts)}
    got = {}
    for b, r in rows.items():
        s = int(batch.cu_seqlens[b])
        got[b] = out.index_select(0, torch.from_numpy(s + r).to(out.device)).cpu().numpy()
    del db, out
    torch.cuda.synchronize()
    H.note(f"  oracle rows per request: {[len(r) for r in rows.values()]} "
           f"(subset for requests {list(SUBSET_REQUESTS[idx])}), {sum(len(r) for r in rows.values())} in all")
    want = P.workload_rows(idx, rows)
    for b in rows:
        H.assert_close(got[b], want[b], f"workload {idx} request {b} ({len(rows[b])} rows)")
    H.assert_close(np.concatenate([got[b] for b in rows]), np.concatenate([want[b] for b in rows]),
                   f"workload {idx}: all checked rows")


def test_prefill_default_scale_is_one_over_sqrt_d():
    """softmax_scale = 0 (the binding's default) gives bit for bit the output of an explicit 1/sqrt(d)."""
    H.need_gpu()
    batch = W.make_batch("scale", [W.RequestLayout(20, [70, 33], [9, 4], 40)], 8, 2, 128, seed=2)
    outs = []
    for scale in (None, 1.0 / np.sqrt(128.0)):
        db = H.device_batch(batch)
        st = sonic.segment_attn_prefill(db.cu, db.role, db.turn_id, db.q, db.k, db.v, db.out, db.prefill_ws,
                                        db.status, softmax_scale=scale)
        assert st == sonic.OK
        torch.cuda.synchronize()
        assert db.read_status() == 0
        outs.append(db.out.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])
