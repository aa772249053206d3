"""Decode over the compacted cache on the GPU against the fp64 oracle."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import decode as OD
from paper_2601_21927_amd import sonic
from paper_2601_21927_amd.runner import bf16_to_device, bf16_to_host
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu


def compacted(batch, extra_rows):
    """Compact the batch on the GPU (its bit-exactness is tested elsewhere) and check it here too."""
    db = H.device_batch(batch)
    kept = H.kept_counts(batch)
    cache = db.alloc_cache(kept + extra_rows)
    assert db.compact() == sonic.OK
    torch.cuda.synchronize()
    assert db.read_status() == 0
    kc, vc, ki, n, off = H.oracle_compact(batch, kept + extra_rows)
    assert np.array_equal(cache.length.cpu().numpy(), n)
    return db, cache, (kc, vc, n, off)


def run_steps(batch, db, cache, steps, check_steps, row_role=None, oracle_ctx=None):
    """Run `steps` decode steps; compare the outputs of `check_steps` with the oracle.
    oracle_ctx(b, t) -> (k_ctx, v_ctx) bits for request b before step t."""
    B, Hq, d = batch.batch, batch.num_q_heads, batch.head_dim
    max_ctx = int(cache.row_cap_host.max())
    out = torch.empty((B, Hq, d), dtype=torch.float32, device="cuda")
    qs = bf16_to_device(batch.dec_q[:steps])
    ks = bf16_to_device(batch.dec_k[:steps])
    vs = bf16_to_device(batch.dec_v[:steps])
    errs = []
    for t in range(steps):
        st = cache.decode(qs[t], ks[t], vs[t], out, db.status, max_ctx, row_role=row_role)
        assert st == sonic.OK, sonic.status_string(st)
        if t in check_steps:
            torch.cuda.synchronize()
            assert db.read_status() == 0, sonic.status_string(db.read_status())
            got = out.cpu().numpy()
            for b in range(B):
                kc, vc = oracle_ctx(b, t)
                want = OD.decode_step(batch.dec_q[t, b], kc, vc, batch.dec_k[t, b], batch.dec_v[t, b])
                errs.append(np.abs(got[b] - want))
                H.assert_close(got[b], want, f"{batch.name} step {t} request {b}")
    torch.cuda.synchronize()
    return np.concatenate([e.ravel() for e in errs]) if errs else np.zeros(0)


def compact_ctx_fn(batch, ref):
    kc, vc, n, off = ref

    def ctx(b, t):
        base, ln = int(off[b]), int(n[b])
        k = np.concatenate([kc[base:base + ln], batch.dec_k[:t, b]])
        v = np.concatenate([vc[base:base + ln], batch.dec_v[:t, b]])
        return k, v
    return ctx


@pytest.mark.parametrize("Hq,Hkv,d", [(4, 2, 64), (32, 8, 128), (28, 4, 128), (8, 8, 128), (8, 1, 64)])
def test_decode_random_layouts(Hq, Hkv, d):
    H.need_gpu()
    rng = np.random.default_rng(200 + Hq + Hkv + d)
    lays = [W.random_layout(rng, max_h=4, max_b=400, max_k=150, max_s=300, max_c=200) for _ in range(5)]
    lays.append(W.RequestLayout(0, [], [], 1))     # a context of one row
    steps = 6
    batch = W.make_batch("rand", lays, Hq, Hkv, d, seed=int(rng.integers(1 << 30)), decode_steps=steps)
    db, cache, ref = compacted(batch, steps)
    run_steps(batch, db, cache, steps, set(range(steps)), oracle_ctx=compact_ctx_fn(batch, ref))
    # lengths advanced on the device and appended rows are in the cache, bit for bit
    kc, vc, n, off = ref
    assert np.array_equal(cache.length.cpu().numpy(), n + steps)
    k = bf16_to_host(cache.k)
    for b in range(batch.batch):
        base = int(off[b]) + int(n[b])
        assert np.array_equal(k[base:base + steps], batch.dec_k[:steps, b])


def test_masked_full_cache_decode_equals_compact():
    """Full-cache mode (history rows masked by role) against the oracle's masked decode."""
    H.need_gpu()
    rng = np.random.default_rng(77)
    lays = [W.random_layout(rng, max_h=4, max_b=300, max_k=100, max_s=200, max_c=100) for _ in range(4)]
    steps = 4
    batch = W.make_batch("full", lays, 32, 8, 128, seed=77, decode_steps=steps)
    db = H.device_batch(batch)
    # the full cache is the uncompacted augmented K/V, with room for the steps
    lens = np.array([l.length for l in lays], np.int64)
    cache = db.alloc_cache(lens + steps)
    kf = bf16_to_host(cache.k)
    vf = bf16_to_host(cache.v)
    roles = np.full(int((lens + steps).sum()), sonic.ROLE_CURRENT, np.uint8)
    for b in range(batch.batch):
        s, e = int(batch.cu_seqlens[b]), int(batch.cu_seqlens[b + 1])
        o = int(cache.row_off_host[b])
        kf[o:o + e - s] = batch.k[s:e]
        vf[o:o + e - s] = batch.v[s:e]
        roles[o:o + e - s] = batch.role[s:e]
    cache.k.copy_(bf16_to_device(kf))
    cache.v.copy_(bf16_to_device(vf))
    cache.length.copy_(torch.from_numpy(lens.astype(np.int32)))
    row_role = torch.from_numpy(roles).cuda()

    def ctx_masked(b, t):
        raise AssertionError("unused")

    B, Hq, d = batch.batch, batch.num_q_heads, batch.head_dim
    out = torch.empty((B, Hq, d), dtype=torch.float32, device="cuda")
    max_ctx = int(cache.row_cap_host.max())
    for t in range(steps):
        st = cache.decode(bf16_to_device(batch.dec_q[t]), bf16_to_device(batch.dec_k[t]),
                          bf16_to_device(batch.dec_v[t]), out, db.status, max_ctx, row_role=row_role)
        assert st == sonic.OK
        torch.cuda.synchronize()
        assert db.read_status() == 0
        got = out.cpu().numpy()
        for b in range(B):
            s, e = int(batch.cu_seqlens[b]), int(batch.cu_seqlens[b + 1])
            kfull = np.concatenate([batch.k[s:e], batch.dec_k[:t, b]])
            vfull = np.concatenate([batch.v[s:e], batch.dec_v[:t, b]])
            rfull = np.concatenate([batch.role[s:e], np.full(t, sonic.ROLE_CURRENT, np.uint8)])
            want = OD.masked_decode_step(batch.dec_q[t, b], kfull, vfull, rfull, batch.dec_k[t, b],
                                         batch.dec_v[t, b])
            H.assert_close(got[b], want, f"masked full decode step {t} request {b}")


@pytest.mark.parametrize("idx,check", [(1, None), (2, (0, 1, 100, 255)), (3, (0, 255)), (4, (0, 511)),
                                       (5, (0, 1, 1023))])
def test_decode_workloads(idx, check):
    H.need_gpu()
    batch = W.workload(idx)
    steps = batch.decode_steps
    check = set(range(steps)) if check is None else set(check)
    H.note(f"decode workload {idx}: B={batch.batch} steps={steps}")
    db, cache, ref = compacted(batch, steps)
    errs = run_steps(batch, db, cache, steps, check, oracle_ctx=compact_ctx_fn(batch, ref))
    H.note(f"  workload {idx} decode overall: max_abs={errs.max():.3e} mean_abs={errs.mean():.3e}")
    kc, vc, n, off = ref
    assert np.array_equal(cache.length.cpu().numpy(), n + steps)


def test_decode_capacity_overflow():
    """A request whose append would overflow is left unchanged; the others proceed."""
    H.need_gpu()
    lays = [W.RequestLayout(4, [10], [3], 2), W.RequestLayout(2, [5], [1], 1)]
    batch = W.make_batch("cap", lays, 4, 2, 64, seed=3, decode_steps=3)
    db, cache, ref = compacted(batch, np.array([1, 3]))
    kc, vc, n, off = ref
    out = torch.full((2, 4, 64), 5.0, dtype=torch.float32, device="cuda")
    max_ctx = int(cache.row_cap_host.max())
    q, kn, vn = (bf16_to_device(x) for x in (batch.dec_q, batch.dec_k, batch.dec_v))
    assert cache.decode(q[0], kn[0], vn[0], out, db.status, max_ctx) == sonic.OK
    torch.cuda.synchronize()
    assert db.read_status() == 0
    assert np.array_equal(cache.length.cpu().numpy(), n + 1)
    out.fill_(5.0)
    assert cache.decode(q[1], kn[1], vn[1], out, db.status, max_ctx) == sonic.OK   # request 0 is full now
    torch.cuda.synchronize()
    assert db.read_status() == sonic.ERR_CAPACITY
    assert np.array_equal(cache.length.cpu().numpy(), n + np.array([1, 2]))
    got = out.cpu().numpy()
    assert np.all(got[0] == 5.0)
    o, ln = int(off[1]), int(n[1])
    want = OD.decode_step(batch.dec_q[1, 1], np.concatenate([kc[o:o + ln], batch.dec_k[:1, 1]]),
                          np.concatenate([vc[o:o + ln], batch.dec_v[:1, 1]]), batch.dec_k[1, 1], batch.dec_v[1, 1])
    H.assert_close(got[1], want, "request 1 after request 0 overflowed")


def test_decode_honours_pending_layout_error():
    """A layout error left by an earlier call stops decode (no append, no output, no length change);
    a pending capacity error does not (capacity is per request); afterwards decode still matches the
    oracle, so the split counters were left consistent."""
    H.need_gpu()
    # long enough contexts for several splits per (request, kv-head) pair
    lays = [W.RequestLayout(700, [30], [12], 9), W.RequestLayout(650, [20], [4], 3)]
    steps = 2
    batch = W.make_batch("pending", lays, 8, 2, 128, seed=4, decode_steps=steps)
    db, cache, ref = compacted(batch, steps)
    kc, vc, n, off = ref
    max_ctx = int(cache.row_cap_host.max())
    out = torch.full((2, 8, 128), 5.0, dtype=torch.float32, device="cuda")
    q, kn, vn = (bf16_to_device(x) for x in (batch.dec_q, batch.dec_k, batch.dec_v))
    k_before, v_before = bf16_to_host(cache.k).copy(), bf16_to_host(cache.v).copy()
    db.status.fill_(sonic.ERR_BAD_LAYOUT)
    assert cache.decode(q[0], kn[0], vn[0], out, db.status, max_ctx) == sonic.OK
    torch.cuda.synchronize()
    assert db.read_status() == sonic.ERR_BAD_LAYOUT
    assert np.array_equal(cache.length.cpu().numpy(), n)
    assert torch.all(out == 5.0)
    assert np.array_equal(bf16_to_host(cache.k), k_before) and np.array_equal(bf16_to_host(cache.v), v_before)
    ctx = compact_ctx_fn(batch, ref)
    db.status.fill_(sonic.ERR_CAPACITY)
    for t in range(steps):
        assert cache.decode(q[t], kn[t], vn[t], out, db.status, max_ctx) == sonic.OK
        torch.cuda.synchronize()
        assert db.read_status() == (sonic.ERR_CAPACITY if t == 0 else 0)
        got = out.cpu().numpy()
        for b in range(2):
            kk, vv = ctx(b, t)
            want = OD.decode_step(batch.dec_q[t, b], kk, vv, batch.dec_k[t, b], batch.dec_v[t, b])
            H.assert_close(got[b], want, f"step {t} request {b} after a pending status")
        db.clear_status()
    assert np.array_equal(cache.length.cpu().numpy(), n + steps)


def test_decode_default_scale_is_one_over_sqrt_d():
    """softmax_scale = 0 (the binding's default) gives bit for bit the output of an explicit 1/sqrt(d)."""
    H.need_gpu()
    lays = [W.RequestLayout(40, [30], [12], 9), W.RequestLayout(3, [20], [4], 3)]
    batch = W.make_batch("scale", lays, 8, 2, 64, seed=5, decode_steps=1)
    outs = []
    for scale in (None, 1.0 / np.sqrt(64.0)):
        db, cache, ref = compacted(batch, 1)
        out = torch.empty((2, 8, 64), dtype=torch.float32, device="cuda")
        st = sonic.compressed_decode(cache.k, cache.v, cache.row_off, cache.row_cap, cache.length,
                                     bf16_to_device(batch.dec_q[0]), bf16_to_device(batch.dec_k[0]),
                                     bf16_to_device(batch.dec_v[0]), out,
                                     torch.zeros(sonic.decode_workspace_bytes(2, 8, 64, 64), dtype=torch.uint8,
                                                 device="cuda"), db.status, 64, softmax_scale=scale)
        assert st == sonic.OK
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])
