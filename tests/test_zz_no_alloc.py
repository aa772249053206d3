"""The decode entry point that allocates nothing, called through the C ABI, against the entry
point with a workspace: two calls in a row, the second with a smaller batch, each bit for bit
equal to the workspace entry point on an identical cache and within the attention bar of the
fp64 oracle."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import decode as OD
from paper_2601_21927_amd import sonic
from paper_2601_21927_amd.runner import bf16_to_device, bf16_to_host
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu


def _compacted_pair(batch, extra):
    """Two identical compacted caches of the batch (and the oracle's copy)."""
    caps = H.kept_counts(batch) + extra
    out = []
    for _ in range(2):
        db = H.device_batch(batch)
        cache = db.alloc_cache(caps)
        assert db.compact() == sonic.OK
        out.append((db, cache))
    torch.cuda.synchronize()
    for db, _ in out:
        assert db.read_status() == 0
    return out, H.oracle_compact(batch, caps)


def _one_call(batch):
    ((db1, c1), (db2, c2)), (kc, vc, _, n, off) = _compacted_pair(batch, 1)
    B, Hq, d = batch.batch, batch.num_q_heads, batch.head_dim
    max_ctx = int(c1.row_cap_host.max())
    q, kn, vn = (bf16_to_device(x[0]) for x in (batch.dec_q, batch.dec_k, batch.dec_v))
    o1 = torch.full((B, Hq, d), 7.0, dtype=torch.float32, device="cuda")
    o2 = torch.full((B, Hq, d), 9.0, dtype=torch.float32, device="cuda")
    assert c1.decode(q, kn, vn, o1, db1.status, max_ctx) == sonic.OK
    st = sonic.compressed_decode_noalloc(c2.k, c2.v, c2.row_off, c2.row_cap, c2.length, q, kn, vn, o2, db2.status,
                                         max_ctx)
    assert st == sonic.OK, sonic.status_string(st)
    torch.cuda.synchronize()
    assert db1.read_status() == 0 and db2.read_status() == 0
    assert torch.equal(o1, o2), "no-allocation decode differs from the workspace decode"
    assert torch.equal(c1.length, c2.length)
    assert np.array_equal(c2.length.cpu().numpy(), n + 1)
    assert np.array_equal(bf16_to_host(c1.k), bf16_to_host(c2.k))
    assert np.array_equal(bf16_to_host(c1.v), bf16_to_host(c2.v))
    got = o2.cpu().numpy()
    for b in range(B):
        o, ln = int(off[b]), int(n[b])
        want = OD.decode_step(batch.dec_q[0, b], kc[o:o + ln], vc[o:o + ln], batch.dec_k[0, b], batch.dec_v[0, b])
        H.assert_close(got[b], want, f"{batch.name} request {b} (no-allocation decode)")


def test_no_alloc_decode_matches_workspace_decode_two_calls():
    H.need_gpu()
    # first call: 6 requests with contexts long enough for several splits per pair
    lays_a = [W.RequestLayout(600 + 37 * i, [40, 30], [9, 5], 11 + i) for i in range(6)]
    big = W.make_batch("noalloc-big", lays_a, 8, 2, 128, seed=21, decode_steps=1)
    H.note("no-allocation decode, call 1: B=6, Hq/Hkv=8/2, d=128")
    _one_call(big)
    # second call, smaller: 2 requests, other head shape
    lays_b = [W.RequestLayout(300, [20], [6], 5), W.RequestLayout(9, [12], [3], 2)]
    small = W.make_batch("noalloc-small", lays_b, 4, 2, 64, seed=22, decode_steps=1)
    H.note("no-allocation decode, call 2: B=2, Hq/Hkv=4/2, d=64")
    _one_call(small)


def test_no_alloc_decode_rejects_more_than_its_scratch():
    H.need_gpu()
    B = 4097   # more requests than the fixed counter region holds
    q = torch.zeros((B, 1, 64), dtype=torch.bfloat16, device="cuda")
    kn = torch.zeros((B, 1, 64), dtype=torch.bfloat16, device="cuda")
    out = torch.full((B, 1, 64), 3.0, dtype=torch.float32, device="cuda")
    kc = torch.zeros((B + 1, 1, 64), dtype=torch.bfloat16, device="cuda")
    off = torch.arange(B, dtype=torch.int64, device="cuda")
    cap = torch.ones(B, dtype=torch.int32, device="cuda")
    ln = torch.zeros(B, dtype=torch.int32, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    st = sonic.compressed_decode_noalloc(kc, kc, off, cap, ln, q, kn, kn, out, status, 2)
    assert st == sonic.ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.all(out == 3.0) and torch.all(ln == 0) and int(status.item()) == 0
