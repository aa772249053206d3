"""Next-turn Nexus step on the GPU against the fp64 oracle.

A batch of conversations ends with a history segment and no current query.  The
compact cache holds, per request, the system prompt, the earlier segments' Nexus
tokens and the last segment's body (the turn that just ended); the new rows are
the last segment's Nexus tokens.  The GPU output must match oracle.extend to the
attention tolerance, and the new cache (the earlier rows plus the new Nexus K/V)
must match bit for bit.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import extend as OE
from paper_2601_21927_amd import sonic
from paper_2601_21927_amd.runner import bf16_to_device, bf16_to_host
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu


class ExtendCase:
    """Device buffers of one next-turn step for a batch whose layouts end with a segment."""

    def __init__(self, batch: W.Batch, extra_cap=0, keep_delta=None):
        self.batch = batch
        B, Hkv, d = batch.batch, batch.num_kv_heads, batch.head_dim
        cu = batch.cu_seqlens
        self.cache_pos, self.keep, self.nexus_pos = [], [], []
        for b, lay in enumerate(batch.layouts):
            cp, keep, npos = W.extend_positions(lay)
            self.cache_pos.append(cp + int(cu[b]))
            self.keep.append(keep)
            self.nexus_pos.append(npos + int(cu[b]))
        self.len0 = np.array([len(c) for c in self.cache_pos], np.int64)
        self.kn = np.array([len(n) for n in self.nexus_pos], np.int64)
        self.cap = np.maximum(self.len0, np.array(self.keep) + self.kn) + extra_cap
        self.off = np.concatenate([[0], np.cumsum(self.cap)[:-1]]).astype(np.int64)
        rows = int(self.cap.sum())
        kc = np.full((rows, Hkv, d), 0x7FC1, np.uint16)
        vc = kc.copy()
        for b in range(B):
            o, n = int(self.off[b]), int(self.len0[b])
            kc[o:o + n] = batch.k[self.cache_pos[b]]
            vc[o:o + n] = batch.v[self.cache_pos[b]]
        self.kc_host, self.vc_host = kc, vc
        self.kc, self.vc = bf16_to_device(kc), bf16_to_device(vc)
        self.row_off = torch.from_numpy(self.off).cuda()
        self.row_cap = torch.from_numpy(self.cap.astype(np.int32)).cuda()
        self.length = torch.from_numpy(self.len0.astype(np.int32)).cuda()
        keep = np.array(self.keep, np.int32) + (0 if keep_delta is None else np.asarray(keep_delta))
        self.keep_len = torch.from_numpy(keep.astype(np.int32)).cuda()
        allpos = np.concatenate(self.nexus_pos) if B else np.zeros(0, np.int64)
        self.nexus_cu = torch.from_numpy(np.concatenate([[0], np.cumsum(self.kn)]).astype(np.int32)).cuda()
        self.q = bf16_to_device(batch.q[allpos])
        self.k = bf16_to_device(batch.k[allpos])
        self.v = bf16_to_device(batch.v[allpos])
        self.out = torch.full((len(allpos), batch.num_q_heads, d), 7.0, dtype=torch.float32, device="cuda")
        self.ws = torch.empty(max(sonic.nexus_extend_workspace_bytes(B, len(allpos), int(self.cap.max()), Hkv, d),
                                  256), dtype=torch.uint8, device="cuda")
        self.status = torch.zeros(1, dtype=torch.int32, device="cuda")

    def run(self):
        st = sonic.nexus_extend(self.nexus_cu, self.keep_len, self.kc, self.vc, self.row_off, self.row_cap,
                                self.length, self.q, self.k, self.v, self.out, self.ws, self.status,
                                max_rows=int(self.cap.max()))
        torch.cuda.synchronize()
        return st

    def oracle(self, b):
        bt = self.batch
        npos, cpos = self.nexus_pos[b], self.cache_pos[b]
        return OE.extend_request(bt.q[npos], bt.k[npos], bt.v[npos], bt.k[cpos], bt.v[cpos], self.keep[b])


def check_case(case: ExtendCase, label):
    assert case.run() == sonic.OK
    assert int(case.status.item()) == 0, sonic.status_string(int(case.status.item()))
    got = case.out.cpu().numpy()
    kc, vc = bf16_to_host(case.kc), bf16_to_host(case.vc)
    lens = case.length.cpu().numpy()
    cu = case.nexus_cu.cpu().numpy()
    for b in range(case.batch.batch):
        want, nk, nv = case.oracle(b)
        if len(want):
            H.assert_close(got[cu[b]:cu[b + 1]], want, f"{label} request {b}")
        o = int(case.off[b])
        assert lens[b] == len(nk), f"{label} request {b}: length {lens[b]} != {len(nk)}"
        assert np.array_equal(kc[o:o + len(nk)], nk), f"{label} request {b}: K cache rows differ"
        assert np.array_equal(vc[o:o + len(nv)], nv), f"{label} request {b}: V cache rows differ"
        # rows past the old end and the capacity were not touched
        end = max(len(nk), int(case.len0[b]))
        assert np.array_equal(kc[o + end:o + int(case.cap[b])], case.kc_host[o + end:o + int(case.cap[b])])


def _ending_layouts(rng, n, **kw):
    out = []
    while len(out) < n:
        lay = W.random_layout(rng, max_c=0, **kw)
        if lay.bodies:
            out.append(lay)
    return out


@pytest.mark.parametrize("Hq,Hkv,d", [(4, 2, 64), (32, 8, 128), (28, 4, 128), (8, 1, 64), (6, 2, 128),
                                      (2, 2, 128), (3, 1, 64)])
def test_extend_random(Hq, Hkv, d):
    H.need_gpu()
    rng = np.random.default_rng(300 + Hq + Hkv + d)
    lays = _ending_layouts(rng, 6, max_h=4, max_b=300, max_k=120, max_s=200)
    batch = W.make_batch("ext", lays, Hq, Hkv, d, seed=int(rng.integers(1 << 30)))
    check_case(ExtendCase(batch), f"random {Hq}/{Hkv}/{d}")


def test_extend_edges():
    """No new Nexus rows (the body is only dropped), a one-row body, more Nexus rows than body
    rows, an empty system prompt, and a single segment."""
    H.need_gpu()
    lays = [W.RequestLayout(5, [7, 4], [3, 0], 0), W.RequestLayout(3, [1], [1], 0),
            W.RequestLayout(2, [6, 2], [4, 40], 0), W.RequestLayout(0, [33, 65], [31, 33], 0),
            W.RequestLayout(64, [96], [65], 0)]
    batch = W.make_batch("ext-edge", lays, 8, 2, 128, seed=5)
    check_case(ExtendCase(batch, extra_cap=3), "edges")


def test_extend_matches_gpu_prefill_rows():
    """The step's output equals the full prefill's rows of the same Nexus tokens, both on the GPU."""
    H.need_gpu()
    rng = np.random.default_rng(77)
    lays = _ending_layouts(rng, 4, max_h=3, max_b=200, max_k=80, max_s=100)
    batch = W.make_batch("ext-vs-prefill", lays, 16, 4, 128, seed=78)
    db = H.device_batch(batch)
    assert db.prefill() == sonic.OK
    torch.cuda.synchronize()
    full = db.out.cpu().numpy()
    case = ExtendCase(batch)
    assert case.run() == sonic.OK
    got = case.out.cpu().numpy()
    allpos = np.concatenate(case.nexus_pos)
    diff = np.abs(got - full[allpos])
    H.note(f"  extend vs prefill on the GPU: max_abs={diff.max():.3e}")
    assert diff.max() <= 2 * H.MAX_ABS


@pytest.mark.parametrize("idx", [2, 4])
def test_extend_workload_shapes(idx):
    """The last turn of the 8B-shaped and long-dialogue workloads (no current query)."""
    H.need_gpu()
    st = W.workload_structure(idx)
    # earlier bodies are gone from the cache, so one row each keeps the draw small
    lays = [W.RequestLayout(l.system, [1] * (len(l.bodies) - 1) + l.bodies[-1:], l.nexus, 0)
            for l in st["layouts"]]
    batch = W.make_batch(f"ext-w{idx}", lays, st["Hq"], st["Hkv"], st["d"], seed=400 + idx)
    case = ExtendCase(batch)
    assert case.run() == sonic.OK
    assert int(case.status.item()) == 0
    got = case.out.cpu().numpy()
    cu = case.nexus_cu.cpu().numpy()
    rng = np.random.default_rng(idx)
    for b in range(batch.batch):
        want, nk, _ = case.oracle(b)
        rows = np.unique(np.concatenate([[0, len(want) - 1], rng.integers(0, len(want), 8)]))
        H.assert_close(got[cu[b] + rows], want[rows], f"workload {idx} request {b}")
    lens = case.length.cpu().numpy()
    assert np.array_equal(lens, np.array(case.keep) + case.kn)


def test_extend_capacity_and_bad_lengths():
    """Capacity overflow, keep_len > cache_len and cache_len > max_rows are reported on the
    device, and then nothing is written: not the output, the cache rows or the lengths."""
    H.need_gpu()
    # request 0: cache 4 + 3 + 6 = 13 rows, keeps 7, adds 9; request 1: cache 2 + 5 = 7 rows
    lays = [W.RequestLayout(4, [10, 6], [3, 9], 0), W.RequestLayout(2, [5], [2], 0)]
    batch = W.make_batch("ext-err", lays, 4, 2, 64, seed=9)
    for what in ("capacity", "keep", "max_rows"):
        case = ExtendCase(batch, keep_delta=np.array([0, 6 if what == "keep" else 0]))
        max_rows = int(case.cap.max())
        code = sonic.ERR_BAD_LAYOUT
        if what == "capacity":      # 15 rows: holds the 13 of now, not the 7 + 9 of afterwards
            case.cap[0] = 15
            case.row_cap.copy_(torch.from_numpy(case.cap.astype(np.int32)))
            code = sonic.ERR_CAPACITY
        elif what == "max_rows":
            max_rows = int(case.len0.max()) - 1
        before_k = bf16_to_host(case.kc).copy()
        st = sonic.nexus_extend(case.nexus_cu, case.keep_len, case.kc, case.vc, case.row_off, case.row_cap,
                                case.length, case.q, case.k, case.v, case.out, case.ws, case.status,
                                max_rows=max_rows)
        torch.cuda.synchronize()
        assert st == sonic.OK, what
        assert int(case.status.item()) == code, f"{what}: {sonic.status_string(int(case.status.item()))}"
        assert np.all(case.out.cpu().numpy() == 7.0), what
        assert np.array_equal(bf16_to_host(case.kc), before_k), what
        assert np.array_equal(case.length.cpu().numpy(), case.len0), what


def test_extend_argument_errors():
    H.need_gpu()
    lays = [W.RequestLayout(4, [10], [3], 0)]
    batch = W.make_batch("ext-args", lays, 4, 2, 64, seed=1)
    case = ExtendCase(batch)
    small = torch.empty(8, dtype=torch.uint8, device="cuda")
    st = sonic.nexus_extend(case.nexus_cu, case.keep_len, case.kc, case.vc, case.row_off, case.row_cap, case.length,
                            case.q, case.k, case.v, case.out, small, case.status, max_rows=int(case.cap.max()))
    assert st == sonic.ERR_WORKSPACE
    st = sonic.nexus_extend(case.nexus_cu, case.keep_len, case.kc, case.vc, case.row_off, case.row_cap, case.length,
                            case.q, case.k, case.v, case.out, case.ws, case.status, max_rows=int(case.cap.max()),
                            softmax_scale=-1.0)
    assert st == sonic.ERR_INVALID_ARG
    with pytest.raises(TypeError):
        sonic.nexus_extend(case.nexus_cu, case.keep_len.long(), case.kc, case.vc, case.row_off, case.row_cap,
                           case.length, case.q, case.k, case.v, case.out, case.ws, case.status,
                           max_rows=int(case.cap.max()))


def test_extend_many_new_rows():
    """Enough new rows that the work items outnumber twice the CUs (one wave group per
    item, no key split), with ragged blocks: 4 requests, 2,396 new Nexus rows."""
    H.need_gpu()
    lays = [W.RequestLayout(40, [100, 700], [20, 600], 0), W.RequestLayout(3, [650], [599], 0),
            W.RequestLayout(17, [30, 612], [5, 598], 0), W.RequestLayout(0, [720], [599], 0)]
    batch = W.make_batch("ext-many", lays, 32, 8, 128, seed=21)
    check_case(ExtendCase(batch), "many rows")


def _turn_layouts(rng, n, **kw):
    out = []
    while len(out) < n:
        lay = W.random_layout(rng, max_c=0, **kw)
        if len(lay.bodies) >= 2:
            out.append(lay)
    return out


@pytest.mark.parametrize("Hq,Hkv,d", [(4, 2, 64), (28, 4, 128), (32, 8, 128)])
def test_extend_two_segment_turn(Hq, Hkv, d):
    """A turn of two segments (utterance, response), one call each with the utterance's body
    length first: outputs against the oracle's two steps, cache rows and lengths bit for bit
    after each call."""
    H.need_gpu()
    rng = np.random.default_rng(700 + Hq + Hkv + d)
    lays = _turn_layouts(rng, 4, max_h=5, max_b=150, max_k=60, max_s=80)
    lays.append(W.RequestLayout(9, [40, 3, 70], [5, 20, 0], 0))    # more Nexus rows than utterance rows
    batch = W.make_batch("turn", lays, Hq, Hkv, d, seed=int(rng.integers(1 << 30)))
    B, cu = batch.batch, batch.cu_seqlens
    pos = [W.turn_positions(l) for l in lays]
    len0 = np.array([len(p[0]) for p in pos], np.int64)
    ku = np.array([len(p[3]) for p in pos], np.int64)
    kr = np.array([len(p[4]) for p in pos], np.int64)
    keep = np.array([p[1] for p in pos], np.int64)
    rb = len0 - keep - np.array([p[2] for p in pos])
    cap = np.maximum(np.maximum(len0, keep + ku + rb), keep + ku + kr) + 3
    off = np.concatenate([[0], np.cumsum(cap)[:-1]]).astype(np.int64)
    kc = np.full((int(cap.sum()), Hkv, d), 0x7FC1, np.uint16)
    vc = kc.copy()
    for b in range(B):
        o = int(off[b])
        kc[o:o + len0[b]] = batch.k[pos[b][0] + int(cu[b])]
        vc[o:o + len0[b]] = batch.v[pos[b][0] + int(cu[b])]
    dkc, dvc = bf16_to_device(kc), bf16_to_device(vc)
    row_off = torch.from_numpy(off).cuda()
    row_cap = torch.from_numpy(cap.astype(np.int32)).cuda()
    length = torch.from_numpy(len0.astype(np.int32)).cuda()
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    max_rows = int(cap.max())
    # oracle state per request: the cache rows as bf16 bits
    ok = [kc[int(off[b]):int(off[b]) + len0[b]].copy() for b in range(B)]
    ov = [vc[int(off[b]):int(off[b]) + len0[b]].copy() for b in range(B)]
    for step, (kn, sel, body) in enumerate(((ku, 3, np.array([p[2] for p in pos])), (kr, 4, None))):
        kp = keep if step == 0 else keep + ku
        rows = [pos[b][sel] + int(cu[b]) for b in range(B)]
        allpos = np.concatenate(rows)
        ncu = torch.from_numpy(np.concatenate([[0], np.cumsum(kn)]).astype(np.int32)).cuda()
        out = torch.full((len(allpos), Hq, d), 7.0, dtype=torch.float32, device="cuda")
        ws = torch.empty(sonic.nexus_extend_workspace_bytes(B, len(allpos), max_rows, Hkv, d), dtype=torch.uint8,
                         device="cuda")
        bl = None if body is None else torch.from_numpy(body.astype(np.int32)).cuda()
        st = sonic.nexus_extend(ncu, torch.from_numpy(kp.astype(np.int32)).cuda(), dkc, dvc, row_off, row_cap, length,
                                bf16_to_device(batch.q[allpos]), bf16_to_device(batch.k[allpos]),
                                bf16_to_device(batch.v[allpos]), out, ws, status, max_rows=max_rows, body_len=bl)
        assert st == sonic.OK
        torch.cuda.synchronize()
        assert int(status.item()) == 0, sonic.status_string(int(status.item()))
        got = out.cpu().numpy()
        gk, gv, gl = bf16_to_host(dkc), bf16_to_host(dvc), length.cpu().numpy()
        c = np.concatenate([[0], np.cumsum(kn)])
        for b in range(B):
            r = rows[b]
            want, ok[b], ov[b] = OE.extend_request(batch.q[r], batch.k[r], batch.v[r], ok[b], ov[b], int(kp[b]),
                                                   body_len=None if body is None else int(body[b]))
            if len(want):
                H.assert_close(got[c[b]:c[b + 1]], want, f"turn step {step} request {b}")
            o = int(off[b])
            assert gl[b] == len(ok[b]), (step, b, gl[b], len(ok[b]))
            assert np.array_equal(gk[o:o + len(ok[b])], ok[b]) and np.array_equal(gv[o:o + len(ov[b])], ov[b]), \
                (step, b)


def test_extend_body_longer_than_the_tail_is_a_layout_error():
    H.need_gpu()
    rng = np.random.default_rng(41)
    lays = _ending_layouts(rng, 2, max_h=3, max_b=40, max_k=12, max_s=20)
    batch = W.make_batch("bodylen", lays, 4, 2, 64, seed=41)
    case = ExtendCase(batch)
    tail = case.len0 - np.array(case.keep)
    bl = torch.from_numpy((tail + np.array([0, 1])).astype(np.int32)).cuda()
    kc0, len0 = bf16_to_host(case.kc).copy(), case.length.cpu().numpy().copy()
    st = sonic.nexus_extend(case.nexus_cu, case.keep_len, case.kc, case.vc, case.row_off, case.row_cap, case.length,
                            case.q, case.k, case.v, case.out, case.ws, case.status, max_rows=int(case.cap.max()),
                            body_len=bl)
    assert st == sonic.OK
    torch.cuda.synchronize()
    assert int(case.status.item()) == sonic.ERR_BAD_LAYOUT
    assert np.array_equal(bf16_to_host(case.kc), kc0) and np.array_equal(case.length.cpu().numpy(), len0)
    assert torch.all(case.out == 7.0)


def test_extend_with_a_pending_layout_error_writes_nothing():
    """A layout error left on the status word by an earlier call stops the whole step: no output,
    no cache row or length changes, and the status keeps the earlier error."""
    H.need_gpu()
    rng = np.random.default_rng(43)
    lays = _ending_layouts(rng, 3, max_h=3, max_b=40, max_k=12, max_s=20)
    batch = W.make_batch("pending", lays, 4, 2, 64, seed=43)
    case = ExtendCase(batch)
    case.status.fill_(sonic.ERR_BAD_LAYOUT)
    kc0, vc0, len0 = bf16_to_host(case.kc).copy(), bf16_to_host(case.vc).copy(), case.length.cpu().numpy().copy()
    assert case.run() == sonic.OK
    assert int(case.status.item()) == sonic.ERR_BAD_LAYOUT
    assert np.array_equal(bf16_to_host(case.kc), kc0) and np.array_equal(bf16_to_host(case.vc), vc0)
    assert np.array_equal(case.length.cpu().numpy(), len0)
    assert torch.all(case.out == 7.0)
