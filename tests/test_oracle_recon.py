"""Pins of the reconstruction-target oracle (CPU only).

* brute force: pure-Python loops (independent widening, cosine, softmax, entropy);
* the sub-intervals tile each body: disjoint, in order, sizes within one of each
  other when b >= K; single tokens covering every body token when b < K;
* closed cases: identical rows give exactly that row and ratio 1; a zero Nexus
  state gives uniform weights (the mean, ratio 1); a one-token interval gives
  that token;
* cosine weights do not change when h(N) is scaled;
* planted mistakes (dot products instead of cosines, overlapping intervals) are caught.
"""
import math
import struct

import numpy as np
import pytest

import workloads as W
from oracle import recon as OR


def _widen(bits):
    return struct.unpack("<f", struct.pack("<I", int(bits) << 16))[0]


def _bits(rng, shape):
    return W.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def _brute(h, lay):
    """Targets, cosines and ratios by plain loops, position order."""
    Dm = h.shape[1]
    vec = lambda p: [_widen(h[p, i]) for i in range(Dm)]
    dot = lambda a, b: sum(u * v for u, v in zip(a, b))
    cos = lambda a, b: (dot(a, b) / math.sqrt(dot(a, a) * dot(b, b))) if dot(a, a) > 0 and dot(b, b) > 0 else 0.0
    out = []
    p = lay.system
    for b, k in zip(lay.bodies, lay.nexus):
        for j in range(k):
            s = j * b // k
            e = max((j + 1) * b // k, s + 1)
            hn = vec(p + b + j)
            rows = [vec(p + x) for x in range(s, e)]
            ws = [math.exp(cos(hn, r)) for r in rows]
            z = sum(ws)
            al = [w / z for w in ws]
            t = [sum(al[r] * rows[r][i] for r in range(len(rows))) for i in range(Dm)]
            H = -sum(a * math.log(a) for a in al)
            out.append((t, cos(hn, t), H / math.log(len(rows)) if len(rows) > 1 else 1.0))
        p += b + k
    return out


def test_matches_brute_force():
    rng = np.random.default_rng(1700)
    for lay in [W.RequestLayout(2, [7, 3, 1], [3, 5, 2], 2), W.RequestLayout(0, [10], [4], 0),
                W.RequestLayout(1, [2, 9], [0, 9], 1)]:
        h = _bits(rng, (lay.length, 6))
        role, turn = lay.roles_and_turns()
        t, c, r = OR.recon_request(h, role, turn)
        want = _brute(h, lay)
        assert len(want) == len(t)
        for i, (wt, wc, wr) in enumerate(want):
            np.testing.assert_allclose(t[i], wt, rtol=0, atol=1e-12)
            assert abs(c[i] - wc) < 1e-12 and abs(r[i] - wr) < 1e-12


@pytest.mark.parametrize("b", list(range(1, 40)))
def test_intervals_tile_the_body(b):
    for K in range(1, 45):
        iv = [OR.interval(j, b, K) for j in range(K)]
        assert all(0 <= s < e <= b for s, e in iv)
        if b >= K:
            assert iv[0][0] == 0 and iv[-1][1] == b
            assert all(iv[j][1] == iv[j + 1][0] for j in range(K - 1))
            sizes = [e - s for s, e in iv]
            assert max(sizes) - min(sizes) <= 1
        else:
            assert all(e - s == 1 for s, e in iv)
            starts = [s for s, _ in iv]
            assert starts == sorted(starts) and set(starts) == set(range(b))


def test_closed_cases():
    rng = np.random.default_rng(1701)
    lay = W.RequestLayout(1, [12, 5], [3, 5], 0)   # intervals of 4 rows, then single rows
    role, turn = lay.roles_and_turns()
    h = _bits(rng, (lay.length, 16))
    body0 = np.arange(1, 13)
    h[body0] = h[body0[0]]                          # identical rows in segment 1
    t, c, r = OR.recon_request(h, role, turn)
    row = OR.bf16_bits_to_f64(h[body0[0]])
    for j in range(3):
        assert np.array_equal(t[j], row) and abs(r[j] - 1) < 1e-12
    for j in range(5):                              # one-token intervals: the token itself
        assert np.array_equal(t[3 + j], OR.bf16_bits_to_f64(h[1 + 12 + 3 + j])) and r[3 + j] == 1.0
    h2 = h.copy()
    h2[13:16] = 0                                   # zero Nexus states of segment 1: the plain mean
    body0_rows = OR.bf16_bits_to_f64(_bits(rng, (12, 16)))
    h2[body0] = W.f32_to_bf16_bits(body0_rows.astype(np.float32))
    t2, c2, r2 = OR.recon_request(h2, role, turn)
    hf = OR.bf16_bits_to_f64(h2)
    for j in range(3):
        np.testing.assert_allclose(t2[j], hf[1 + 4 * j:1 + 4 * j + 4].mean(axis=0), rtol=0, atol=1e-12)
        assert abs(r2[j] - 1) < 1e-12 and c2[j] == 0


def test_scaling_the_nexus_state_changes_nothing():
    rng = np.random.default_rng(1702)
    lay = W.RequestLayout(3, [20, 9], [4, 3], 2)
    role, turn = lay.roles_and_turns()
    h = _bits(rng, (lay.length, 32))
    h2 = h.copy()
    nexus = np.nonzero(role == W.ROLE_NEXUS)[0]
    h2[nexus] = W.f32_to_bf16_bits((OR.bf16_bits_to_f64(h[nexus]) * 4.0).astype(np.float32))   # exact in bf16
    a, b = OR.recon_request(h, role, turn), OR.recon_request(h2, role, turn)
    for u, v in zip(a, b):
        np.testing.assert_allclose(u, v, rtol=1e-12, atol=1e-12)


def _scale_pin_holds():
    try:
        test_scaling_the_nexus_state_changes_nothing()
        return True
    except AssertionError:
        return False


def _tiling_pin_holds():
    try:
        for b in (5, 17, 33):
            test_intervals_tile_the_body(b)
        return True
    except AssertionError:
        return False


def test_pins_hold_unmutated():
    assert _scale_pin_holds() and _tiling_pin_holds()


def test_dot_products_instead_of_cosines_are_caught(monkeypatch):
    monkeypatch.setattr(OR, "_cos", lambda a, B: B @ a)
    assert not _scale_pin_holds()


def test_overlapping_intervals_are_caught(monkeypatch):
    monkeypatch.setattr(OR, "interval", lambda j, b, K: ((j * b) // K, min(b, -(-((j + 1) * b) // K) + 1)))
    assert not _tiling_pin_holds()
