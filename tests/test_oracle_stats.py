"""Pins of the attention-statistics oracle (CPU only).

* brute force: pure-Python loops over the rule-by-rule mask of tests/brute.py and
  a textbook softmax, on tiny inputs, under both Nexus scopes;
* uniform attention (Q = 0): closed forms from the visible counts of the rules;
* invariants: the key weights of a request sum to its number of current rows, and
  their Nexus part equals the head-averaged Nexus mass of the current rows;
* planted mistakes (wrong row set, wrong key set) are caught.
"""
import math
import struct

import numpy as np
import pytest

import workloads as W
from oracle import layout as OL
from oracle import mask as OM
from oracle import stats as OS
from tests import brute


def _widen(bits):
    return struct.unpack("<f", struct.pack("<I", int(bits) << 16))[0]


def _brute_stats(q, k, role, turn, scope):
    """A_nexus [L][Hq] and w [L] by plain loops."""
    L, Hq, d = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    vis = brute.brute_force_mask(role.tolist(), turn.tolist(), scope)
    scale = 1.0 / math.sqrt(d)
    mass = [[0.0] * Hq for _ in range(L)]
    w = [0.0] * L
    for h in range(Hq):
        g = h // G
        for p in range(L):
            s = {}
            for x in range(L):
                if vis[p][x]:
                    s[x] = scale * sum(_widen(q[p, h, i]) * _widen(k[x, g, i]) for i in range(d))
            mx = max(s.values())
            z = sum(math.exp(v - mx) for v in s.values())
            for x, v in s.items():
                pr = math.exp(v - mx) / z
                if role[x] == OL.NEXUS:
                    mass[p][h] += pr
                if role[p] == OL.CURRENT:
                    w[x] += pr / Hq
    return np.array(mass), np.array(w)


@pytest.mark.parametrize("scope", [OM.NEXUS_ALL, OM.NEXUS_UP_TO_OWN])
def test_stats_match_brute_force(scope):
    rng = np.random.default_rng(1500)
    lays = [W.RequestLayout(2, [3, 2], [2, 3], 3), W.RequestLayout(0, [4], [0], 2),
            W.RequestLayout(1, [2, 1, 2], [1, 2, 1], 0)]
    lays += [W.random_layout(rng, max_h=3, max_b=4, max_k=3, max_s=3, max_c=3) for _ in range(4)]
    for lay in lays:
        b = W.make_batch("stats", [lay], 4, 2, 8, seed=int(rng.integers(1 << 30)))
        mass, w = _brute_stats(b.q, b.k, b.role, b.turn_id, scope)
        np.testing.assert_allclose(OS.nexus_mass(b.q, b.k, b.role, b.turn_id, nexus_scope=scope), mass,
                                   rtol=0, atol=1e-12)
        np.testing.assert_allclose(OS.key_weight(b.q, b.k, b.role, b.turn_id, nexus_scope=scope), w,
                                   rtol=0, atol=1e-12)


def _uniform_closed_forms(lay):
    """Q = 0: every visible key gets 1/|vis(p)|.  Returns (A_nexus per row, w per key)."""
    S, C, K = lay.system, lay.current, sum(lay.nexus)
    mass, w = [0.0] * S, []
    P = 0
    for b, k in zip(lay.bodies, lay.nexus):
        mass += [P / (S + P + r + 1) for r in range(b)]
        mass += [K / (S + b + K)] * k
        P += k
    mass += [K / (S + K + r + 1) for r in range(C)]
    to_all = sum(1.0 / (S + K + r + 1) for r in range(C))     # a system or Nexus key
    w += [to_all] * S
    for b, k in zip(lay.bodies, lay.nexus):
        w += [0.0] * b + [to_all] * k
    w += [sum(1.0 / (S + K + r + 1) for r in range(j, C)) for j in range(C)]
    return np.array(mass), np.array(w)


def test_uniform_attention_closed_forms():
    rng = np.random.default_rng(1510)
    lays = [W.random_layout(rng, max_h=4, max_b=20, max_k=6, max_s=8, max_c=9) for _ in range(25)]
    lays.append(W.workload_structure(1)["layouts"][0])
    for lay in lays:
        b = W.make_batch("uniform", [lay], 4, 2, 16, seed=3)
        q = np.zeros_like(b.q)
        mass_cf, w_cf = _uniform_closed_forms(lay)
        mass = OS.nexus_mass(q, b.k, b.role, b.turn_id)
        for h in range(4):
            np.testing.assert_allclose(mass[:, h], mass_cf, rtol=0, atol=1e-12)
        np.testing.assert_allclose(OS.key_weight(q, b.k, b.role, b.turn_id), w_cf, rtol=0, atol=1e-12)


@pytest.mark.parametrize("scope", [OM.NEXUS_ALL, OM.NEXUS_UP_TO_OWN])
def test_weights_sum_to_current_rows_and_tie_to_nexus_mass(scope):
    rng = np.random.default_rng(1520)
    for _ in range(6):
        lay = W.random_layout(rng, max_h=4, max_b=30, max_k=9, max_s=10, max_c=12)
        b = W.make_batch("tie", [lay], 6, 2, 16, seed=int(rng.integers(1 << 30)))
        w = OS.key_weight(b.q, b.k, b.role, b.turn_id, nexus_scope=scope)
        assert abs(w.sum() - lay.current) < 1e-10
        assert np.all(w[b.role == OL.HISTORY_TEXT] == 0)
        cur = np.nonzero(b.role == OL.CURRENT)[0]
        mass = OS.nexus_mass(b.q, b.k, b.role, b.turn_id, rows=cur, nexus_scope=scope)
        assert abs(w[b.role == OL.NEXUS].sum() - mass.sum() / mass.shape[1] if len(cur) else 0) < 1e-10


def test_weights_over_wrong_rows_are_caught(monkeypatch):
    lay = W.RequestLayout(3, [6, 4], [2, 3], 5)
    b = W.make_batch("mut", [lay], 4, 2, 16, seed=11)
    monkeypatch.setattr(OS, "CURRENT", OL.HISTORY_TEXT)
    w = OS.key_weight(b.q, b.k, b.role, b.turn_id)
    assert abs(w.sum() - lay.current) > 1e-3


def test_mass_over_wrong_keys_is_caught(monkeypatch):
    lay = W.RequestLayout(3, [6, 4], [2, 3], 5)
    b = W.make_batch("mut", [lay], 4, 2, 16, seed=11)
    monkeypatch.setattr(OS, "NEXUS", OL.SYSTEM)
    mass = OS.nexus_mass(np.zeros_like(b.q), b.k, b.role, b.turn_id)
    assert np.max(np.abs(mass[:, 0] - _uniform_closed_forms(lay)[0])) > 1e-3
