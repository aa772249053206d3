"""Pins of the role-routed projection oracle (CPU only).

* brute force: pure-Python loops with an independent bf16 widening, tiny sizes;
* one-hot probe: x[t] = e_k picks column k of the weight set of row t's role, so
  a transposed weight or a row sent to the wrong set shows up exactly;
* equal weight sets make the roles irrelevant; exchanging the weight sets equals
  exchanging Nexus and non-Nexus roles;
* planted mistakes (current rows routed like Nexus rows, weights transposed) are caught.
"""
import struct

import numpy as np

import workloads as W
from oracle import layout as OL
from oracle import projection as OP


def _widen(bits):
    return struct.unpack("<f", struct.pack("<I", int(bits) << 16))[0]


def _bits(rng, shape):
    return W.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def _roles(rng, T):
    lay = W.RequestLayout(2, [3, 2], [2, 3], T - 12)
    role, _ = lay.roles_and_turns()
    return role


def test_matches_brute_force():
    rng = np.random.default_rng(1600)
    T, K, N = 12 + 5, 9, 6
    role = _roles(rng, T)
    x, wt, wn = _bits(rng, (T, K)), _bits(rng, (N, K)), _bits(rng, (N, K))
    y = OP.role_routed_linear(x, role, wt, wn)
    for t in range(T):
        w = wn if role[t] == OL.NEXUS else wt
        for n in range(N):
            want = sum(_widen(x[t, k]) * _widen(w[n, k]) for k in range(K))
            assert abs(y[t, n] - want) < 1e-12


def test_one_hot_inputs_select_weight_columns():
    rng = np.random.default_rng(1601)
    T, K, N = 12 + 4, 8, 5
    role = _roles(rng, T)
    wt, wn = _bits(rng, (N, K)), _bits(rng, (N, K))
    x = np.zeros((T, K), np.uint16)
    cols = rng.integers(0, K, T)
    x[np.arange(T), cols] = 0x3F80   # 1.0
    y = OP.role_routed_linear(x, role, wt, wn)
    for t in range(T):
        w = wn if role[t] == OL.NEXUS else wt
        assert np.array_equal(y[t], [_widen(b) for b in w[:, cols[t]]])


def test_equal_weights_and_role_exchange():
    rng = np.random.default_rng(1602)
    T, K, N = 12 + 8, 32, 16
    role = _roles(rng, T)
    x, wt, wn = _bits(rng, (T, K)), _bits(rng, (N, K)), _bits(rng, (N, K))
    all_text = np.full(T, OL.CURRENT, np.uint8)
    assert np.array_equal(OP.role_routed_linear(x, role, wt, wt), OP.role_routed_linear(x, all_text, wt, wt))
    flipped = np.where(role == OL.NEXUS, OL.CURRENT, OL.NEXUS).astype(np.uint8)
    assert np.array_equal(OP.role_routed_linear(x, role, wt, wn), OP.role_routed_linear(x, flipped, wn, wt))


def _one_hot_pin_holds():
    try:
        test_one_hot_inputs_select_weight_columns()
        return True
    except AssertionError:
        return False


def test_pin_holds_unmutated():
    assert _one_hot_pin_holds()


def test_current_rows_routed_to_nexus_weights_is_caught(monkeypatch):
    real = OP.role_routed_linear

    def misrouted(x, role, w_text, w_nexus):
        role = np.where(np.asarray(role) == OL.CURRENT, OL.NEXUS, role)
        return real(x, role, w_text, w_nexus)
    monkeypatch.setattr(OP, "role_routed_linear", misrouted)
    assert not _one_hot_pin_holds()


def test_transposed_weights_are_caught(monkeypatch):
    real = OP.role_routed_linear

    def transposed(x, role, w_text, w_nexus):
        K = x.shape[1]
        pad = lambda w: np.pad(w.T, ((0, 0), (0, max(0, K - w.shape[0]))))[:, :K]
        return real(x, role, pad(w_text), pad(w_nexus))[:, :w_text.shape[0]]
    monkeypatch.setattr(OP, "role_routed_linear", transposed)
    assert not _one_hot_pin_holds()
