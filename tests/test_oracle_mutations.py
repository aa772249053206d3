"""Planted mistakes in the oracle (CPU only): each must be caught by a pin.

This shows the pins in test_oracle_pins.py are sharp enough: a dropped rule,
a misread reading, a wrong normaliser, a wrong head mapping or a swapped
operand each makes at least one pin fail.  The mistakes are planted with
monkeypatch, in the oracle, on the CPU, and undone after each test.
"""
import numpy as np
import torch

import workloads as W
from oracle import attention as OA
from oracle import mask as OM
from tests import brute


def _brute_pin_holds():
    rng = np.random.default_rng(41)
    for _ in range(40):
        lay = W.random_layout(rng, max_h=3, max_b=4, max_k=3, max_s=2, max_c=2)
        role, turn = lay.roles_and_turns()
        got = OM.visibility(role, turn)
        want = np.array(brute.brute_force_mask(role.tolist(), turn.tolist()), dtype=bool).reshape(got.shape)
        if not np.array_equal(got, want):
            return False
    return True


def _bits(rng, shape):
    return W.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def _rows_sum_pin_holds():
    rng = np.random.default_rng(43)
    lay = W.RequestLayout(3, [5, 4], [2, 3], 3)
    role, turn = lay.roles_and_turns()
    q, k = _bits(rng, (lay.length, 1, 8)), _bits(rng, (lay.length, 1, 8))
    P = OA.request_probs(q, k, role, turn, 0)
    return bool(np.all(np.abs(P.sum(axis=1) - 1) < 1e-12))


def _causal_pin_holds():
    rng = np.random.default_rng(47)
    lay = W.RequestLayout(20, [], [], 0)
    L, H, d = lay.length, 2, 8
    q, k, v = _bits(rng, (L, H, d)), _bits(rng, (L, H, d)), _bits(rng, (L, H, d))
    role, turn = lay.roles_and_turns()
    got = OA.prefill_request(q, k, v, role, turn)
    # widen through torch's own bfloat16 type, independent of the oracle
    t = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).double().permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=True)
    return bool(np.max(np.abs(got - ref.permute(1, 0, 2).numpy())) < 1e-12)


def _gqa_pin_holds():
    rng = np.random.default_rng(53)
    lay = W.RequestLayout(2, [4], [2], 3)
    L = lay.length
    q, k, v = _bits(rng, (L, 6, 8)), _bits(rng, (L, 2, 8)), _bits(rng, (L, 2, 8))
    role, turn = lay.roles_and_turns()
    a = OA.prefill_request(q, k, v, role, turn)
    b = OA.prefill_request(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), role, turn)
    return bool(np.array_equal(a, b))


def test_pins_hold_unmutated():
    assert _brute_pin_holds() and _rows_sum_pin_holds() and _causal_pin_holds() and _gqa_pin_holds()


def test_dropping_body_removal_is_caught(monkeypatch):
    monkeypatch.setattr(OM, "_last_of_key", lambda parsed: np.full(parsed.length, 1 << 62, dtype=np.int64))
    assert not _brute_pin_holds()


def test_ending_segment_at_its_body_is_caught(monkeypatch):
    def last_body_only(parsed):
        last = np.full(parsed.length, 1 << 62, dtype=np.int64)
        for s in parsed.segments:
            last[s.body_start:s.body_start + s.body_len] = s.body_start + s.body_len - 1
        return last
    monkeypatch.setattr(OM, "_last_of_key", last_body_only)
    assert not _brute_pin_holds()


def test_nexus_visibility_only_within_segment_is_caught(monkeypatch):
    real = OM.visibility_rows

    def within_segment_only(role, turn_id, rows=None, parsed=None, nexus_scope=OM.NEXUS_ALL):
        vis = real(role, turn_id, rows, parsed, nexus_scope)
        role = np.asarray(role)
        turn_id = np.asarray(turn_id)
        p = np.arange(len(role)) if rows is None else np.asarray(rows)
        cross = (role[p] == 2)[:, None] & (role == 2)[None, :] & (turn_id[p][:, None] != turn_id[None, :])
        return vis & ~cross
    monkeypatch.setattr(OM, "visibility_rows", within_segment_only)
    assert not _brute_pin_holds()


def test_softmax_over_all_keys_is_caught(monkeypatch):
    def unmasked_denominator(scores, vis):
        e = np.exp(scores - scores.max(axis=1, keepdims=True))
        return np.where(vis, e, 0.0) / e.sum(axis=1, keepdims=True)
    monkeypatch.setattr(OA, "softmax_probs", unmasked_denominator)
    assert not _rows_sum_pin_holds()


def test_wrong_gqa_mapping_is_caught(monkeypatch):
    monkeypatch.setattr(OA, "kv_head", lambda h, hq, hkv: h % hkv)
    assert not _gqa_pin_holds()


def test_keys_used_as_values_is_caught(monkeypatch):
    real = OA.bf16_bits_to_f64
    calls = {"n": 0}

    def swap_third(bits):
        # prefill_request widens q, k, v in that order; hand back k for v
        calls["n"] += 1
        if calls["n"] % 3 == 0:
            return swap_third.last_k
        out = real(bits)
        if calls["n"] % 3 == 2:
            swap_third.last_k = out
        return out
    monkeypatch.setattr(OA, "bf16_bits_to_f64", swap_third)
    assert not _causal_pin_holds()


def _up_to_own_pin_holds():
    rng = np.random.default_rng(59)
    for _ in range(40):
        lay = W.random_layout(rng, max_h=3, max_b=4, max_k=3, max_s=2, max_c=2)
        role, turn = lay.roles_and_turns()
        got = OM.visibility(role, turn, OM.NEXUS_UP_TO_OWN)
        want = np.array(brute.brute_force_mask(role.tolist(), turn.tolist(), "up_to_own"),
                        dtype=bool).reshape(got.shape)
        if not np.array_equal(got, want):
            return False
    return True


def test_up_to_own_pin_holds_unmutated():
    assert _up_to_own_pin_holds()


def test_up_to_own_seeing_every_segment_is_caught(monkeypatch):
    """Reading A3' collapsed back to Eq.(5) as written (one segment index for all)."""
    monkeypatch.setattr(OM, "_nexus_segment", lambda parsed: np.zeros(parsed.length, dtype=np.int64))
    assert not _up_to_own_pin_holds()


def test_up_to_own_reversed_segment_order_is_caught(monkeypatch):
    """Later segments seen instead of earlier ones."""
    real = OM._nexus_segment
    monkeypatch.setattr(OM, "_nexus_segment", lambda parsed: -real(parsed))
    assert not _up_to_own_pin_holds()
