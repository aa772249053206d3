"""Seeded input generator: determinism and the stated structure of each workload (CPU)."""
import numpy as np
import pytest

import workloads as W


def test_same_seed_same_bytes():
    a = W.workload(1)
    b = W.workload(1)
    for name in ("q", "k", "v", "dec_q", "dec_k", "dec_v", "role", "turn_id", "cu_seqlens"):
        assert np.array_equal(getattr(a, name), getattr(b, name)), name


@pytest.mark.parametrize("idx,B,L,kept", [(1, 1, 504, 120), (2, 8, 5424, 1328), (4, 4, 40320, 7552)])
def test_uniform_workload_shapes(idx, B, L, kept):
    st = W.workload_structure(idx)
    lays = st["layouts"]
    assert len(lays) == B
    for lay in lays:
        assert lay.length == L
        assert lay.system + sum(lay.nexus) + lay.current == kept


def test_ragged_workload_ranges():
    st = W.workload_structure(3)
    assert len(st["layouts"]) == 16 and st["scales"]
    for lay in st["layouts"]:
        assert 2 <= len(lay.bodies) <= 12
        assert 128 <= lay.system <= 512 and 32 <= lay.current <= 512
        assert all(64 <= b <= 1024 for b in lay.bodies)
        assert lay.nexus == [b // 2 for b in lay.bodies]


def test_ragged_scales_in_range():
    b = W.workload(3, decode_steps=1)
    for s in (b.scale_q, b.scale_k, b.scale_v):
        assert np.all((s >= 0.5) & (s <= 2.0))


def test_dynamic_budget_workload_ranges():
    st = W.workload_structure(5)
    assert len(st["layouts"]) == 64
    for lay, r, full in zip(st["layouts"], st["ratios"], st["full_lengths"]):
        assert r in (0.1, 0.2, 0.5)
        assert 1024 <= full <= 8192
        assert lay.system + sum(lay.bodies) + lay.current == full
        assert all(k == max(1, int(np.floor(r * b))) for b, k in zip(lay.bodies, lay.nexus))


def test_roles_and_turns_follow_sequence_order():
    lay = W.RequestLayout(2, [3, 1], [1, 0], 2)
    role, turn = lay.roles_and_turns()
    assert role.tolist() == [0, 0, 1, 1, 1, 2, 1, 3, 3]
    assert turn.tolist() == [0, 0, 1, 1, 1, 1, 2, 3, 3]


def test_text_only_layout_drops_nexus():
    lay = W.RequestLayout(2, [3, 4], [1, 2], 5)
    t = W.text_only_layout(lay)
    assert t.length == 2 + 7 + 5 and sum(t.nexus) == 0
