"""Pins of the oracle's Nexus-scope reading A3' (CPU only).

Under A3' a Nexus token sees the Nexus tokens of its own and earlier segments
only.  It is pinned by facts that do not come from the oracle's mask code:

* an independent rule-by-rule enumeration (tests/brute.py) on every small layout;
* a hand-derived golden matrix (tests/golden/mask_two_segments_up_to_own.txt);
* closed-form visible counts per row (Nexus row of segment i: S + b_i + P_i + k_i);
* the incremental identity: the A3' prefill rows of segment i's Nexus tokens equal
  the next-turn step computed when turn i ends, over the cache that turn leaves
  (system prompt, the earlier Nexus tokens, body i), for every segment i;
* A3 and A3' agree on every row except the Nexus rows of segments that have
  Nexus tokens after them.
"""
import os

import numpy as np
import pytest

import workloads as W
from oracle import attention as OA
from oracle import extend as OE
from oracle import mask as OM
from tests import brute
from tests.test_oracle_pins import _layouts_small

UP = OM.NEXUS_UP_TO_OWN


def test_up_to_own_matches_brute_force_on_all_small_layouts():
    for lay in _layouts_small():
        role, turn = lay.roles_and_turns()
        got = OM.visibility(role, turn, UP)
        want = np.array(brute.brute_force_mask(role.tolist(), turn.tolist(), "up_to_own"),
                        dtype=bool).reshape(got.shape)
        assert np.array_equal(got, want), lay


def test_up_to_own_matches_hand_derived_golden(golden_dir):
    roles, turns, rows = brute.read_golden_mask(os.path.join(golden_dir, "mask_two_segments_up_to_own.txt"))
    got = OM.visibility(np.array(roles, np.uint8), np.array(turns, np.int32), UP)
    assert np.array_equal(got, np.array(rows, dtype=bool))


def test_up_to_own_closed_form_counts():
    rng = np.random.default_rng(1201)
    lays = [W.random_layout(rng, max_h=5, max_b=30, max_k=9, max_s=12, max_c=10) for _ in range(60)]
    lays.append(W.workload_structure(1)["layouts"][0])
    for lay in lays:
        role, turn = lay.roles_and_turns()
        got = OM.visibility(role, turn, UP).sum(axis=1)
        want = brute.closed_form_row_counts(lay.system, lay.bodies, lay.nexus, lay.current, "up_to_own")
        assert got.tolist() == want, lay


def test_scopes_differ_only_on_nexus_rows_with_later_nexus():
    rng = np.random.default_rng(1207)
    for _ in range(40):
        lay = W.random_layout(rng, max_h=4, max_b=8, max_k=4, max_s=4, max_c=4)
        role, turn = lay.roles_and_turns()
        a = OM.visibility(role, turn)
        u = OM.visibility(role, turn, UP)
        later = np.zeros(lay.length, bool)   # Nexus rows with Nexus tokens of later segments
        p = lay.system
        for i, (b, k) in enumerate(zip(lay.bodies, lay.nexus)):
            p += b
            later[p:p + k] = sum(lay.nexus[i + 1:]) > 0
            p += k
        assert np.array_equal(a[~later], u[~later])
        assert np.all(u <= a)
        # the difference is exactly the later segments' Nexus keys
        diff = a & ~u
        assert np.all(diff.sum(axis=1)[later] > 0)
        assert np.all(role[np.nonzero(diff)[1]] == W.ROLE_NEXUS)


def _segment_step(lay, i):
    """Positions of the next-turn step that ends turn i: cache rows (system, Nexus of the
    segments before i, body i), the rows kept, and segment i's Nexus positions."""
    S = lay.system
    cache = list(range(S))
    p = S
    for j, (b, k) in enumerate(zip(lay.bodies, lay.nexus)):
        if j < i:
            cache += list(range(p + b, p + b + k))
        elif j == i:
            keep = len(cache)
            cache += list(range(p, p + b))
            return np.array(cache, np.int64), keep, np.arange(p + b, p + b + k)
        p += b + k
    raise ValueError("no such segment")


@pytest.mark.parametrize("seed", range(5))
def test_up_to_own_equals_incremental_steps(seed):
    """Generating each segment's Nexus rows when its turn ends, over the compact cache,
    gives the A3' prefill rows; under A3 it does not once a later segment has Nexus."""
    rng = np.random.default_rng(1300 + seed)
    n_checked = n_differs = 0
    for _ in range(3):
        lay = W.random_layout(rng, max_h=4, max_b=30, max_k=8, max_s=10, max_c=6)
        b = W.make_batch("scope", [lay], 4, 2, 16, seed=int(rng.integers(1 << 30)))
        full_up = OA.prefill_request(b.q, b.k, b.v, b.role, b.turn_id, nexus_scope=UP)
        full_all = OA.prefill_request(b.q, b.k, b.v, b.role, b.turn_id)
        for i, k in enumerate(lay.nexus):
            if k == 0:
                continue
            cache, keep, npos = _segment_step(lay, i)
            out, _, _ = OE.extend_request(b.q[npos], b.k[npos], b.v[npos], b.k[cache], b.v[cache], keep)
            np.testing.assert_allclose(out, full_up[npos], rtol=0, atol=1e-12)
            n_checked += 1
            if sum(lay.nexus[i + 1:]) > 0:
                n_differs += 1
                assert np.max(np.abs(out - full_all[npos])) > 1e-6
    assert n_checked > 0 and n_differs > 0
