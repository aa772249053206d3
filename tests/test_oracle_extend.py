"""Pins of the next-turn Nexus oracle (CPU only).

The incremental step must reproduce, row for row, what the full masked prefill
computes for the newest segment's Nexus tokens (Sec. 3.2 mask, explicit), and
leave exactly the cache that compaction of the whole layout leaves.
"""
import numpy as np
import pytest

import workloads as W
from oracle import attention as OA
from oracle import compaction as OC
from oracle import extend as OE


def _case(rng, lay, Hq=4, Hkv=2, d=32, seed=None):
    b = W.make_batch("ext", [lay], Hq, Hkv, d, seed=int(rng.integers(1 << 30)) if seed is None else seed)
    cache_pos, keep, nexus_pos = W.extend_positions(lay)
    return b, cache_pos, keep, nexus_pos


def _layouts(rng, n):
    out = []
    while len(out) < n:
        lay = W.random_layout(rng, max_h=4, max_b=40, max_k=12, max_s=20, max_c=0)
        if lay.bodies and lay.nexus[-1] > 0:
            out.append(lay)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_extend_equals_full_prefill_rows(seed):
    rng = np.random.default_rng(900 + seed)
    for lay in _layouts(rng, 3):
        b, cache_pos, keep, nexus_pos = _case(rng, lay)
        full = OA.prefill_request(b.q, b.k, b.v, b.role, b.turn_id, rows=nexus_pos)
        out, nk, nv = OE.extend_request(b.q[nexus_pos], b.k[nexus_pos], b.v[nexus_pos], b.k[cache_pos],
                                        b.v[cache_pos], keep)
        np.testing.assert_allclose(out, full, rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_extend_cache_equals_compaction(seed):
    rng = np.random.default_rng(950 + seed)
    for lay in _layouts(rng, 3):
        b, cache_pos, keep, nexus_pos = _case(rng, lay)
        _, nk, nv = OE.extend_request(b.q[nexus_pos], b.k[nexus_pos], b.v[nexus_pos], b.k[cache_pos],
                                      b.v[cache_pos], keep)
        L = lay.length
        kc = np.zeros((L, b.num_kv_heads, b.head_dim), np.uint16)
        vc = kc.copy()
        n = OC.compact_batch(b.k, b.v, b.role, np.array([0, L]), [0], [L], kc, vc, np.zeros(L, np.int32))
        assert np.array_equal(nk, kc[:n[0]]) and np.array_equal(nv, vc[:n[0]])


def test_body_excluded_mutation_is_caught():
    """Leaving the turn's own body out of the keys (a plausible mistake) breaks the pin."""
    rng = np.random.default_rng(990)
    lay = W.RequestLayout(6, [5, 9], [3, 4], 0)
    b, cache_pos, keep, nexus_pos = _case(rng, lay)
    full = OA.prefill_request(b.q, b.k, b.v, b.role, b.turn_id, rows=nexus_pos)
    wrong, _, _ = OE.extend_request(b.q[nexus_pos], b.k[nexus_pos], b.v[nexus_pos], b.k[cache_pos[:keep]],
                                    b.v[cache_pos[:keep]], keep)
    assert np.abs(wrong - full).max() > 1e-3


def test_no_nexus_rows_only_drops_the_body():
    rng = np.random.default_rng(991)
    lay = W.RequestLayout(4, [3, 5], [2, 0], 0)
    b, cache_pos, keep, nexus_pos = _case(rng, lay)
    out, nk, _ = OE.extend_request(b.q[nexus_pos], b.k[nexus_pos], b.v[nexus_pos], b.k[cache_pos],
                                   b.v[cache_pos], keep)
    assert out.shape[0] == 0 and np.array_equal(nk, b.k[cache_pos[:keep]])


def _two_segment_layouts(rng, n):
    out = []
    while len(out) < n:
        lay = W.random_layout(rng, max_h=5, max_b=40, max_k=12, max_s=20, max_c=0)
        if len(lay.bodies) >= 2 and lay.nexus[-2] > 0:
            out.append(lay)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_two_segment_turn_equals_own_and_earlier_scope_prefill(seed):
    """Utterance then response, one step each: the Nexus rows of both segments equal the full
    prefill's under the own-and-earlier Nexus scope, and the final cache equals the compaction
    of the whole layout."""
    from oracle import mask as OM
    rng = np.random.default_rng(1200 + seed)
    for lay in _two_segment_layouts(rng, 3):
        b = W.make_batch("turn", [lay], 4, 2, 32, seed=int(rng.integers(1 << 30)))
        cache, keep, ulen, nu, nr = W.turn_positions(lay)
        out1, k1, v1 = OE.extend_request(b.q[nu], b.k[nu], b.v[nu], b.k[cache], b.v[cache], keep, body_len=ulen)
        out2, k2, v2 = OE.extend_request(b.q[nr], b.k[nr], b.v[nr], k1, v1, keep + len(nu))
        full = OA.prefill_request(b.q, b.k, b.v, b.role, b.turn_id, rows=np.concatenate([nu, nr]),
                                  nexus_scope=OM.NEXUS_UP_TO_OWN)
        np.testing.assert_allclose(np.concatenate([out1, out2]), full, rtol=0, atol=1e-12)
        L = lay.length
        kc = np.zeros((L, b.num_kv_heads, b.head_dim), np.uint16)
        vc = kc.copy()
        n = OC.compact_batch(b.k, b.v, b.role, np.array([0, L]), [0], [L], kc, vc, np.zeros(L, np.int32))
        assert np.array_equal(k2, kc[:n[0]]) and np.array_equal(v2, vc[:n[0]])


def test_two_segment_turn_with_the_whole_tail_as_body_is_caught():
    """Treating utterance and response as one body (a plausible mistake) gives the utterance's
    Nexus rows keys they must not see (the response comes after them)."""
    from oracle import mask as OM
    rng = np.random.default_rng(1290)
    lay = W.RequestLayout(5, [7, 9, 11], [3, 4, 2], 0)
    b = W.make_batch("turn", [lay], 4, 2, 32, seed=5)
    cache, keep, ulen, nu, nr = W.turn_positions(lay)
    full = OA.prefill_request(b.q, b.k, b.v, b.role, b.turn_id, rows=nu, nexus_scope=OM.NEXUS_UP_TO_OWN)
    wrong, _, _ = OE.extend_request(b.q[nu], b.k[nu], b.v[nu], b.k[cache], b.v[cache], keep)
    assert np.abs(wrong - full).max() > 1e-3
    right, _, _ = OE.extend_request(b.q[nu], b.k[nu], b.v[nu], b.k[cache], b.v[cache], keep, body_len=ulen)
    np.testing.assert_allclose(right, full, rtol=0, atol=1e-12)
