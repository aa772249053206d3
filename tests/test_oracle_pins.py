"""Pins of the fp64 oracle against things other than itself (CPU only).

Each check is chosen so that a plausible slip in the oracle (a dropped rule, a
wrong index, a transposed operand, a wrong normaliser) fails at least one:

* mask == brute-force application of the Sec. 3.2 rules on every small layout;
* mask == hand-derived golden matrices (tests/golden);
* per-row visible counts == closed forms derived from the rules;
* a layout without history reduces to textbook causal attention (torch SDPA);
* softmax rows sum to one and vanish exactly on masked keys;
* Q = 0 gives the plain mean of V over the visible keys;
* decode over the compacted cache == masked decode over the full cache (App. C);
* the prefill row of the last current token == decode of that token over the
  compacted cache, tying the prefill to the decode definition;
* GQA == MHA with every kv-head repeated for its q-heads.
"""
import itertools
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import attention as OA
from oracle import compaction as OC
from oracle import decode as OD
from oracle import layout as OL
from oracle import mask as OM
from tests import brute


def _layouts_small():
    """Every layout with S in {0,1,2}, h <= 2, b_i in {1,2,3}, k_i in {0..3}, C in {0,1,2},
    plus a seeded sample of h = 3 layouts."""
    out = []
    for S, C in itertools.product(range(3), range(3)):
        for h in range(3):
            for bk in itertools.product(itertools.product(range(1, 4), range(4)), repeat=h):
                out.append(W.RequestLayout(S, [b for b, _ in bk], [k for _, k in bk], C))
    rng = np.random.default_rng(7)
    for _ in range(300):
        out.append(W.RequestLayout(int(rng.integers(0, 3)), [int(x) for x in rng.integers(1, 4, 3)],
                                   [int(x) for x in rng.integers(0, 4, 3)], int(rng.integers(0, 3))))
    return out


def test_mask_matches_brute_force_on_all_small_layouts():
    lays = _layouts_small()
    assert len(lays) > 1500
    for lay in lays:
        role, turn = lay.roles_and_turns()
        got = OM.visibility(role, turn)
        want = np.array(brute.brute_force_mask(role.tolist(), turn.tolist()), dtype=bool).reshape(got.shape)
        assert np.array_equal(got, want), lay


@pytest.mark.parametrize("name", ["mask_two_segments.txt", "mask_empty_nexus.txt"])
def test_mask_matches_hand_derived_golden(golden_dir, name):
    roles, turns, rows = brute.read_golden_mask(os.path.join(golden_dir, name))
    got = OM.visibility(np.array(roles, np.uint8), np.array(turns, np.int32))
    assert np.array_equal(got, np.array(rows, dtype=bool))


def test_additive_mask_values():
    lay = W.RequestLayout(1, [2], [1], 1)
    role, turn = lay.roles_and_turns()
    M = OM.additive_mask(role, turn)
    assert set(np.unique(M).tolist()) <= {0.0, -np.inf}
    assert np.array_equal(M == 0.0, OM.visibility(role, turn))


@pytest.mark.parametrize("idx", [1, 2])
def test_visible_counts_closed_form_workloads(idx):
    st = W.workload_structure(idx)
    lay = st["layouts"][0]
    role, turn = lay.roles_and_turns()
    counts = OM.visibility(role, turn).sum(axis=1)
    want = brute.closed_form_row_counts(lay.system, lay.bodies, lay.nexus, lay.current)
    assert counts.tolist() == want
    # totals per request quoted for these workloads: 50,736 (L=504) and 5,194,240 (L=5,424)
    assert int(counts.sum()) == {1: 50736, 2: 5194240}[idx]


def test_visible_counts_closed_form_random():
    rng = np.random.default_rng(11)
    for _ in range(60):
        lay = W.random_layout(rng)
        role, turn = lay.roles_and_turns()
        counts = OM.visibility(role, turn).sum(axis=1)
        assert counts.tolist() == brute.closed_form_row_counts(lay.system, lay.bodies, lay.nexus, lay.current)


def test_long_dialogue_total_visible_pairs_by_rows():
    # L = 40,320 is too large for one explicit matrix in a unit test; count row blocks.
    st = W.workload_structure(4)
    lay = st["layouts"][0]
    role, turn = lay.roles_and_turns()
    parsed = OL.parse(role, turn)
    total = 0
    rows = np.arange(lay.length)
    for r0 in range(0, lay.length, 4096):
        total += int(OM.visibility_rows(role, turn, rows[r0:r0 + 4096], parsed=parsed).sum())
    assert total == 193692160
    assert total == sum(brute.closed_form_row_counts(lay.system, lay.bodies, lay.nexus, lay.current))


# ---------------------------------------------------------------------------
# grammar
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("roles,turns", [
    ([2, 2], [1, 1]),                  # Nexus without a body
    ([0, 2], [0, 1]),                  # Nexus right after the system prompt
    ([1, 0], [1, 0]),                  # system after history
    ([3, 1], [2, 1]),                  # history after the current query
    ([1, 2, 2], [1, 1, 2]),            # Nexus segment id changes inside N_i
    ([1, 1], [2, 1]),                  # segment id decreases
    ([1, 2, 1], [1, 1, 1]),            # next segment reuses the id
    ([0, 4], [0, 0]),                  # unknown role code
    ([3, 2], [1, 1]),                  # Nexus inside the current query
])
def test_grammar_rejects(roles, turns):
    with pytest.raises(OL.LayoutError):
        OL.parse(np.array(roles), np.array(turns))


def test_grammar_accepts_degenerate():
    for roles, turns in [([], []), ([0], [0]), ([3], [0]), ([1], [5]), ([1, 1, 3], [1, 2, 0])]:
        OL.parse(np.array(roles, dtype=np.int64), np.array(turns, dtype=np.int64))


# ---------------------------------------------------------------------------
# attention core
# ---------------------------------------------------------------------------
def _bits(rng, shape, scale=1.0):
    return W.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * scale)


@pytest.mark.parametrize("lay", [W.RequestLayout(37, [], [], 0), W.RequestLayout(11, [], [], 29),
                                 W.RequestLayout(0, [40], [0], 0)])
def test_causal_reduction_matches_sdpa(lay):
    rng = np.random.default_rng(3)
    L, Hq, Hkv, d = lay.length, 4, 2, 16
    q, k, v = _bits(rng, (L, Hq, d)), _bits(rng, (L, Hkv, d)), _bits(rng, (L, Hkv, d))
    role, turn = lay.roles_and_turns()
    got = OA.prefill_request(q, k, v, role, turn)
    wide = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).double()  # torch's own widening
    qt = wide(q).permute(1, 0, 2)
    kt = wide(k).repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)
    vt = wide(v).repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True).permute(1, 0, 2).numpy()
    assert np.max(np.abs(got - ref)) < 1e-12


def test_softmax_rows_sum_to_one_and_zero_on_masked():
    rng = np.random.default_rng(5)
    lay = W.RequestLayout(5, [9, 4, 7], [3, 0, 5], 6)
    L, Hq, Hkv, d = lay.length, 2, 1, 8
    q, k = _bits(rng, (L, Hq, d), 3.0), _bits(rng, (L, Hkv, d), 3.0)
    role, turn = lay.roles_and_turns()
    vis = np.array(brute.brute_force_mask(role.tolist(), turn.tolist()))
    for h in range(Hq):
        P = OA.request_probs(q, k, role, turn, h)
        assert np.all(np.abs(P.sum(axis=1) - 1.0) < 1e-12)
        assert np.all(P[~vis] == 0.0)
        assert np.all(P[vis] > 0.0)


def test_zero_query_gives_mean_of_visible_values():
    rng = np.random.default_rng(9)
    lay = W.RequestLayout(3, [6, 5], [2, 3], 4)
    L, Hq, Hkv, d = lay.length, 4, 2, 8
    q = np.zeros((L, Hq, d), np.uint16)
    k, v = _bits(rng, (L, Hkv, d)), _bits(rng, (L, Hkv, d))
    role, turn = lay.roles_and_turns()
    got = OA.prefill_request(q, k, v, role, turn)
    vis = brute.brute_force_mask(role.tolist(), turn.tolist())
    vf = OA.bf16_bits_to_f64(v)
    for p in range(L):
        keys = [qq for qq in range(L) if vis[p][qq]]
        for h in range(Hq):
            want = sum(vf[qq, h // 2, :] for qq in keys) / len(keys)
            assert np.max(np.abs(got[p, h] - want)) < 1e-14


def test_gqa_equals_mha_with_repeated_kv_heads():
    rng = np.random.default_rng(13)
    lay = W.RequestLayout(4, [7, 3], [2, 2], 5)
    L, Hq, Hkv, d = lay.length, 6, 2, 8
    q, k, v = _bits(rng, (L, Hq, d)), _bits(rng, (L, Hkv, d)), _bits(rng, (L, Hkv, d))
    role, turn = lay.roles_and_turns()
    gqa = OA.prefill_request(q, k, v, role, turn)
    mha = OA.prefill_request(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), role, turn)
    assert np.array_equal(gqa, mha)


def test_row_subset_equals_full():
    rng = np.random.default_rng(17)
    lay = W.RequestLayout(6, [10, 8], [3, 4], 5)
    L, Hq, Hkv, d = lay.length, 2, 1, 8
    q, k, v = _bits(rng, (L, Hq, d)), _bits(rng, (L, Hkv, d)), _bits(rng, (L, Hkv, d))
    role, turn = lay.roles_and_turns()
    full = OA.prefill_request(q, k, v, role, turn, block=7)
    rows = [0, 5, 17, L - 1]
    sub = OA.prefill_request(q, k, v, role, turn, rows=rows)
    assert np.max(np.abs(full[rows] - sub)) < 1e-13  # BLAS may block the row sets differently


def test_bf16_widening_exact():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x7F7F, 0x0001, 0x3E80], dtype=np.uint16)
    want = [1.0, -2.0, 0.0, -0.0, 3.3895313892515355e38, 2.0 ** -133, 0.25]
    assert OA.bf16_bits_to_f64(bits).tolist() == want


def test_generator_bf16_rounding_matches_torch():
    x = np.random.default_rng(1).standard_normal(10000).astype(np.float32) * 7
    x = np.concatenate([x, np.array([1.00390625, 1.01171875, -1.00390625], np.float32)])  # ties
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


# ---------------------------------------------------------------------------
# compaction and decode
# ---------------------------------------------------------------------------
def _compact_one(lay, k, v, cap_extra=0):
    role, turn = lay.roles_and_turns()
    cap = lay.system + sum(lay.nexus) + lay.current + cap_extra
    Hkv, d = k.shape[1], k.shape[2]
    kc = np.full((max(cap, 1), Hkv, d), 0xFFFF, np.uint16)
    vc = np.full((max(cap, 1), Hkv, d), 0xFFFF, np.uint16)
    ki = np.full(max(cap, 1), -7, np.int32)
    n = OC.compact_batch(k, v, role, np.array([0, lay.length]), [0], [cap], kc, vc, ki)
    return role, turn, kc, vc, ki, int(n[0])


def test_compaction_closed_forms():
    rng = np.random.default_rng(21)
    for _ in range(40):
        lay = W.random_layout(rng)
        L = lay.length
        k, v = _bits(rng, (L, 2, 4)), _bits(rng, (L, 2, 4))
        role, turn, kc, vc, ki, n = _compact_one(lay, k, v, cap_extra=3)
        assert n == lay.system + sum(lay.nexus) + lay.current
        assert L - n == sum(lay.bodies)
        keep = ki[:n]
        assert np.all(np.diff(keep) > 0)
        assert np.all(role[keep] != OL.HISTORY_TEXT)
        assert np.array_equal(kc[:n], k[keep]) and np.array_equal(vc[:n], v[keep])
        assert np.all(kc[n:] == 0xFFFF) and np.all(ki[n:] == -7)


def test_compaction_capacity_overflow():
    lay = W.RequestLayout(2, [3], [2], 2)
    role, turn = lay.roles_and_turns()
    k = np.zeros((lay.length, 1, 2), np.uint16)
    with pytest.raises(OverflowError):
        OC.compact_batch(k, k, role, np.array([0, lay.length]), [0], [5], np.zeros((5, 1, 2), np.uint16),
                         np.zeros((5, 1, 2), np.uint16), np.zeros(5, np.int32))


def test_compact_decode_equals_masked_full_decode():
    rng = np.random.default_rng(23)
    for _ in range(25):
        lay = W.random_layout(rng)
        L, Hq, Hkv, d = lay.length, 4, 2, 16
        k, v = _bits(rng, (L, Hkv, d), 2.0), _bits(rng, (L, Hkv, d))
        role, turn, kc, vc, ki, n = _compact_one(lay, k, v)
        q1, k1, v1 = _bits(rng, (Hq, d), 2.0), _bits(rng, (Hkv, d), 2.0), _bits(rng, (Hkv, d))
        a = OD.decode_step(q1, kc[:n], vc[:n], k1, v1)
        b = OD.masked_decode_step(q1, k, v, role, k1, v1)
        assert np.max(np.abs(a - b)) <= 1e-12 * max(1.0, np.max(np.abs(b)))


def test_prefill_last_current_row_equals_compact_decode():
    rng = np.random.default_rng(29)
    for _ in range(10):
        lay = W.random_layout(rng)
        lay.current = max(lay.current, 1)
        L, Hq, Hkv, d = lay.length, 4, 2, 16
        q, k, v = _bits(rng, (L, Hq, d)), _bits(rng, (L, Hkv, d)), _bits(rng, (L, Hkv, d))
        role, turn, kc, vc, ki, n = _compact_one(lay, k, v)
        pre = OA.prefill_request(q, k, v, role, turn, rows=[L - 1])[0]
        dec = OD.decode_step(q[L - 1], kc[:n - 1], vc[:n - 1], kc[n - 1], vc[n - 1])
        assert np.max(np.abs(pre - dec)) < 1e-12


def test_decode_run_matches_stepwise_cache_growth():
    rng = np.random.default_rng(31)
    n, Hq, Hkv, d, T = 9, 4, 2, 8, 5
    kc, vc = _bits(rng, (n, Hkv, d)), _bits(rng, (n, Hkv, d))
    qs, ks, vs = _bits(rng, (T, Hq, d)), _bits(rng, (T, Hkv, d)), _bits(rng, (T, Hkv, d))
    run = OD.decode_run(qs, ks, vs, kc, vc)
    for t in range(T):
        want = OD.decode_step(qs[t], np.concatenate([kc, ks[:t]]), np.concatenate([vc, vs[:t]]), ks[t], vs[t])
        assert np.array_equal(run[t], want)


def test_decode_single_row_context_returns_that_value():
    # with only the appended row visible, softmax puts all mass on it
    rng = np.random.default_rng(37)
    Hq, Hkv, d = 4, 2, 8
    q1, k1, v1 = _bits(rng, (Hq, d)), _bits(rng, (Hkv, d)), _bits(rng, (Hkv, d))
    out = OD.decode_step(q1, np.zeros((0, Hkv, d), np.uint16), np.zeros((0, Hkv, d), np.uint16), k1, v1)
    vf = OA.bf16_bits_to_f64(v1)
    assert np.array_equal(out, vf[[0, 0, 1, 1]])
