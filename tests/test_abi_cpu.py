"""The C-ABI library on the CPU: it loads, exports every declared symbol, and its
host-side helpers agree with the oracle.  No GPU call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

import workloads as W
from oracle import layout as OL
from oracle import mask as OM
from paper_2601_21927_amd import sonic
from tests import brute

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "sonic.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sonic_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 9
    L = sonic.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(sonic.EXPORTS)


def test_abi_version_and_status_strings():
    assert sonic.abi_version() == 10
    assert sonic.status_string(0) == "ok"
    for code in range(1, 7):
        assert sonic.status_string(code) != "unknown status"
    assert sonic.status_string(99) == "unknown status"


def _pack(lays):
    role, turn, cu = W.pack_layouts(lays)
    return cu, role, turn


def test_host_validation_accepts_generated_layouts():
    rng = np.random.default_rng(61)
    lays = [W.random_layout(rng) for _ in range(50)] + [W.RequestLayout(0, [], [], 0)]
    cu, role, turn = _pack(lays)
    st, bad = sonic.validate_layout_host(cu, role, turn)
    assert st == sonic.OK


@pytest.mark.parametrize("roles,turns", [
    ([2, 2], [1, 1]), ([0, 2], [0, 1]), ([1, 0], [1, 0]), ([3, 1], [2, 1]), ([1, 2, 2], [1, 1, 2]),
    ([1, 1], [2, 1]), ([1, 2, 1], [1, 1, 1]), ([0, 4], [0, 0]), ([3, 2], [1, 1]),
])
def test_host_validation_rejects_like_the_oracle(roles, turns):
    with pytest.raises(OL.LayoutError):
        OL.parse(np.array(roles), np.array(turns))
    good = W.RequestLayout(2, [3], [1], 2)
    r0, t0 = good.roles_and_turns()
    role = np.concatenate([r0, np.array(roles, np.uint8)])
    turn = np.concatenate([t0, np.array(turns, np.int32)])
    cu = np.array([0, good.length, good.length + len(roles)], np.int32)
    st, bad = sonic.validate_layout_host(cu, role, turn)
    assert st == sonic.ERR_BAD_LAYOUT and bad == 1


def test_host_validation_random_mutations_agree_with_oracle():
    rng = np.random.default_rng(67)
    for _ in range(300):
        lay = W.random_layout(rng, max_h=3, max_b=4, max_k=3, max_s=3, max_c=3)
        role, turn = lay.roles_and_turns()
        if len(role) == 0:
            continue
        i = int(rng.integers(0, len(role)))
        role = role.copy()
        turn = turn.copy()
        if rng.random() < 0.5:
            role[i] = rng.integers(0, 4)
        else:
            turn[i] += int(rng.integers(-2, 3))
        try:
            OL.parse(role, turn)
            want = sonic.OK
        except OL.LayoutError:
            want = sonic.ERR_BAD_LAYOUT
        st, _ = sonic.validate_layout_host(np.array([0, len(role)], np.int32), role, turn)
        assert st == want, (role.tolist(), turn.tolist())


def test_layout_stats_match_oracle_mask_counts():
    rng = np.random.default_rng(71)
    lays = [W.random_layout(rng) for _ in range(40)]
    cu, role, turn = _pack(lays)
    vis, kept = sonic.layout_stats_host(cu, role, turn)
    for b, lay in enumerate(lays):
        r, t = lay.roles_and_turns()
        assert vis[b] == int(OM.visibility(r, t).sum())
        assert kept[b] == int(np.sum(r != OL.HISTORY_TEXT))


def test_layout_stats_up_to_own_scope_match_oracle_mask_counts():
    rng = np.random.default_rng(73)
    lays = [W.random_layout(rng) for _ in range(40)]
    cu, role, turn = _pack(lays)
    vis, _ = sonic.layout_stats_host(cu, role, turn, sonic.NEXUS_UP_TO_OWN)
    for b, lay in enumerate(lays):
        r, t = lay.roles_and_turns()
        assert vis[b] == int(OM.visibility(r, t, OM.NEXUS_UP_TO_OWN).sum())
    with pytest.raises(sonic.SonicError):
        sonic.layout_stats_host(cu, role, turn, 7)


@pytest.mark.parametrize("idx,pairs", [(1, 50736), (2, 5194240), (4, 193692160)])
def test_layout_stats_on_workloads(idx, pairs):
    st = W.workload_structure(idx)
    cu, role, turn = _pack(st["layouts"])
    vis, kept = sonic.layout_stats_host(cu, role, turn)
    assert np.all(vis == pairs)
    lay = st["layouts"][0]
    assert np.all(kept == lay.system + sum(lay.nexus) + lay.current)


def test_workspace_sizes():
    # plan (44 B per token) plus the prefix copies of K and V (Hkv * d * 4 B per token)
    # plan (44 B per token), K/V prefix copies, softmax normalisers and key-weight partials
    assert sonic.prefill_workspace_bytes(8, 43392, 32, 8, 128) >= 43392 * (44 + 8 * 128 * 4 + (32 + 8) * 4)
    assert sonic.prefill_workspace_bytes(0, 0, 1, 1, 64) > 0
    assert sonic.prefill_workspace_bytes(1, 10, 4, 0, 64) == 0
    assert sonic.prefill_workspace_bytes(1, 10, 0, 2, 64) == 0
    assert sonic.decode_workspace_bytes(8, 32, 128, 1584) >= 8 * 32 * 130 * 4
    # enough for every kv-head count dividing Hq: with 128 requests and 2 kv-heads there are 256
    # (request, kv-head) pairs, which take three splits at contexts of 2048 rows and more
    assert sonic.decode_workspace_bytes(128, 8, 128, 4096) >= 128 * 8 * 3 * 130 * 4


def test_softmax_scale_argument_checks_without_gpu():
    """softmax_scale = 0 selects 1/sqrt(d) inside the C ABI; a negative or non-finite scale is an
    argument error.  An empty batch returns before any GPU call, so this runs on the CPU."""
    L = sonic.lib()
    st = ctypes.c_int32(0)
    sp = ctypes.byref(st)
    n = None

    def prefill(scale):
        return L.sonic_segment_attn_prefill(0, 0, 4, 2, 64, n, n, n, n, n, n, scale, 0, n, n, n, n, 0, sp, n)

    def decode(scale):
        return L.sonic_compressed_decode(0, 4, 2, 64, 16, n, n, n, n, n, n, n, n, n, scale, n, n, 0, sp, n)

    def extend(scale):
        return L.sonic_nexus_extend(0, 0, 4, 2, 64, 16, n, n, n, n, n, n, n, n, n, n, n, scale, n, n, 0, sp, n)

    for call in (prefill, decode, extend):
        assert call(0.0) == sonic.OK
        assert call(-0.0) == sonic.OK
        assert call(0.125) == sonic.OK
        assert call(-0.125) == sonic.ERR_INVALID_ARG
        assert call(float("nan")) == sonic.ERR_INVALID_ARG
        assert call(float("inf")) == sonic.ERR_INVALID_ARG
    assert st.value == 0
