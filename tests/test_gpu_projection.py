"""Role-routed projection on the GPU against the fp64 oracle.

Each output is a sum of K exact bf16 products accumulated in fp32, so it is
checked against |err| <= 2 * K * 2^-24 * sum_k |x_k w_k| + 1e-6 (the classic
bound for recursive fp32 summation, with a factor of 2 to spare): the bound
scales with the terms, so it is tight for every row whatever its magnitude.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import layout as OL
from oracle import projection as OP
from oracle.attention import bf16_bits_to_f64
from paper_2601_21927_amd import sonic
from paper_2601_21927_amd.runner import bf16_to_device
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu


def _bits(rng, shape, scale=1.0):
    return W.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def run(role, x, wt, wn):
    H.need_gpu()
    T, K = x.shape
    N = wt.shape[0]
    y = torch.full((max(T, 1), N), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(sonic.role_projection_workspace_bytes(T), 256), dtype=torch.uint8, device="cuda")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    r = torch.from_numpy(np.ascontiguousarray(role, np.uint8)).cuda()
    st = sonic.role_projection(r, bf16_to_device(x), bf16_to_device(wt), bf16_to_device(wn), y[:T] if T else y[:0],
                               ws, status)
    torch.cuda.synchronize()
    assert st == sonic.OK, sonic.status_string(st)
    assert int(status.item()) == 0
    return y[:T].cpu().numpy()


def check(got, role, x, wt, wn, what, rows=None):
    rows = np.arange(len(role)) if rows is None else rows
    want = OP.role_routed_linear(x[rows], role[rows], wt, wn)
    xf, wtf, wnf = bf16_bits_to_f64(x[rows]), bf16_bits_to_f64(wt), bf16_bits_to_f64(wn)
    mag = np.where((role[rows] == OL.NEXUS)[:, None], np.abs(xf) @ np.abs(wnf).T, np.abs(xf) @ np.abs(wtf).T)
    K = x.shape[1]
    err = np.abs(got[rows] - want)
    bound = 2 * K * 2.0 ** -24 * mag + 1e-6
    H.note(f"  {what}: max_abs={err.max() if err.size else 0:.3e} worst err/bound="
           f"{(err / bound).max() if err.size else 0:.3f} n={err.size}")
    assert np.all(np.isfinite(got[rows])), what
    assert np.all(err <= bound), what


def _roles(rng, T):
    lays = []
    while sum(l.length for l in lays) < T:
        lays.append(W.random_layout(rng, max_h=4, max_b=60, max_k=30, max_s=20, max_c=20))
    role = np.concatenate([l.roles_and_turns()[0] for l in lays])[:T]
    return role


@pytest.mark.parametrize("T,K,N", [(1, 64, 1), (37, 64, 5), (300, 128, 128), (1000, 192, 300),
                                   (2500, 512, 257), (129, 4096, 130)])
def test_projection_random(T, K, N):
    rng = np.random.default_rng(T + K + N)
    role = _roles(rng, T)
    x, wt, wn = _bits(rng, (T, K)), _bits(rng, (N, K), 0.05), _bits(rng, (N, K), 0.05)
    got = run(role, x, wt, wn)
    check(got, role, x, wt, wn, f"T={T} K={K} N={N} nexus={int((role == OL.NEXUS).sum())}")


@pytest.mark.parametrize("which", ["all_text", "all_nexus", "alternating", "tile_edges"])
def test_projection_role_patterns(which):
    rng = np.random.default_rng(17)
    T, K, N = 515, 128, 200
    if which == "all_text":
        role = np.full(T, OL.CURRENT, np.uint8)
    elif which == "all_nexus":
        role = np.full(T, OL.NEXUS, np.uint8)
    elif which == "alternating":
        role = np.where(np.arange(T) % 2 == 0, OL.NEXUS, OL.HISTORY_TEXT).astype(np.uint8)
    else:   # exactly 128 Nexus rows, then 128 + 1 text rows, ...
        role = np.where((np.arange(T) // 128) % 2 == 0, OL.NEXUS, OL.SYSTEM).astype(np.uint8)
    x, wt, wn = _bits(rng, (T, K)), _bits(rng, (N, K), 0.1), _bits(rng, (N, K), 0.1)
    check(run(role, x, wt, wn), role, x, wt, wn, which)


def test_projection_one_hot_routing():
    """x[t] = e_k: y[t] is column k of the weight set of row t's role, exactly."""
    rng = np.random.default_rng(23)
    T, K, N = 700, 64, 150
    role = _roles(rng, T)
    wt, wn = _bits(rng, (N, K)), _bits(rng, (N, K))
    x = np.zeros((T, K), np.uint16)
    cols = rng.integers(0, K, T)
    x[np.arange(T), cols] = 0x3F80
    got = run(role, x, wt, wn)
    want = np.where((role == OL.NEXUS)[:, None], bf16_bits_to_f64(wn)[:, cols].T, bf16_bits_to_f64(wt)[:, cols].T)
    assert np.array_equal(got, want)


def test_projection_llama3_8b_qkv_shape_rows():
    """One request of the 8B-shaped workload through the fused QKV projection: K = 4096,
    N = 4096 + 2 * 1024; sampled rows of both roles."""
    rng = np.random.default_rng(29)
    lay = W.workload_structure(2)["layouts"][0]
    role, _ = lay.roles_and_turns()
    T, K, N = len(role), 4096, 6144
    x, wt, wn = _bits(rng, (T, K)), _bits(rng, (N, K), 0.02), _bits(rng, (N, K), 0.02)
    got = run(role, x, wt, wn)
    rows = np.unique(np.concatenate([rng.integers(0, T, 48), np.nonzero(role == OL.NEXUS)[0][::40]]))
    check(got, role, x, wt, wn, "8B qkv", rows)


def test_projection_argument_errors():
    H.need_gpu()
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    st0 = torch.zeros(1, dtype=torch.int32, device="cuda")
    role = torch.zeros(10, dtype=torch.uint8, device="cuda")
    x = torch.zeros((10, 96), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 96), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((10, 8), dtype=torch.float32, device="cuda")
    assert sonic.role_projection(role, x, w, w, y, ws, st0) == sonic.ERR_UNSUPPORTED   # K not a multiple of 64
    x = torch.zeros((10, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda")
    assert sonic.role_projection(role, x, w, w, y, ws[:16], st0) == sonic.ERR_WORKSPACE
