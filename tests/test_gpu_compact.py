"""KV compaction on the GPU: bit-exact against the oracle (keep_idx, lengths, cache bytes)."""
import numpy as np
import pytest
import torch

import workloads as W
from paper_2601_21927_amd import sonic
from paper_2601_21927_amd.runner import bf16_to_host
from tests import gpu_helpers as H

pytestmark = pytest.mark.gpu


def run_compact(batch, caps):
    H.need_gpu()
    db = H.device_batch(batch)
    cache = db.alloc_cache(caps)
    st = db.compact()
    assert st == sonic.OK, sonic.status_string(st)
    torch.cuda.synchronize()
    return db, cache


def check_bit_exact(batch, caps):
    db, cache = run_compact(batch, caps)
    assert db.read_status() == 0, sonic.status_string(db.read_status())
    kc, vc, ki, n, off = H.oracle_compact(batch, caps)
    assert np.array_equal(cache.length.cpu().numpy(), n)
    assert np.array_equal(cache.keep_idx.cpu().numpy(), ki)
    assert np.array_equal(bf16_to_host(cache.k), kc)
    assert np.array_equal(bf16_to_host(cache.v), vc)
    H.note(f"  compaction {batch.name}: bit-exact, kept {int(n.sum())} of {batch.total_tokens} rows")


@pytest.mark.parametrize("seed,Hkv,d", [(1, 2, 64), (2, 8, 128), (3, 1, 128), (4, 4, 64)])
def test_compact_random_layouts(seed, Hkv, d):
    rng = np.random.default_rng(seed)
    lays = [W.random_layout(rng, max_h=5, max_b=900, max_k=300, max_s=600, max_c=500) for _ in range(7)]
    lays.append(W.RequestLayout(0, [], [], 0))
    lays.append(W.RequestLayout(0, [5000], [0], 0))     # nothing kept
    batch = W.make_batch("random", lays, Hkv, Hkv, d, seed=seed)
    caps = H.kept_counts(batch) + rng.integers(0, 40, size=len(lays))
    check_bit_exact(batch, caps)


@pytest.mark.parametrize("idx", [1, 2, 3, 4, 5])
def test_compact_workloads(idx):
    batch = W.workload(idx, decode_steps=0)
    H.note(f"compaction workload {idx}: B={batch.batch} T={batch.total_tokens}")
    caps = H.kept_counts(batch) + 3
    check_bit_exact(batch, caps)


def test_compact_repeatable():
    rng = np.random.default_rng(9)
    lays = [W.random_layout(rng, max_h=6, max_b=700, max_k=200, max_s=300, max_c=300) for _ in range(5)]
    batch = W.make_batch("rep", lays, 4, 4, 128, seed=9)
    caps = H.kept_counts(batch)
    db, cache = run_compact(batch, caps)
    first = (bf16_to_host(cache.k).copy(), cache.keep_idx.cpu().numpy().copy())
    for _ in range(3):
        cache.k.view(torch.int16).fill_(0)
        cache.keep_idx.fill_(-1)
        assert db.compact() == sonic.OK
        torch.cuda.synchronize()
        assert np.array_equal(bf16_to_host(cache.k), first[0])
        assert np.array_equal(cache.keep_idx.cpu().numpy(), first[1])


def test_compact_capacity_overflow_stays_inside_capacity():
    lays = [W.RequestLayout(40, [100], [30], 20), W.RequestLayout(10, [50], [5], 5)]
    batch = W.make_batch("cap", lays, 2, 2, 64, seed=5)
    kept = H.kept_counts(batch)
    caps = np.array([kept[0] - 7, kept[1]])
    db, cache = run_compact(batch, caps)
    assert db.read_status() == sonic.ERR_CAPACITY
    assert cache.length.cpu().numpy()[0] == 0          # the overflowing request gets no length
    # every row of request 1 is either untouched or exactly its own kept row: request 0's
    # overflow never spills into it
    k = bf16_to_host(cache.k)
    kc, _, _, _, _ = H.oracle_compact(batch, kept)
    start1 = int(caps[0])
    for j in range(int(caps[1])):
        row = k[start1 + j]
        assert np.all(row == 0xFFFF) or np.array_equal(row, kc[int(kept[0]) + j]), j


def test_compact_understated_max_seqlen_is_an_error_and_writes_nothing():
    """The grid is sized from max_seqlen; a longer request raises INVALID_ARG and none of its rows is
    written."""
    lays = [W.RequestLayout(300, [900], [200], 1200), W.RequestLayout(10, [50], [5], 5)]
    batch = W.make_batch("maxlen", lays, 2, 2, 64, seed=6)
    caps = H.kept_counts(batch)
    H.need_gpu()
    db = H.device_batch(batch)
    cache = db.alloc_cache(caps)
    st = sonic.kv_compact(db.cu, db.role, db.k, db.v, cache.k, cache.v, cache.row_off, cache.row_cap, cache.length,
                          cache.keep_idx, db.status, max_seqlen=1024)
    assert st == sonic.OK
    torch.cuda.synchronize()
    assert db.read_status() == sonic.ERR_INVALID_ARG
    k = bf16_to_host(cache.k)
    assert np.all(k[:int(caps[0])] == 0xFFFF)
    assert np.all(cache.keep_idx.cpu().numpy()[:int(caps[0])] == -1)
    assert cache.length.cpu().numpy()[0] == 0
