"""Benchmark of the SONIC hot path on one MI355X.

One step = the whole path over one batch of the Llama-3-8B-shaped workload
(B=8, 32/8 heads, d=128, 256 system + 8 x (512 text + 102 Nexus) + 256 current
tokens per request): masked prefill, KV compaction, then 256 decode steps
over the compacted cache.  Inputs are synthetic (seeded bf16 N(0,1)) and
resident in HBM before the timed region.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline] [--no-graph]

Prints one JSON line.  value = generated tokens per second of the whole step
(B x 256 decode tokens / step time, the step including its prefill and
compaction).  Per-phase figures, the roofline of the dominant kernel and the
fp64 CPU oracle's rate on a bounded sample of the same work are attached.
After the timed region, the next-turn Nexus step (the finished turn becomes a
history segment whose Nexus rows attend to the whole cache) is timed on its
own; it is reported as a phase and is not part of value.
"""
from __future__ import annotations

import argparse
import hashlib
import glob
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "masked-prefill visible TFLOP/s; compressed-decode tok/s; % of MFMA/HBM peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_2601_21927_amd", "csrc", "*"))):
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter runs, if they were taken
    on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    data = json.load(open(path))
    ent = data.get(kernel)
    if not ent or ent.get("source_hash") != kernel_source_hash():
        return None
    return ent.get("bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying a HIP graph")
    ap.add_argument("--decode-steps", type=int, default=256)
    ap.add_argument("--decode-workloads", type=lambda v: [int(x) for x in v.split(",") if x], default=[],
                    help="also time the compressed decode loop of these workloads (e.g. 3,4,5)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import workloads as W
    from paper_2601_21927_amd import sonic
    from paper_2601_21927_amd.runner import SonicBatch, CompactCache, bf16_to_device

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    sonic.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    batch = W.workload(2, decode_steps=args.decode_steps)
    B, Hq, Hkv, d = batch.batch, batch.num_q_heads, batch.num_kv_heads, batch.head_dim
    steps_dec = batch.decode_steps
    vis_pairs, kept = sonic.layout_stats_host(batch.cu_seqlens, batch.role, batch.turn_id)
    visible_flops = float(4 * d * Hq * vis_pairs.sum())

    db = SonicBatch(batch.role, batch.turn_id, batch.cu_seqlens, batch.q, batch.k, batch.v, device=dev)
    caps = kept.astype(np.int64) + steps_dec
    cache = db.alloc_cache(caps)
    max_ctx = int(caps.max())
    dq = bf16_to_device(batch.dec_q, dev)
    dk = bf16_to_device(batch.dec_k, dev)
    dv = bf16_to_device(batch.dec_v, dev)
    dec_out = torch.empty((B, Hq, d), dtype=torch.float32, device=dev)
    # allocate the decode workspace outside the timed region
    assert cache.decode(dq[0], dk[0], dv[0], dec_out, db.status, max_ctx) == sonic.OK
    torch.cuda.synchronize()

    # full-context baseline: the same conversations without Nexus tokens, every row visible
    text_lays = [W.text_only_layout(l) for l in batch.layouts]
    full_rows = np.array([l.length for l in text_lays], np.int64)
    full = CompactCache(int((full_rows + steps_dec).sum()), Hkv, d,
                        np.concatenate([[0], np.cumsum(full_rows + steps_dec)[:-1]]),
                        (full_rows + steps_dec).astype(np.int32), dev)
    keep_text = batch.role != W.ROLE_NEXUS
    kt, vt = batch.k[keep_text], batch.v[keep_text]
    fk = np.zeros((full.rows, Hkv, d), np.uint16)
    fv = np.zeros_like(fk)
    src = 0
    for b in range(B):
        o, n = int(full.row_off_host[b]), int(full_rows[b])
        fk[o:o + n], fv[o:o + n] = kt[src:src + n], vt[src:src + n]
        src += n
    full.k.copy_(bf16_to_device(fk, dev))
    full.v.copy_(bf16_to_device(fv, dev))
    full_len0 = torch.from_numpy(full_rows.astype(np.int32)).to(dev)
    full.length.copy_(full_len0)
    assert full.decode(dq[0], dk[0], dv[0], dec_out, db.status, int(full.row_cap_host.max())) == sonic.OK
    torch.cuda.synchronize()
    del fk, fv, kt, vt

    stream = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def run_prefill():
        st = db.prefill()
        assert st == sonic.OK, sonic.status_string(st)

    def run_compact():
        st = db.compact()
        assert st == sonic.OK, sonic.status_string(st)

    full_max_ctx = int(full.row_cap_host.max())

    def run_decode_loop(c: CompactCache):
        mc = max_ctx if c is cache else full_max_ctx
        for t in range(steps_dec):
            st = c.decode(dq[t], dk[t], dv[t], dec_out, db.status, mc)
            assert st == sonic.OK, sonic.status_string(st)

    phases = {"prefill": run_prefill, "compact": run_compact, "decode": lambda: run_decode_loop(cache)}
    for _ in range(max(1, args.warmup)):
        for f in phases.values():
            f()
    torch.cuda.synchronize()
    use_graph = not args.no_graph
    graphs = {}
    if use_graph:
        # the step as one HIP graph (prefill, compaction, the 256 decode calls); and one
        # graph per phase, replayed apart to split a step's time into its phases
        for name, f in phases.items():
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                f()
            graphs[name] = g
        step_graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(step_graph):
            for f in phases.values():
                f()
        torch.cuda.synchronize()
        full_graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(full_graph):
            run_decode_loop(full)
        torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def step(marks=None):
        if marks: marks[0].record(stream)
        if use_graph:
            step_graph.replay()
        else:
            for f in phases.values():
                f()
        if marks: marks[1].record(stream)

    def phase_split(marks):
        for i, name in enumerate(("prefill", "compact", "decode")):
            marks[i].record(stream)
            if use_graph:
                graphs[name].replay()
            else:
                phases[name]()
        marks[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    assert db.read_status() == 0, sonic.status_string(db.read_status())

    # ---- timed region: exactly K steps ----
    all_marks = [[ev() for _ in range(2)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(all_marks[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert db.read_status() == 0, sonic.status_string(db.read_status())
    ms_per_step = wall * 1e3 / args.steps
    step_ms_ev = float(np.median([m[0].elapsed_time(m[1]) for m in all_marks]))

    # ---- the phases of a step, each replayed as its own graph (after the timed region) ----
    split_marks = [[ev() for _ in range(4)] for _ in range(max(3, args.steps))]
    for m in split_marks:
        phase_split(m)
    torch.cuda.synchronize()
    assert db.read_status() == 0, sonic.status_string(db.read_status())
    med = lambda i, j: float(np.median([m[i].elapsed_time(m[j]) for m in split_marks]))
    pf_ms, cp_ms, dc_ms = med(0, 1), med(1, 2), med(2, 3)

    # ---- back-to-back launches of the two single-launch phases (no graph-launch gap
    # between phases): their per-launch rate ----
    def back_to_back(f, n):
        if use_graph:   # n calls in one graph, so no graph launch separates them
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for _ in range(n):
                    phases[f]()
            torch.cuda.synchronize()
        a, b_ = ev(), ev()
        a.record(stream)
        if use_graph:
            g.replay()
        else:
            for _ in range(n):
                phases[f]()
        b_.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b_) / n
    pf_b2b_ms = back_to_back("prefill", 10)
    # the same prefill with both attention statistics (Nexus mass per row and head, key weights)
    stat_mass = torch.empty((batch.total_tokens, Hq), dtype=torch.float32, device=dev)
    stat_w = torch.empty((batch.total_tokens,), dtype=torch.float32, device=dev)

    def run_prefill_stats():
        st = db.prefill(nexus_mass=stat_mass, key_weight=stat_w)
        assert st == sonic.OK, sonic.status_string(st)
    phases["prefill_stats"] = run_prefill_stats
    run_prefill_stats()
    torch.cuda.synchronize()
    pfs_b2b_ms = back_to_back("prefill_stats", 10)
    cp_b2b_ms = back_to_back("compact", 20)
    assert db.read_status() == 0

    # ---- cold single launches: a 1 GiB write before each launch evicts the 256 MB
    # Infinity Cache, so the kernel reads its inputs from HBM ----
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)

    def cold(f, pre=None, n=9):
        ts = []
        for i in range(n):
            if pre is not None:
                pre()
            flush.fill_(float(i))
            a, b_ = ev(), ev()
            a.record(stream)
            f()
            b_.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b_))
        return float(np.median(ts))
    cp_cold_ms = cold(run_compact)

    def one_decode():
        st = cache.decode(dq[0], dk[0], dv[0], dec_out, db.status, max_ctx)
        assert st == sonic.OK, sonic.status_string(st)
    dc_cold_ms = cold(one_decode, pre=run_compact)   # each call from the freshly compacted cache
    assert db.read_status() == 0
    del flush
    # bytes of one decode call from the compacted cache: its rows plus the appended one
    dec1_bytes = float((np.asarray(kept, np.float64) + 1).sum() * Hkv * d * 2 * 2)

    # ---- full-context decode (same kernel, text-only cache) for the speedup ----
    fms = []
    for _ in range(3):
        full.length.copy_(full_len0)
        a, b_ = ev(), ev()
        a.record(stream)
        if use_graph:
            full_graph.replay()
        else:
            run_decode_loop(full)
        b_.record(stream)
        torch.cuda.synchronize()
        fms.append(a.elapsed_time(b_))
    full_ms = float(np.median(fms))
    assert db.read_status() == 0

    # ---- next-turn Nexus step: the turn that just ended (C query rows + the decoded rows)
    # becomes segment h+1; its K Nexus rows attend to the whole cache, then replace the
    # turn's rows.  The decode loop left those rows at kept..kept+steps of every request.
    cu = batch.cu_seqlens
    ext_keep_np = np.array([l.system + sum(l.nexus) for l in batch.layouts], np.int32)
    ext_len_np = (kept + steps_dec).astype(np.int32)
    npos = []   # the last segment's Nexus rows serve as the new segment's inputs
    for b, l in enumerate(batch.layouts):
        p0 = int(cu[b]) + l.system + sum(l.bodies) + sum(l.nexus[:-1])
        npos.append(np.arange(p0, p0 + l.nexus[-1]))
    kn_np = np.array([len(x) for x in npos], np.int64)
    allpos = np.concatenate(npos)
    ext_cu = torch.from_numpy(np.concatenate([[0], np.cumsum(kn_np)]).astype(np.int32)).to(dev)
    ext_keep = torch.from_numpy(ext_keep_np).to(dev)
    ext_len0 = torch.from_numpy(ext_len_np).to(dev)
    ext_len = ext_len0.clone()
    ext_k, ext_v = cache.k.clone(), cache.v.clone()
    eq, ek, e_v = (bf16_to_device(x[allpos], dev) for x in (batch.q, batch.k, batch.v))
    ext_out = torch.empty((len(allpos), Hq, d), dtype=torch.float32, device=dev)
    ext_ws = torch.empty(max(sonic.nexus_extend_workspace_bytes(B, len(allpos)), 256), dtype=torch.uint8,
                         device=dev)

    def run_extend():
        st = sonic.nexus_extend(ext_cu, ext_keep, ext_k, ext_v, cache.row_off, cache.row_cap, ext_len, eq, ek, e_v,
                                ext_out, ext_ws, db.status, max_rows=max_ctx)
        assert st == sonic.OK, sonic.status_string(st)

    run_extend()
    torch.cuda.synchronize()
    if use_graph:
        ext_graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(ext_graph):
            run_extend()
        torch.cuda.synchronize()
    xms = []
    for _ in range(20):
        ext_len.copy_(ext_len0)     # the step consumes the turn's rows: start again from them
        a, b_ = ev(), ev()
        a.record(stream)
        if use_graph:
            ext_graph.replay()
        else:
            run_extend()
        b_.record(stream)
        torch.cuda.synchronize()
        xms.append(a.elapsed_time(b_))
    ext_ms = float(np.median(xms))
    assert db.read_status() == 0, sonic.status_string(db.read_status())
    assert np.array_equal(ext_len.cpu().numpy(), ext_keep_np + kn_np)
    ext_flops = float(4 * d * Hq * np.sum(kn_np * (ext_len_np + kn_np)))

    # ---- role-routed projection: the fused QKV product of the 8B shape over the whole batch,
    # Nexus rows with their own weight set (K = 4096 model width, N = 4096 + 2 x 1024) ----
    pj_K, pj_N = 4096, Hq * d + 2 * Hkv * d
    gen = torch.Generator(device=dev).manual_seed(11)
    pj_x = torch.randn((batch.total_tokens, pj_K), generator=gen, device=dev).to(torch.bfloat16)
    pj_wt = (torch.randn((pj_N, pj_K), generator=gen, device=dev) * 0.02).to(torch.bfloat16)
    pj_wn = (torch.randn((pj_N, pj_K), generator=gen, device=dev) * 0.02).to(torch.bfloat16)
    pj_y = torch.empty((batch.total_tokens, pj_N), dtype=torch.float32, device=dev)
    pj_ws = torch.empty(sonic.role_projection_workspace_bytes(batch.total_tokens), dtype=torch.uint8, device=dev)

    def run_projection():
        st = sonic.role_projection(db.role, pj_x, pj_wt, pj_wn, pj_y, pj_ws, db.status)
        assert st == sonic.OK, sonic.status_string(st)
    phases["projection"] = run_projection
    run_projection()
    torch.cuda.synchronize()
    pj_ms = back_to_back("projection", 5)
    pj_flops = 2.0 * batch.total_tokens * pj_K * pj_N
    assert db.read_status() == 0
    del pj_x, pj_y

    # ---- reconstruction targets of the whole batch, hidden size 4096 (training side) ----
    rc_Dm = 4096
    rc_h = torch.randn((batch.total_tokens, rc_Dm), generator=gen, device=dev).to(torch.bfloat16)
    rc_n = int((batch.role == W.ROLE_NEXUS).sum())
    rc_t = torch.empty((rc_n, rc_Dm), dtype=torch.float32, device=dev)
    rc_c = torch.empty((rc_n,), dtype=torch.float32, device=dev)
    rc_r = torch.empty((rc_n,), dtype=torch.float32, device=dev)
    rc_ws = torch.empty(sonic.nexus_recon_workspace_bytes(B, batch.total_tokens), dtype=torch.uint8, device=dev)

    def run_recon():
        st = sonic.nexus_recon_targets(db.cu, db.role, db.turn_id, rc_h, rc_t, rc_c, rc_r, rc_ws, db.status)
        assert st == sonic.OK, sonic.status_string(st)
    phases["recon"] = run_recon
    run_recon()
    torch.cuda.synchronize()
    rc_ms = back_to_back("recon", 10)
    assert db.read_status() == 0
    body_rows = sum(sum(l.bodies[i] for i in range(len(l.bodies)) if l.nexus[i] > 0) for l in batch.layouts)
    rc_bytes = float(body_rows + rc_n) * rc_Dm * 2 + rc_n * (rc_Dm * 4 + 8)
    del rc_h

    # ---- optional: the compressed decode loop of other workloads (their whole step count,
    # one graph, from the freshly compacted cache) ----
    dec_other = {}
    for wl in args.decode_workloads:
        ob = W.workload(wl)
        odb = SonicBatch(ob.role, ob.turn_id, ob.cu_seqlens, None, ob.k, ob.v, device=dev)
        okept = np.array([l.system + sum(l.nexus) + l.current for l in ob.layouts], np.int64)
        ost = ob.decode_steps
        oc = odb.alloc_cache(okept + ost)
        omc = int((okept + ost).max())
        oq, okn, ovn = (bf16_to_device(x, dev) for x in (ob.dec_q, ob.dec_k, ob.dec_v))
        oout = torch.empty((ob.batch, ob.num_q_heads, ob.head_dim), dtype=torch.float32, device=dev)
        assert odb.compact() == sonic.OK
        assert oc.decode(oq[0], okn[0], ovn[0], oout, odb.status, omc) == sonic.OK   # allocates the workspace

        def oloop():
            for t in range(ost):
                st = oc.decode(oq[t], okn[t], ovn[t], oout, odb.status, omc)
                assert st == sonic.OK, sonic.status_string(st)
        og = None
        if use_graph:
            og = torch.cuda.CUDAGraph()
            assert odb.compact() == sonic.OK
            with torch.cuda.graph(og):
                oloop()
        ots = []
        for _ in range(3):
            assert odb.compact() == sonic.OK
            a, b_ = ev(), ev()
            a.record(stream)
            if use_graph:
                og.replay()
            else:
                oloop()
            b_.record(stream)
            torch.cuda.synchronize()
            ots.append(a.elapsed_time(b_))
        assert odb.read_status() == 0
        oms = float(np.median(ots))
        octx = okept[None, :].astype(np.float64) + np.arange(1, ost + 1)[:, None]
        obytes = float(octx.sum()) * ob.num_kv_heads * ob.head_dim * 2 * 2
        dec_other[f"workload{wl}"] = {
            "batch": ob.batch, "steps": ost, "us_per_step": round(oms * 1e3 / ost, 2),
            "tok_s": round(ob.batch * ost / (oms * 1e-3), 1), "gbs": round(obytes / (oms * 1e-3) / 1e9, 1),
            "frac_hbm_peak": round(obytes / (oms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
        del og, oc, odb, oq, okn, ovn
        torch.cuda.synchronize()

    # ---- algorithmic work ----
    row_bytes = Hkv * d * 2                       # one token's K (or V) over all kv-heads, bf16
    compact_bytes = float(kept.sum()) * row_bytes * 2 * 2 + batch.total_tokens + float(kept.sum()) * 4
    ctx = kept[None, :].astype(np.float64) + np.arange(1, steps_dec + 1)[:, None]   # rows read per step
    decode_bytes = float(ctx.sum()) * row_bytes * 2
    full_ctx = full_rows[None, :].astype(np.float64) + np.arange(1, steps_dec + 1)[:, None]
    full_bytes = float(full_ctx.sum()) * row_bytes * 2

    prefill_tflops = visible_flops / (pf_ms * 1e-3) / 1e12
    compact_gbs = compact_bytes / (cp_ms * 1e-3) / 1e9
    decode_gbs = decode_bytes / (dc_ms * 1e-3) / 1e9
    decode_tok_s = B * steps_dec / (dc_ms * 1e-3)
    value = B * steps_dec / (ms_per_step * 1e-3)

    shares = {"prefill": pf_ms, "compact": cp_ms, "decode": dc_ms}
    dominant = max(shares, key=shares.get)
    if dominant == "prefill":
        roof = {"bound": "mfma", "achieved": round(prefill_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(prefill_tflops / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic("prefill"), "kernel": "sonic_segment_attn_prefill (plan + prefill_kernel)"}
    elif dominant == "decode":
        per_launch = decode_bytes / steps_dec
        ach = per_launch / (dc_ms * 1e-3 / steps_dec) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": measured_traffic("decode"),
                "kernel": "sonic_compressed_decode, one call (decode_kernel)"}
    else:
        roof = {"bound": "hbm", "achieved": round(compact_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(compact_gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic("compact"),
                "kernel": "sonic_kv_compact (compact_kernel)"}

    rec = {
        "metric": METRIC, "value": round(value, 1), "unit": "tok/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "llama3-8b-shape: B=8, Hq/Hkv=32/8, d=128, S=256, 8 x (512 text + 102 Nexus), "
                               "C=256, L=5424, 256 decode steps", "global_batch": B, "seq_len": int(batch.max_seqlen),
                   "parallelism": "single-gpu", "graph": use_graph},
        "phases": {
            "prefill_ms": round(pf_ms, 4), "prefill_visible_tflops": round(prefill_tflops, 2),
            "prefill_frac_bf16_peak": round(prefill_tflops / PEAK_BF16_TFLOPS, 4),
            "compact_us": round(cp_ms * 1e3, 2), "compact_gbs": round(compact_gbs, 1),
            "compact_frac_hbm_peak": round(compact_gbs / PEAK_HBM_GBS, 4),
            "prefill_ms_back_to_back": round(pf_b2b_ms, 4),
            "prefill_visible_tflops_back_to_back": round(visible_flops / (pf_b2b_ms * 1e-3) / 1e12, 2),
            "prefill_with_statistics_ms_back_to_back": round(pfs_b2b_ms, 4),
            "compact_us_back_to_back": round(cp_b2b_ms * 1e3, 2),
            "compact_gbs_back_to_back": round(compact_bytes / (cp_b2b_ms * 1e-3) / 1e9, 1),
            "compact_us_cold": round(cp_cold_ms * 1e3, 2),
            "compact_gbs_cold": round(compact_bytes / (cp_cold_ms * 1e-3) / 1e9, 1),
            "decode_us_one_call_cold": round(dc_cold_ms * 1e3, 2),
            "decode_gbs_one_call_cold": round(dec1_bytes / (dc_cold_ms * 1e-3) / 1e9, 1),
            "decode_ms_256_steps": round(dc_ms, 4), "decode_us_per_step": round(dc_ms * 1e3 / steps_dec, 2),
            "decode_tok_s": round(decode_tok_s, 1), "decode_gbs": round(decode_gbs, 1),
            "decode_frac_hbm_peak": round(decode_gbs / PEAK_HBM_GBS, 4),
            "full_context_decode_ms": round(full_ms, 4), "full_context_decode_gbs": round(full_bytes / (full_ms * 1e-3) / 1e9, 1),
            "decode_speedup_vs_full_context": round(full_ms / dc_ms, 3),
            "step_ms_event_median": round(step_ms_ev, 4),
            "next_turn_nexus_us": round(ext_ms * 1e3, 2),
            "next_turn_nexus_tflops": round(ext_flops / (ext_ms * 1e-3) / 1e12, 2),
            "next_turn_nexus_frac_bf16_peak": round(ext_flops / (ext_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "role_projection_qkv_ms": round(pj_ms, 4),
            "role_projection_qkv_tflops": round(pj_flops / (pj_ms * 1e-3) / 1e12, 2),
            "role_projection_qkv_frac_bf16_peak": round(pj_flops / (pj_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "recon_targets_us": round(rc_ms * 1e3, 2),
            "recon_targets_gbs": round(rc_bytes / (rc_ms * 1e-3) / 1e9, 1),
            "recon_targets_frac_hbm_peak": round(rc_bytes / (rc_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        },
        "work": {"visible_flops": visible_flops, "compact_bytes": compact_bytes, "decode_bytes": decode_bytes,
                 "full_decode_bytes": full_bytes, "next_turn_nexus_flops": ext_flops,
                 "next_turn_nexus": f"{len(allpos)} new Nexus rows over caches of {int(ext_len_np.max())} rows",
                 "role_projection_qkv_flops": pj_flops,
                 "role_projection_qkv": f"T={batch.total_tokens} K={pj_K} N={pj_N}, fp32 out",
                 "recon_targets_bytes": rc_bytes,
                 "recon_targets": f"{rc_n} Nexus tokens, hidden size {rc_Dm}"},
        "roofline": roof,
    }
    if dec_other:
        rec["decode_other_workloads"] = dec_other
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(batch, kept)
    print(json.dumps(rec), flush=True)


def cpu_baseline(batch, kept):
    """The fp64 oracle, as it stands, on a bounded sample of one step (about 10 s of CPU
    work); scaled to tok/s."""
    from oracle import attention as OA
    from oracle import compaction as OC
    from oracle import decode as OD
    cores = len(os.sched_getaffinity(0))
    cu = batch.cu_seqlens
    B = batch.batch
    steps = batch.decode_steps
    rows_per_req, dec_per_req = 400, 64
    # prefill: rows_per_req query rows of every request, spread over its length
    t0 = time.perf_counter()
    n_rows = 0
    for b in range(B):
        s, e = int(cu[b]), int(cu[b + 1])
        rows = np.linspace(0, e - s - 1, rows_per_req).astype(np.int64)
        OA.prefill_request(batch.q[s:e], batch.k[s:e], batch.v[s:e], batch.role[s:e], batch.turn_id[s:e],
                           rows=rows)
        n_rows += len(rows)
    t_pre = (time.perf_counter() - t0) * batch.total_tokens / n_rows
    # compaction: every request
    caps = kept.astype(np.int64)
    off = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    kc = np.zeros((int(caps.sum()), batch.num_kv_heads, batch.head_dim), np.uint16)
    vc = kc.copy()
    t0 = time.perf_counter()
    OC.compact_batch(batch.k, batch.v, batch.role, cu, off, caps, kc, vc, np.zeros(int(caps.sum()), np.int32))
    t_cmp = time.perf_counter() - t0
    # decode: dec_per_req steps of every request, from the middle of the loop, over its compact cache
    # plus the decoded rows before them; scaled to B x steps
    mid = steps // 2
    t0 = time.perf_counter()
    for b in range(B):
        o, n = int(off[b]), int(caps[b])
        kctx = np.concatenate([kc[o:o + n], batch.dec_k[:mid, b]])
        vctx = np.concatenate([vc[o:o + n], batch.dec_v[:mid, b]])
        for t in range(dec_per_req):
            OD.decode_step(batch.dec_q[mid + t, b], kctx, vctx, batch.dec_k[mid + t, b], batch.dec_v[mid + t, b])
    t_dec = (time.perf_counter() - t0) / (B * dec_per_req) * B * steps
    total = t_pre + t_cmp + t_dec
    widened = widened_rows_oracle(batch)
    return {"value": round(B * steps / total, 3), "unit": "tok/s", "cores": cores, "kind": "oracle",
            "sample": f"fp64 oracle: {rows_per_req} prefill rows of each of the {B} requests (scaled to "
                      f"{batch.total_tokens} rows), compaction of the whole batch, {dec_per_req} decode steps of each "
                      f"request from mid-loop context (scaled to {B}x{steps}); estimated step time {total:.1f} s",
            "prefill_s_est": round(t_pre, 2), "compact_s_est": round(t_cmp, 3), "decode_s_est": round(t_dec, 2),
            "widened_rows": widened}


def widened_rows_oracle(batch):
    """The fp64 oracle of the four widened rows on bounded samples of the bench's shapes
    (request 0 of the batch, or a block of rows), each scaled to the bench's whole call.
    Inputs are seeded bf16 bit patterns of those shapes; only the time is used."""
    from oracle import extend as OE
    from oracle import projection as OP
    from oracle import recon as OR
    from oracle import stats as OS
    import workloads as W
    rng = np.random.default_rng(11)
    bits = lambda shape, sc=1.0: W.f32_to_bf16_bits((rng.standard_normal(shape) * sc).astype(np.float32))
    B = batch.batch
    cu = batch.cu_seqlens
    s0, e0 = int(cu[0]), int(cu[1])
    lay = batch.layouts[0]
    role0, turn0 = batch.role[s0:e0], batch.turn_id[s0:e0]
    res = {}
    # next-turn Nexus step: the last segment's Nexus rows over a cache of kept + decoded rows
    kn = lay.nexus[-1]
    cache_rows = lay.system + sum(lay.nexus) + lay.current + batch.decode_steps
    q_new, k_new, v_new = bits((kn, batch.num_q_heads, batch.head_dim)), bits((kn, batch.num_kv_heads, batch.head_dim)), \
        bits((kn, batch.num_kv_heads, batch.head_dim))
    kc, vc = batch.k[s0:s0 + cache_rows], batch.v[s0:s0 + cache_rows]
    t0 = time.perf_counter()
    OE.extend_request(q_new, k_new, v_new, kc, vc, lay.system + sum(lay.nexus[:-1]))
    res["next_turn_nexus_ms_est"] = round((time.perf_counter() - t0) * B * 1e3, 1)
    # attention statistics: Nexus mass of 200 rows of request 0 (scaled to every row), key weights of request 0
    rows = np.linspace(0, e0 - s0 - 1, 200).astype(np.int64)
    t0 = time.perf_counter()
    OS.nexus_mass(batch.q[s0:e0], batch.k[s0:e0], role0, turn0, rows=rows)
    t_m = (time.perf_counter() - t0) * batch.total_tokens / len(rows)
    t0 = time.perf_counter()
    OS.key_weight(batch.q[s0:e0], batch.k[s0:e0], role0, turn0)
    t_w = (time.perf_counter() - t0) * B
    res["attention_statistics_ms_est"] = round((t_m + t_w) * 1e3, 1)
    # role-routed QKV projection (K = 4096, N = Hq d + 2 Hkv d): 128 and 640 rows give the
    # per-row and the per-call (weight widening) parts, extrapolated to every row
    K, N = 4096, (batch.num_q_heads + 2 * batch.num_kv_heads) * batch.head_dim
    x, wt, wn = bits((640, K)), bits((N, K), 0.02), bits((N, K), 0.02)
    OP.role_routed_linear(x[:128], batch.role[s0:s0 + 128], wt, wn)   # warm (threads, pages)
    tp = []
    for n in (128, 640):
        t0 = time.perf_counter()
        OP.role_routed_linear(x[:n], batch.role[s0:s0 + n], wt, wn)
        tp.append(time.perf_counter() - t0)
    per_row = max(tp[1] - tp[0], 0.0) / 512
    res["role_projection_qkv_ms_est"] = round((max(tp[0] - 128 * per_row, 0.0) + per_row * batch.total_tokens) * 1e3, 1)
    # reconstruction targets, hidden size 4096: request 0, scaled to the batch
    h = bits((e0 - s0, 4096))
    t0 = time.perf_counter()
    OR.recon_request(h, role0, turn0)
    res["recon_targets_ms_est"] = round((time.perf_counter() - t0) * B * 1e3, 1)
    res["sample"] = ("request 0 of the batch (next-turn step, key weights, reconstruction), 200 rows of it "
                     "(Nexus mass), 128 and 640 rows (projection), each scaled to the bench's whole call")
    return res



if __name__ == "__main__":
    main()
