"""Benchmark of the SONIC hot path on one MI355X.

One step = the whole path over one batch of the long-dialogue workload (B=4,
28/4 heads, d=128; per request 512 system tokens, 32 history turns of 1024
text tokens each followed by 204 Nexus tokens, 512 current tokens: L = 40,320):
masked prefill, KV compaction, then 512 decode steps over the compacted cache.
Inputs are synthetic (seeded bf16 N(0,1)) and resident in HBM before the timed
region.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline] [--no-extras]

Prints one JSON line.  value = generated tokens per second of the whole step
(B x 512 decode tokens / step time, the step including its prefill and
compaction).  A step is three HIP graph replays (prefill, compaction, the 512
decode calls) with HIP events between them on the launch stream, so the phase
times come from the timed steps themselves.  Attached:

* phases of the step, the back-to-back and cold-cache rates of each kernel
  (a 1 GiB write before a single launch; "clean" cold also reads the 1 GiB
  back, so that the launch evicts clean lines), a plain copy of one decode
  call's bytes under both cold protocols for reference, and the same 512-step
  decode over the full, uncompressed context in two forms: the text-only cache
  (what a model without Nexus tokens keeps) and the augmented cache with the
  hierarchical mask applied per row;
* the roofline of the kernel that dominates the step, with the HBM traffic,
  MFMA-busy fraction and tile efficiency of the committed counter runs when they
  were taken on the current kernel sources;
* other_workloads: the 8B-shaped workload's whole step, the ragged workload's
  prefill and decode, the dynamic-budget workload's 1024-step decode against
  its uncompressed caches, and the four widened rows on the 8B shape;
* cpu_baseline: the fp64 oracle on the host cores, on a bounded sample.

--profile-pass runs only the headline path a few times, eagerly (for counter
collection with rocprofv3); --calibration-copy MIB runs a plain copy of known size
(the reference that scales the HBM byte counters).
"""
from __future__ import annotations

import argparse
import hashlib
import glob
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "masked-prefill visible TFLOP/s; compressed-decode tok/s; % of MFMA/HBM peak"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
HEADLINE = 4                   # the long-dialogue workload: the largest one that fits one GPU
COLD_REPS = 9


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_2601_21927_amd", "csrc", "*"))):
        h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(key: str):
    """HBM bytes per launch from the committed rocprofv3 counter runs, if they were taken
    on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    data = json.load(open(path))
    ent = data.get(key)
    if not ent or ent.get("source_hash") != kernel_source_hash():
        return None
    return ent.get("bytes_per_launch")


def measured_counters(key: str) -> dict:
    """MFMA-busy fraction and tile efficiency (visible flops / flops of the executed MFMAs)
    from the committed rocprofv3 counter runs, if they were taken on the current kernel
    sources (else null)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    ent = json.load(open(path)).get(key) if os.path.exists(path) else None
    if not ent or ent.get("source_hash") != kernel_source_hash():
        return {"mfma_busy": None, "tile_efficiency": None}
    return {"mfma_busy": ent.get("mfma_busy"), "tile_efficiency": ent.get("tile_efficiency")}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="only the headline workload")
    ap.add_argument("--calibration-copy", type=int, default=0, metavar="MIB",
                    help="run a plain device copy of MIB MiB three times and exit (the known-size "
                         "reference for the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--profile-pass", action="store_true",
                    help="run the headline path twice eagerly (prefill, compaction, decode loop) and exit")
    return ap.parse_args()


# --------------------------------------------------------------------------- device state
class Path:
    """One workload on the device: packed inputs, the compact cache, the decode inputs."""

    def __init__(self, idx: int, dev, prefill: bool = True):
        import torch
        import workloads as W
        from paper_2601_21927_amd import sonic
        from paper_2601_21927_amd.runner import SonicBatch, bf16_to_device
        self.torch, self.W, self.sonic = torch, W, sonic
        self.idx, self.dev = idx, dev
        b = W.workload(idx)
        self.b = b
        self.B, self.Hq, self.Hkv, self.d = b.batch, b.num_q_heads, b.num_kv_heads, b.head_dim
        self.steps = b.decode_steps
        vis, kept = sonic.layout_stats_host(b.cu_seqlens, b.role, b.turn_id)
        self.kept = kept.astype(np.int64)
        self.visible_flops = float(4 * self.d * self.Hq * vis.sum()) if prefill else 0.0
        self.db = SonicBatch(b.role, b.turn_id, b.cu_seqlens, b.q if prefill else None, b.k, b.v, device=dev)
        self.caps = self.kept + self.steps
        self.cache = self.db.alloc_cache(self.caps)
        self.max_ctx = int(self.caps.max())
        self.dq, self.dk, self.dv = (bf16_to_device(x, dev) for x in (b.dec_q, b.dec_k, b.dec_v))
        self.out = torch.empty((self.B, self.Hq, self.d), dtype=torch.float32, device=dev)
        self.row_bytes = self.Hkv * self.d * 2          # one token's K (or V), bf16
        # the decode workspace is allocated by a first call (the compaction of every step
        # resets the lengths it advances)
        self.ok(self.cache.decode(self.dq[0], self.dk[0], self.dv[0], self.out, self.db.status, self.max_ctx))
        self.ok(self.db.compact())
        torch.cuda.synchronize()

    def ok(self, st):
        assert st == self.sonic.OK, self.sonic.status_string(st)

    def prefill(self):
        self.ok(self.db.prefill())

    def compact(self):
        self.ok(self.db.compact())

    def decode_loop(self, cache=None, row_role=None, max_ctx=None):
        c = self.cache if cache is None else cache
        mc = self.max_ctx if max_ctx is None else max_ctx
        for t in range(self.steps):
            self.ok(c.decode(self.dq[t], self.dk[t], self.dv[t], self.out, self.db.status, mc, row_role=row_role))

    def decode_one(self, cache=None, row_role=None, max_ctx=None):
        c = self.cache if cache is None else cache
        mc = self.max_ctx if max_ctx is None else max_ctx
        self.ok(c.decode(self.dq[0], self.dk[0], self.dv[0], self.out, self.db.status, mc, row_role=row_role))

    # bytes of the compressed decode: context rows of every step (kept + appended)
    def decode_bytes(self, rows0):
        ctx = np.asarray(rows0, np.float64)[None, :] + np.arange(1, self.steps + 1)[:, None]
        return float(ctx.sum()) * self.row_bytes * 2

    def compact_bytes(self):
        return float(self.kept.sum()) * self.row_bytes * 2 * 2 + self.b.total_tokens + float(self.kept.sum()) * 4

    def full_cache(self, masked: bool):
        """The same conversations uncompressed, with room for the decode steps: the text-only
        cache (no Nexus rows, every row visible), or the augmented cache whose history-body
        rows the decode masks by their role.  Returns (cache, initial lengths, row_role)."""
        import torch
        from paper_2601_21927_amd.runner import CompactCache, bf16_to_device
        b, W = self.b, self.W
        if masked:
            rows = np.array([l.length for l in b.layouts], np.int64)
            keep = np.ones(b.total_tokens, bool)
        else:
            rows = np.array([W.text_only_layout(l).length for l in b.layouts], np.int64)
            keep = b.role != W.ROLE_NEXUS
        caps = rows + self.steps
        off = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
        c = CompactCache(int(caps.sum()), self.Hkv, self.d, off, caps.astype(np.int32), self.dev)
        kk, vv = b.k[keep], b.v[keep]
        fk = np.zeros((c.rows, self.Hkv, self.d), np.uint16)
        fv = np.zeros_like(fk)
        roles = np.full(c.rows, W.ROLE_CURRENT, np.uint8)
        src = 0
        rk = b.role[keep]
        for i in range(self.B):
            o, n = int(off[i]), int(rows[i])
            fk[o:o + n], fv[o:o + n] = kk[src:src + n], vv[src:src + n]
            roles[o:o + n] = rk[src:src + n]
            src += n
        c.k.copy_(bf16_to_device(fk, self.dev))
        c.v.copy_(bf16_to_device(fv, self.dev))
        len0 = torch.from_numpy(rows.astype(np.int32)).to(self.dev)
        c.length.copy_(len0)
        row_role = torch.from_numpy(roles).to(self.dev) if masked else None
        c.full_rows = rows
        return c, len0, row_role


def capture(fn):
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


class Timer:
    def __init__(self, torch):
        self.torch = torch
        self.stream = torch.cuda.current_stream()
        self.flush = None

    def ev(self):
        return self.torch.cuda.Event(enable_timing=True)

    def once(self, fn, pre=None):
        if pre is not None:
            pre()
        a, b = self.ev(), self.ev()
        a.record(self.stream)
        fn()
        b.record(self.stream)
        self.torch.cuda.synchronize()
        return a.elapsed_time(b)

    def median(self, fn, n, pre=None):
        return float(np.median([self.once(fn, pre) for _ in range(n)]))

    def cold(self, fn, pre=None, n=COLD_REPS, clean=False):
        """Single launches with the 256 MB Infinity Cache evicted: a 1 GiB write before each.
        The write leaves the cache full of dirty lines, which the timed launch then writes
        back as it misses; clean=True reads the 1 GiB once more after the write, so that
        the launch finds clean lines to evict (reported beside, labelled)."""
        torch = self.torch
        if self.flush is None:
            self.flush = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
            self.flush_sum = torch.empty((), dtype=torch.float32, device="cuda")
        ts = []
        for i in range(n):
            if pre is not None:
                pre()
            self.flush.fill_(float(i))
            if clean:
                torch.sum(self.flush, dim=0, out=self.flush_sum)
            ts.append(self.once(fn))
        return float(np.median(ts))

    def back_to_back(self, fn, n):
        g = capture(lambda: [fn() for _ in range(n)])
        return self.once(g.replay) / n


def gbs(nbytes, ms):
    return nbytes / (ms * 1e-3) / 1e9


def rnd(x, k=4):
    return None if x is None else round(float(x), k)


# --------------------------------------------------------------------------- headline
def headline(args, timer):
    import torch
    P = Path(HEADLINE, "cuda:0")
    g_pf = capture(P.prefill)
    g_cp = capture(P.compact)
    g_dc = capture(P.decode_loop)

    def step(marks=None):
        s = timer.stream
        if marks:
            marks[0].record(s)
        g_pf.replay()
        if marks:
            marks[1].record(s)
        g_cp.replay()
        if marks:
            marks[2].record(s)
        g_dc.replay()
        if marks:
            marks[3].record(s)

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    assert P.db.read_status() == 0
    # ---- timed region: exactly K steps ----
    marks = [[timer.ev() for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(marks[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert P.db.read_status() == 0, P.sonic.status_string(P.db.read_status())
    ms_per_step = wall * 1e3 / args.steps
    med = lambda i, j: float(np.median([m[i].elapsed_time(m[j]) for m in marks]))
    pf_ms, cp_ms, dc_ms, step_ev = med(0, 1), med(1, 2), med(2, 3), med(0, 3)

    # ---- back to back (no graph launch between launches) and cold single launches ----
    pf_b2b = timer.back_to_back(P.prefill, 3)
    cp_b2b = timer.back_to_back(P.compact, 20)
    pf_cold = timer.cold(P.prefill, n=3)
    cp_cold = timer.cold(P.compact)
    dc_cold = timer.cold(P.decode_one, pre=P.compact)   # from the freshly compacted cache
    cp_clean = timer.cold(P.compact, clean=True)
    dc_clean = timer.cold(P.decode_one, pre=P.compact, clean=True)
    # reference: a plain device copy moving the same bytes as one decode call (half read,
    # half written), under both cold protocols
    dec1_bytes = float((P.kept + 1).sum()) * P.row_bytes * 2
    cp_src = torch.empty(int(dec1_bytes) // 2, dtype=torch.uint8, device="cuda")
    cp_dst = torch.empty_like(cp_src)
    copy_cold = timer.cold(lambda: cp_dst.copy_(cp_src))
    copy_clean = timer.cold(lambda: cp_dst.copy_(cp_src), clean=True)
    del cp_src, cp_dst
    torch.cuda.synchronize()
    assert P.db.read_status() == 0

    # ---- the same 512 steps over the uncompressed context: text-only and masked augmented ----
    full = {}
    for name, masked in (("text_only", False), ("augmented_masked", True)):
        c, len0, role = P.full_cache(masked)
        mc = int(c.row_cap_host.max())
        reset = lambda c=c, len0=len0: c.length.copy_(len0)
        reset()
        P.decode_one(c, role, mc)     # allocates that cache's decode workspace
        reset()
        g = capture(lambda c=c, role=role, mc=mc: P.decode_loop(c, role, mc))
        loop_ms = timer.median(g.replay, 3, pre=reset)
        one_cold = timer.cold(lambda c=c, role=role, mc=mc: P.decode_one(c, role, mc), pre=reset)
        assert P.db.read_status() == 0
        nbytes = P.decode_bytes(c.full_rows)
        # the masked mode reads every row's role byte and K/V of every row (bodies included)
        full[name] = {"loop_ms": loop_ms, "bytes": nbytes, "one_call_cold_ms": one_cold,
                      "one_call_bytes": float((c.full_rows + 1).sum()) * P.row_bytes * 2}
        del g, c, role
        torch.cuda.empty_cache()

    dec_bytes = P.decode_bytes(P.kept)
    cmp_bytes = P.compact_bytes()
    vf = P.visible_flops
    value = P.B * P.steps / (ms_per_step * 1e-3)
    ph = {
        "prefill_ms": rnd(pf_ms), "prefill_visible_tflops": rnd(vf / (pf_ms * 1e-3) / 1e12, 2),
        "prefill_frac_bf16_peak": rnd(vf / (pf_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS),
        "prefill_ms_back_to_back": rnd(pf_b2b), "prefill_ms_cold": rnd(pf_cold),
        "compact_us": rnd(cp_ms * 1e3, 2), "compact_gbs": rnd(gbs(cmp_bytes, cp_ms), 1),
        "compact_us_back_to_back": rnd(cp_b2b * 1e3, 2), "compact_gbs_back_to_back": rnd(gbs(cmp_bytes, cp_b2b), 1),
        "compact_us_cold": rnd(cp_cold * 1e3, 2), "compact_gbs_cold": rnd(gbs(cmp_bytes, cp_cold), 1),
        "compact_frac_hbm_peak_cold": rnd(gbs(cmp_bytes, cp_cold) / PEAK_HBM_GBS),
        "decode_ms_512_steps": rnd(dc_ms), "decode_us_per_step": rnd(dc_ms * 1e3 / P.steps, 2),
        "decode_tok_s": rnd(P.B * P.steps / (dc_ms * 1e-3), 1),
        "decode_gbs_warm": rnd(gbs(dec_bytes, dc_ms), 1),
        "decode_frac_hbm_peak_warm": rnd(gbs(dec_bytes, dc_ms) / PEAK_HBM_GBS),
        "decode_us_one_call_cold": rnd(dc_cold * 1e3, 2), "decode_gbs_one_call_cold": rnd(gbs(dec1_bytes, dc_cold), 1),
        "decode_frac_hbm_peak_cold": rnd(gbs(dec1_bytes, dc_cold) / PEAK_HBM_GBS),
        "compact_us_cold_clean": rnd(cp_clean * 1e3, 2),
        "compact_frac_hbm_peak_cold_clean": rnd(gbs(cmp_bytes, cp_clean) / PEAK_HBM_GBS),
        "decode_us_one_call_cold_clean": rnd(dc_clean * 1e3, 2),
        "decode_frac_hbm_peak_cold_clean": rnd(gbs(dec1_bytes, dc_clean) / PEAK_HBM_GBS),
        "copy_same_bytes_as_decode_call_us_cold": rnd(copy_cold * 1e3, 2),
        "copy_same_bytes_as_decode_call_frac_hbm_peak_cold": rnd(gbs(dec1_bytes, copy_cold) / PEAK_HBM_GBS),
        "copy_same_bytes_as_decode_call_us_cold_clean": rnd(copy_clean * 1e3, 2),
        "copy_same_bytes_as_decode_call_frac_hbm_peak_cold_clean": rnd(gbs(dec1_bytes, copy_clean) / PEAK_HBM_GBS),
        "step_ms_event_median": rnd(step_ev),
    }
    for name, f in full.items():
        ph[f"full_{name}_decode_ms_512_steps"] = rnd(f["loop_ms"])
        ph[f"full_{name}_decode_gbs"] = rnd(gbs(f["bytes"], f["loop_ms"]), 1)
        ph[f"speedup_vs_full_{name}"] = rnd(f["loop_ms"] / dc_ms, 3)
        ph[f"full_{name}_one_call_cold_us"] = rnd(f["one_call_cold_ms"] * 1e3, 2)
        ph[f"speedup_one_call_cold_vs_full_{name}"] = rnd(f["one_call_cold_ms"] / dc_cold, 3)

    # roofline of the kernel that dominates the step
    shares = {"prefill": pf_ms, "compact": cp_ms, "decode": dc_ms}
    dominant = max(shares, key=shares.get)
    if dominant == "prefill":
        ach = vf / (pf_ms * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": rnd(ach, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": rnd(ach / PEAK_BF16_TFLOPS), "traffic": measured_traffic(f"prefill_w{HEADLINE}"),
                "kernel": "sonic_segment_attn_prefill: plan kernels + prefill_pp_kernel<128, 7>",
                "per_launch": f"{vf:.6g} visible flops (4 d flops per visible (row, key, q-head))",
                "timing": "HIP events around the prefill graph replay of each timed step (median)",
                "cold_achieved": rnd(vf / (pf_cold * 1e-3) / 1e12, 2),
                "cold_frac": rnd(vf / (pf_cold * 1e-3) / 1e12 / PEAK_BF16_TFLOPS)}
        roof.update(measured_counters(f"prefill_w{HEADLINE}"))
    elif dominant == "decode":
        ach = gbs(dec1_bytes, dc_cold)
        roof = {"bound": "hbm", "achieved": rnd(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": rnd(ach / PEAK_HBM_GBS), "traffic": measured_traffic(f"decode_w{HEADLINE}"),
                "kernel": "sonic_compressed_decode: one decode_kernel<128, 7, false> launch",
                "per_launch": f"{dec1_bytes:.6g} B (K and V of every context row of the first call)",
                "timing": "cold: 1 GiB write before each single call, median of 9",
                "warm_achieved": rnd(gbs(dec_bytes, dc_ms), 1),
                "warm_frac": rnd(gbs(dec_bytes, dc_ms) / PEAK_HBM_GBS)}
    else:
        ach = gbs(cmp_bytes, cp_cold)
        roof = {"bound": "hbm", "achieved": rnd(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": rnd(ach / PEAK_HBM_GBS), "traffic": measured_traffic(f"compact_w{HEADLINE}"),
                "kernel": "sonic_kv_compact: compact_kernel<128>", "timing": "cold single launch"}
    work = {"visible_flops": vf, "compact_bytes": cmp_bytes, "decode_bytes_512_steps": dec_bytes,
            "decode_bytes_first_call": dec1_bytes,
            "full_text_only_decode_bytes": full["text_only"]["bytes"],
            "full_augmented_decode_bytes": full["augmented_masked"]["bytes"]}
    res = dict(value=value, ms_per_step=ms_per_step, phases=ph, roofline=roof, work=work, P=P)
    return res


# --------------------------------------------------------------------------- other workloads
def workload2_step(args, timer):
    """The 8B-shaped workload's whole step (prefill, compaction, 256 decode steps) as one graph."""
    import torch
    P = Path(2, "cuda:0")
    g = capture(lambda: (P.prefill(), P.compact(), P.decode_loop()))
    for _ in range(max(1, args.warmup)):
        g.replay()
    torch.cuda.synchronize()
    step_ms = timer.median(g.replay, max(3, args.steps))
    pf = timer.median(capture(P.prefill).replay, 5)
    g_dc = capture(P.decode_loop)
    dc = timer.median(g_dc.replay, 3, pre=P.compact)
    cp_cold = timer.cold(P.compact)
    dc_cold = timer.cold(P.decode_one, pre=P.compact)
    c, len0, _ = P.full_cache(False)
    mc = int(c.row_cap_host.max())
    reset = lambda: c.length.copy_(len0)
    reset()
    P.decode_one(c, None, mc)
    reset()
    gf = capture(lambda: P.decode_loop(c, None, mc))
    full_ms = timer.median(gf.replay, 3, pre=reset)
    assert P.db.read_status() == 0
    dec_bytes = P.decode_bytes(P.kept)
    dec1 = float((P.kept + 1).sum()) * P.row_bytes * 2
    out = {"workload": "llama3-8b-shape: B=8, Hq/Hkv=32/8, d=128, S=256, 8 x (512 text + 102 Nexus), C=256, "
                       "L=5424, 256 decode steps",
           "step_ms": rnd(step_ms), "tok_s": rnd(P.B * P.steps / (step_ms * 1e-3), 1),
           "prefill_ms": rnd(pf), "prefill_visible_tflops": rnd(P.visible_flops / (pf * 1e-3) / 1e12, 2),
           "prefill_frac_bf16_peak": rnd(P.visible_flops / (pf * 1e-3) / 1e12 / PEAK_BF16_TFLOPS),
           "compact_us_cold": rnd(cp_cold * 1e3, 2), "compact_gbs_cold": rnd(gbs(P.compact_bytes(), cp_cold), 1),
           "decode_us_per_step": rnd(dc * 1e3 / P.steps, 2), "decode_gbs_warm": rnd(gbs(dec_bytes, dc), 1),
           "decode_frac_hbm_peak_warm": rnd(gbs(dec_bytes, dc) / PEAK_HBM_GBS),
           "decode_us_one_call_cold": rnd(dc_cold * 1e3, 2), "decode_gbs_one_call_cold": rnd(gbs(dec1, dc_cold), 1),
           "full_text_only_decode_ms": rnd(full_ms), "speedup_vs_full_text_only": rnd(full_ms / dc, 3)}
    del gf, c
    return out, P


def workload3(timer):
    """The ragged, per-head-scaled workload: prefill and its 256-step decode."""
    P = Path(3, "cuda:0")
    pf = timer.back_to_back(P.prefill, 5)
    g_dc = capture(P.decode_loop)
    dc = timer.median(g_dc.replay, 3, pre=P.compact)
    assert P.db.read_status() == 0
    dec_bytes = P.decode_bytes(P.kept)
    return {"workload": "ragged-50pct: B=16, Hq/Hkv=32/8, d=128, 2-12 turns of 64-1024 tokens, Nexus = half of "
                        "each turn, per-head scales U[0.5,2], 256 decode steps",
            "total_tokens": P.b.total_tokens, "visible_flops": P.visible_flops,
            "prefill_ms_back_to_back": rnd(pf), "prefill_visible_tflops": rnd(P.visible_flops / (pf * 1e-3) / 1e12, 2),
            "prefill_frac_bf16_peak": rnd(P.visible_flops / (pf * 1e-3) / 1e12 / PEAK_BF16_TFLOPS),
            "decode_us_per_step": rnd(dc * 1e3 / P.steps, 2), "decode_tok_s": rnd(P.B * P.steps / (dc * 1e-3), 1),
            "decode_gbs_warm": rnd(gbs(dec_bytes, dc), 1),
            "decode_frac_hbm_peak_warm": rnd(gbs(dec_bytes, dc) / PEAK_HBM_GBS)}


def workload5(timer):
    """The dynamic-budget decode batch: 1024 steps over the compacted caches against the same
    requests' uncompressed (text-only) caches."""
    import torch
    P = Path(5, "cuda:0", prefill=False)
    g_dc = capture(P.decode_loop)
    dc = timer.median(g_dc.replay, 3, pre=P.compact)
    dc_cold = timer.cold(P.decode_one, pre=P.compact)
    c, len0, _ = P.full_cache(False)
    mc = int(c.row_cap_host.max())
    reset = lambda: c.length.copy_(len0)
    reset()
    P.decode_one(c, None, mc)
    reset()
    gf = capture(lambda: P.decode_loop(c, None, mc))
    full_ms = timer.median(gf.replay, 3, pre=reset)
    assert P.db.read_status() == 0
    dec_bytes = P.decode_bytes(P.kept)
    dec1 = float((P.kept + 1).sum()) * P.row_bytes * 2
    full_bytes = P.decode_bytes(c.full_rows)
    out = {"workload": "dynamic-budget decode: B=64, Hq/Hkv=32/8, d=128, full context 1k-8k, Nexus budget "
                       "{10,20,50}% per request, 1024 decode steps",
           "decode_ms_1024_steps": rnd(dc), "decode_us_per_step": rnd(dc * 1e3 / P.steps, 2),
           "decode_tok_s": rnd(P.B * P.steps / (dc * 1e-3), 1), "decode_gbs": rnd(gbs(dec_bytes, dc), 1),
           "decode_frac_hbm_peak": rnd(gbs(dec_bytes, dc) / PEAK_HBM_GBS),
           "decode_us_one_call_cold": rnd(dc_cold * 1e3, 2), "decode_frac_hbm_peak_one_call_cold":
               rnd(gbs(dec1, dc_cold) / PEAK_HBM_GBS),
           "full_uncompressed_decode_ms_1024_steps": rnd(full_ms),
           "full_uncompressed_decode_gbs": rnd(gbs(full_bytes, full_ms), 1),
           "speedup_vs_full_uncompressed": rnd(full_ms / dc, 3),
           "compact_rows_mean": rnd(P.kept.mean(), 1), "full_rows_mean": rnd(c.full_rows.mean(), 1)}
    del gf, c, g_dc
    torch.cuda.empty_cache()
    return out


def widened_rows(P, timer):
    """The widened rows on the 8B-shaped workload: next-turn Nexus step, prefill with both
    attention statistics, role-routed QKV projection, reconstruction targets."""
    import torch
    sonic, W = P.sonic, P.W
    from paper_2601_21927_amd.runner import bf16_to_device
    dev = "cuda:0"
    b, db, cache = P.b, P.db, P.cache
    B, Hq, Hkv, d = P.B, P.Hq, P.Hkv, P.d
    res = {}
    # next-turn step: the turn the decode loop left at the end of each cache (C query rows +
    # the decoded rows) becomes a history segment; its Nexus rows attend to the whole cache
    P.compact()
    g_dc = capture(P.decode_loop)
    g_dc.replay()
    torch.cuda.synchronize()
    keep_np = np.array([l.system + sum(l.nexus) for l in b.layouts], np.int32)
    len_np = (P.kept + P.steps).astype(np.int32)
    npos = []
    for i, l in enumerate(b.layouts):
        p0 = int(b.cu_seqlens[i]) + l.system + sum(l.bodies) + sum(l.nexus[:-1])
        npos.append(np.arange(p0, p0 + l.nexus[-1]))
    kn = np.array([len(x) for x in npos], np.int64)
    allpos = np.concatenate(npos)
    ext_cu = torch.from_numpy(np.concatenate([[0], np.cumsum(kn)]).astype(np.int32)).to(dev)
    ext_keep = torch.from_numpy(keep_np).to(dev)
    ext_len0 = torch.from_numpy(len_np).to(dev)
    ext_len = ext_len0.clone()
    ext_k, ext_v = cache.k.clone(), cache.v.clone()
    eq, ek, e_v = (bf16_to_device(x[allpos], dev) for x in (b.q, b.k, b.v))
    ext_out = torch.empty((len(allpos), Hq, d), dtype=torch.float32, device=dev)
    ext_ws = torch.empty(max(sonic.nexus_extend_workspace_bytes(B, len(allpos), P.max_ctx, Hkv, d), 256),
                         dtype=torch.uint8, device=dev)

    def run_extend():
        P.ok(sonic.nexus_extend(ext_cu, ext_keep, ext_k, ext_v, cache.row_off, cache.row_cap, ext_len, eq, ek,
                                e_v, ext_out, ext_ws, db.status, max_rows=P.max_ctx))
    reset = lambda: ext_len.copy_(ext_len0)
    reset()
    run_extend()
    reset()
    g = capture(run_extend)
    ext_ms = timer.median(g.replay, 20, pre=reset)
    assert np.array_equal(ext_len.cpu().numpy(), keep_np + kn)
    ext_flops = float(4 * d * Hq * np.sum(kn * (len_np + kn)))
    res["next_turn_nexus_us"] = rnd(ext_ms * 1e3, 2)
    res["next_turn_nexus_tflops"] = rnd(ext_flops / (ext_ms * 1e-3) / 1e12, 2)
    res["next_turn_nexus_frac_bf16_peak"] = rnd(ext_flops / (ext_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS)
    res["next_turn_nexus"] = f"{len(allpos)} new Nexus rows over caches of {int(len_np.max())} rows"
    # prefill with both attention statistics
    mass = torch.empty((b.total_tokens, Hq), dtype=torch.float32, device=dev)
    kw = torch.empty((b.total_tokens,), dtype=torch.float32, device=dev)
    stats = lambda: P.ok(db.prefill(nexus_mass=mass, key_weight=kw))
    stats()
    res["prefill_with_statistics_ms_back_to_back"] = rnd(timer.back_to_back(stats, 5))
    res["prefill_ms_back_to_back"] = rnd(timer.back_to_back(P.prefill, 5))
    # role-routed fused QKV projection over the whole batch (K = 4096, N = 4096 + 2 x 1024)
    K, N = 4096, Hq * d + 2 * Hkv * d
    gen = torch.Generator(device=dev).manual_seed(11)
    x = torch.randn((b.total_tokens, K), generator=gen, device=dev).to(torch.bfloat16)
    wt = (torch.randn((N, K), generator=gen, device=dev) * 0.02).to(torch.bfloat16)
    wn = (torch.randn((N, K), generator=gen, device=dev) * 0.02).to(torch.bfloat16)
    y = torch.empty((b.total_tokens, N), dtype=torch.float32, device=dev)
    ws = torch.empty(sonic.role_projection_workspace_bytes(b.total_tokens), dtype=torch.uint8, device=dev)
    proj = lambda: P.ok(sonic.role_projection(db.role, x, wt, wn, y, ws, db.status))
    proj()
    pj_ms = timer.back_to_back(proj, 5)
    pj_flops = 2.0 * b.total_tokens * K * N
    res["role_projection_qkv_ms"] = rnd(pj_ms)
    res["role_projection_qkv_tflops"] = rnd(pj_flops / (pj_ms * 1e-3) / 1e12, 2)
    res["role_projection_qkv_frac_bf16_peak"] = rnd(pj_flops / (pj_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS)
    del x, y
    # reconstruction targets, hidden size 4096
    Dm = 4096
    h = torch.randn((b.total_tokens, Dm), generator=gen, device=dev).to(torch.bfloat16)
    n = int((b.role == W.ROLE_NEXUS).sum())
    tgt = torch.empty((n, Dm), dtype=torch.float32, device=dev)
    cs = torch.empty((n,), dtype=torch.float32, device=dev)
    rt = torch.empty((n,), dtype=torch.float32, device=dev)
    rws = torch.empty(sonic.nexus_recon_workspace_bytes(B, b.total_tokens), dtype=torch.uint8, device=dev)
    rec = lambda: P.ok(sonic.nexus_recon_targets(db.cu, db.role, db.turn_id, h, tgt, cs, rt, rws, db.status))
    rec()
    rc_ms = timer.back_to_back(rec, 10)
    body = sum(sum(l.bodies[i] for i in range(len(l.bodies)) if l.nexus[i] > 0) for l in b.layouts)
    rc_bytes = float(body + n) * Dm * 2 + n * (Dm * 4 + 8)
    res["recon_targets_us"] = rnd(rc_ms * 1e3, 2)
    res["recon_targets_gbs"] = rnd(gbs(rc_bytes, rc_ms), 1)
    res["recon_targets_frac_hbm_peak"] = rnd(gbs(rc_bytes, rc_ms) / PEAK_HBM_GBS)
    assert db.read_status() == 0
    return res


# --------------------------------------------------------------------------- CPU oracle
def cpu_baseline(P):
    """The fp64 oracle, as it stands, on a bounded sample of one headline step (about 10-30 s
    of CPU work); scaled to generated tok/s of the whole step."""
    from oracle import attention as OA
    from oracle import compaction as OC
    from oracle import decode as OD
    b = P.b
    cores = len(os.sched_getaffinity(0))
    cu = b.cu_seqlens
    B, steps = b.batch, b.decode_steps
    rows_per_req, dec_per_req = 160, 16
    t0 = time.perf_counter()
    n_rows = 0
    for i in range(B):
        s, e = int(cu[i]), int(cu[i + 1])
        rows = np.linspace(0, e - s - 1, rows_per_req).astype(np.int64)
        OA.prefill_request(b.q[s:e], b.k[s:e], b.v[s:e], b.role[s:e], b.turn_id[s:e], rows=rows)
        n_rows += len(rows)
    t_pre = (time.perf_counter() - t0) * b.total_tokens / n_rows
    caps = P.kept
    off = np.concatenate([[0], np.cumsum(caps)[:-1]]).astype(np.int64)
    kc = np.zeros((int(caps.sum()), b.num_kv_heads, b.head_dim), np.uint16)
    vc = kc.copy()
    t0 = time.perf_counter()
    OC.compact_batch(b.k, b.v, b.role, cu, off, caps, kc, vc, np.zeros(int(caps.sum()), np.int32))
    t_cmp = time.perf_counter() - t0
    mid = steps // 2
    t0 = time.perf_counter()
    for i in range(B):
        o, n = int(off[i]), int(caps[i])
        kctx = np.concatenate([kc[o:o + n], b.dec_k[:mid, i]])
        vctx = np.concatenate([vc[o:o + n], b.dec_v[:mid, i]])
        for t in range(dec_per_req):
            OD.decode_step(b.dec_q[mid + t, i], kctx, vctx, b.dec_k[mid + t, i], b.dec_v[mid + t, i])
    t_dec = (time.perf_counter() - t0) / (B * dec_per_req) * B * steps
    total = t_pre + t_cmp + t_dec
    return {"value": round(B * steps / total, 4), "unit": "tok/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(),
            "sample": f"fp64 oracle on the long-dialogue step: {rows_per_req} prefill rows of each of the {B} "
                      f"requests, evenly spaced (scaled to {b.total_tokens} rows), the compaction of the whole "
                      f"batch, {dec_per_req} decode steps of each request from mid-loop context (scaled to "
                      f"{B}x{steps}); estimated step time {total:.1f} s",
            "prefill_s_est": round(t_pre, 2), "compact_s_est": round(t_cmp, 3), "decode_s_est": round(t_dec, 2)}


# --------------------------------------------------------------------------- main
def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2601_21927_amd import sonic
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    sonic.lib()
    torch.cuda.set_device(0)
    timer = Timer(torch)

    if args.calibration_copy > 0:
        src = torch.empty(args.calibration_copy << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibration_copy_bytes": src.numel()}))
        return

    if args.profile_pass:
        P = Path(HEADLINE, "cuda:0")
        for _ in range(2):
            P.prefill()
            P.compact()
            P.decode_loop()
        torch.cuda.synchronize()
        assert P.db.read_status() == 0
        print(json.dumps({"profile_pass": f"workload {HEADLINE}: 2 x (prefill, compaction, {P.steps} decode calls)"}))
        return

    h = headline(args, timer)
    P4 = h.pop("P")
    rec = {
        "metric": METRIC, "value": round(h["value"], 1), "unit": "tok/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(h["ms_per_step"], 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "long-dialogue: B=4, Hq/Hkv=28/4, d=128, S=512, 32 x (1024 text + 204 Nexus), "
                               "C=512, L=40320 (80% compression), 512 decode steps",
                   "global_batch": P4.B, "seq_len": int(P4.b.max_seqlen), "parallelism": "single-gpu",
                   "graph": True},
        "phases": h["phases"], "roofline": h["roofline"], "work": h["work"],
    }
    cpu = None if args.no_cpu_baseline else cpu_baseline(P4)
    del P4
    torch.cuda.empty_cache()
    if not args.no_extras:
        other = {}
        w2, P2 = workload2_step(args, timer)
        other["workload2"] = w2
        other["widened_rows_workload2"] = widened_rows(P2, timer)
        del P2
        torch.cuda.empty_cache()
        other["workload3"] = workload3(timer)
        torch.cuda.empty_cache()
        other["workload5"] = workload5(timer)
        rec["other_workloads"] = other
    if cpu is not None:
        rec["cpu_baseline"] = cpu
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
