#!/usr/bin/env python3
"""Benchmark of the hot path on one MI355X.

Workload: 4000 rows x 32000 binary32 logits, i.i.d. N(0, 2) from seed 0, with
1% of the rows shifted by +1000 (the paper's large-batch softmax case).  One
step is the whole hot path over that batch, resident in HBM:

  1. online softmax (two loads and one store per element), then
  2. fused online softmax + top-k, K = 5 (one load per element).

The printed JSON line reports the step's algorithmic bytes per second
(online: 12 B/element; fused top-k: 4 B/element + 8 B per output pair), a
per-kernel breakdown timed with HIP events on the launch stream, the roofline
entry of the dominant kernel, and the oracle timed on the host cores.  The
naive and safe modes are timed on the same batch after the steps, for the
paper's memory-access comparison (with the row-resident variant, one load and
one store per element, reported apart), the projection with softmax + top-k in
its epilogue (against the projection writing logits), and the paper's four softmax + top-k
algorithms (online fused, safe fused, online unfused, safe unfused), with a
plain copy and a plain read as reference kernels.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
       python bench.py --sweep FILE   (every workload shape and V sweep)
       python bench.py --traffic-probe KEY   (one operation, for a counter pass)
       python bench.py --traffic-summary DIR (counter passes -> profiles/traffic*)
       python bench.py --sweep-summary FILE  (sweep records -> profiles/sweep_all_workloads.md)
       python bench.py --kernel-stats DIR OUT COMMAND (rocprofv3 statistics -> profiles/OUT)
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0  # MI355X HBM3E, decimal GB/s
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bfloat16 matrix peak
N_ROWS, V_LEN, SIGMA, SHIFT_FRAC, K_TOP = 4000, 32000, 2.0, 0.01, 5
WORKLOAD = "online softmax + fused softmax/top-5, 4000x32000 fp32 N(0,2), 1% rows +1000"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_sha() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(ROOT, "paper_1805_02867_amd", "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_entry(name: str):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    e = data.get(name)
    if not e or e.get("source_sha") != kernel_source_sha():
        return None
    return e.get("bytes_per_launch")


def cpu_model() -> str:
    """The host CPU's model name (Linux), or an empty string."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def timed_calls(fn, reps: int, stream):
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]  # ms


def queued_batches(fn, reps: int, batches: int, stream):
    """Per-call GPU time of `fn`: each batch of `reps` back-to-back calls is
    enqueued behind a spin kernel, so the GPU never waits for the host and
    the events bracket GPU time only (small shapes are host-rate bound
    otherwise).  Returns one per-call time (us) per batch."""
    import torch
    out = []
    for _ in range(batches):
        torch.cuda._sleep(int(2.4e9 * 0.004))  # ~4 ms of spinning while the calls queue
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        out.append(a.elapsed_time(b) * 1e3 / reps)
    return out


def cold_calls(fn, reps: int, stream, flush):
    """Per-call GPU time of `fn` with cold caches: before each call `flush()`
    reads a buffer of at least 512 MB (twice the last-level cache) with
    ordinary, cache-allocating loads: a read evicts the input without leaving
    dirty lines whose write-back would land in the timed call, and
    non-temporal loads would not evict it all.  Events bracket the call
    alone; the calls are queued behind a spin kernel, as in queued_batches.
    Returns one time (us) per call."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    torch.cuda._sleep(int(2.4e9 * 0.004))
    for a, b in evs:
        flush()
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) * 1e3 for a, b in evs]


def proj_compare(osm, torch, N, H, V, K, reps, stream):
    """The projection (bfloat16 h: N x H, w: V x H) with softmax + top-K in its
    epilogue, against the two-kernel path (the same projection writing binary32
    logits, then the fused top-K) and against torch's bfloat16 matmul (a
    library GEMM) followed by the fused top-K.  Times are medians per call."""
    g = torch.Generator(device="cuda").manual_seed(0)
    h = torch.randn(N, H, device="cuda", generator=g).to(torch.bfloat16)
    w = (torch.randn(V, H, device="cuda", generator=g) / H ** 0.5).to(torch.bfloat16)
    logits = torch.empty(N, V, device="cuda")
    lb = torch.empty(N, V, device="cuda", dtype=torch.bfloat16)
    vals = torch.empty((N, K), dtype=torch.float32, device="cuda")
    idx = torch.empty((N, K), dtype=torch.int32, device="cuda")
    runs = {
        "fused": lambda: osm.proj_softmax_topk(h, w, K, vals, idx),
        "proj_then_topk": lambda: (osm.proj(h, w, logits), osm.softmax_topk(logits, K, vals, idx)),
        "proj_only": lambda: osm.proj(h, w, logits),
        "library_gemm_then_topk": lambda: (torch.matmul(h, w.t(), out=lb),
                                           osm.softmax_topk(lb, K, vals, idx)),
    }
    flops = 2.0 * N * H * V
    out = {"N": N, "H": H, "V": V, "K": K, "dtype": "bf16 in, f32 accumulate"}
    for name, fn in runs.items():
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        t = median(timed_calls(fn, reps, stream)) * 1e3
        out[name + "_us"] = round(t, 1)
    out["fused_TFLOPs"] = round(flops / out["fused_us"] / 1e6, 1)
    out["fused_frac_of_mfma_peak"] = round(flops / out["fused_us"] / 1e6 / PEAK_BF16_TFLOPS, 4)
    out["proj_only_TFLOPs"] = round(flops / out["proj_only_us"] / 1e6, 1)
    del h, w, logits, lb
    torch.cuda.empty_cache()
    return out


def median(xs):
    s = sorted(xs)
    n = len(s)
    return s[n // 2] if n % 2 else 0.5 * (s[n // 2 - 1] + s[n // 2])


def pct(xs, q):
    s = sorted(xs)
    return s[min(len(s) - 1, max(0, int(round(q * (len(s) - 1)))))]


def copy_probe():
    """A plain 512 MB device copy, for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = N_ROWS * V_LEN
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    t = timed_calls(lambda: b.copy_(a), 20, torch.cuda.current_stream())
    log(f"copy {n * 4 / 1e6:.0f} MB: median {median(t) * 1e3:.1f} us, "
        f"{2 * n * 4 / (median(t) * 1e-3) / 1e9:.0f} GB/s (read+write)")


def proj_probe(osm):
    """The projection and the fused projection + softmax + top-5 at
    4000 x 4096 x 128256 (bfloat16 h, w), three calls each, for kernel
    statistics and counters under a profiler."""
    import torch
    N, H, V = 4000, 4096, 128256
    g = torch.Generator(device="cuda").manual_seed(0)
    h = torch.randn(N, H, device="cuda", generator=g).to(torch.bfloat16)
    w = (torch.randn(V, H, device="cuda", generator=g) / H ** 0.5).to(torch.bfloat16)
    out = torch.empty(N, V, device="cuda")
    for _ in range(3):
        osm.proj(h, w, out)
        osm.proj_softmax_topk(h, w, 5)
    torch.cuda.synchronize()
    log("proj probe done")


def topk_probe(osm, synth):
    """The fused softmax + top-k at 4000 x 32000 binary32 (K = 5, 50) and
    32768 x 128256 bfloat16 (K = 5, 50), three calls each, for kernel
    statistics and counters under a profiler."""
    import torch
    for N, V, dt, sg in ((4000, 32000, "f32", 2.0), (32768, 128256, "bf16", 4.0)):
        x = synth.logits(N, V, sigma=sg, seed=0, dtype=dt, device="cuda")
        for K in (5, 50):
            for _ in range(3):
                osm.softmax_topk(x, K)
        torch.cuda.synchronize()
        del x
        torch.cuda.empty_cache()
    log("topk probe done")


# HBM traffic: every operation of every workload, one operation per profiled
# process (so that the counters of a process belong to one operation).
# Workloads (synth.logits arguments) and the operations measured on them,
# with the algorithmic bytes of one call (online and naive softmax: two loads
# and one store per element; safe: three loads and one store; fused top-k: one
# load per element and K (value, index) pairs per row).
TRAFFIC_WORKLOADS = {
    "4000x32000_f32": dict(N=4000, V=32000, sigma=2.0, dtype="f32", shift_frac=0.01),
    "10x1000000_f32": dict(N=10, V=1_000_000, sigma=3.0, dtype="f32"),
    "4000x50000_f32_ties": dict(N=4000, V=50000, sigma=2.0, dtype="f32", tie_frac=0.01),
    "32768x128256_bf16": dict(N=32768, V=128256, sigma=4.0, dtype="bf16"),
}
TRAFFIC_OPS = [  # (key, workload, op, mode or K)
    ("softmax_naive_4000x32000_f32", "4000x32000_f32", "softmax", "naive"),
    ("softmax_safe_4000x32000_f32", "4000x32000_f32", "softmax", "safe"),
    ("softmax_online_4000x32000_f32", "4000x32000_f32", "softmax", "online"),
    ("topk5_4000x32000_f32", "4000x32000_f32", "topk", 5),
    ("softmax_online_10x1000000_f32", "10x1000000_f32", "softmax", "online"),
    ("topk5_10x1000000_f32", "10x1000000_f32", "topk", 5),
    ("topk5_4000x50000_f32_ties", "4000x50000_f32_ties", "topk", 5),
    ("topk10_4000x50000_f32_ties", "4000x50000_f32_ties", "topk", 10),
    ("softmax_online_32768x128256_bf16", "32768x128256_bf16", "softmax", "online"),
    ("softmax_safe_32768x128256_bf16", "32768x128256_bf16", "softmax", "safe"),
    ("topk50_32768x128256_bf16", "32768x128256_bf16", "topk", 50),
]
TRAFFIC_CALLS = 3


def traffic_algorithmic_bytes(wl: dict, op: str, arg) -> int:
    es = 2 if wl["dtype"] == "bf16" else 4
    n = wl["N"] * wl["V"]
    if op == "softmax":
        return (4 if arg == "safe" else 3) * es * n
    return es * n + 8 * int(arg) * wl["N"]


def traffic_probe(key: str):
    """One operation of TRAFFIC_OPS (or `copy`: the plain 512 MB copy that
    scales the counters), TRAFFIC_CALLS calls, for a counter pass."""
    import torch
    import paper_1805_02867_amd as osm
    from paper_1805_02867_amd import synth
    if key == "copy":
        copy_probe()
        return
    ops = {k: (w, o, a) for k, w, o, a in TRAFFIC_OPS}
    if key not in ops:
        raise SystemExit(f"unknown traffic probe {key}; one of copy, {', '.join(ops)}")
    w, op, arg = ops[key]
    wl = dict(TRAFFIC_WORKLOADS[w])
    N, V = wl.pop("N"), wl.pop("V")
    x = synth.logits(N, V, seed=0, device="cuda", **wl)
    if op == "softmax":
        y = torch.empty_like(x)
        for _ in range(TRAFFIC_CALLS):
            osm.softmax_fwd(x, y, mode=arg)
    else:
        vals = torch.empty((N, arg), dtype=torch.float32, device="cuda")
        idx = torch.empty((N, arg), dtype=torch.int32, device="cuda")
        for _ in range(TRAFFIC_CALLS):
            osm.softmax_topk(x, arg, vals, idx)
    torch.cuda.synchronize()
    log(f"traffic probe {key}: {TRAFFIC_CALLS} calls")


def _counter_rows(d: str):
    """(dispatch id, kernel, counter, value, start ns, end ns) from the
    counter-collection CSV files of one rocprofv3 output directory."""
    import csv
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    acc = {}
    for fn in files:
        with open(fn, newline="") as f:
            for r in csv.DictReader(f):
                name = r["Kernel_Name"].split("(")[0].strip()
                if name.startswith("void "):
                    name = name[5:]
                key = (fn, r["Dispatch_Id"], name, r["Counter_Name"])
                v = float(r["Counter_Value"])
                s = int(r.get("Start_Timestamp") or 0)
                e = int(r.get("End_Timestamp") or 0)
                if key in acc:  # several instances of one counter: summed
                    acc[key][0] += v
                else:
                    acc[key] = [v, s, e]
    return [(k[1], k[2], k[3], v[0], v[1], v[2]) for k, v in acc.items()]


def _per_kernel(d: str, counter: str):
    """Per library kernel (osm::...): dispatches, median counter value and
    median duration (ns) over its dispatches, in first-dispatch order."""
    out = {}
    for disp, name, cname, v, s, e in sorted(_counter_rows(d), key=lambda r: int(r[0])):
        if cname != counter or not (name.startswith("osm::") or "copyBuffer" in name):
            continue
        out.setdefault(name, ([], []))
        out[name][0].append(v)
        out[name][1].append(e - s)
    return {k: (len(v[0]), median(v[0]), median(v[1])) for k, v in out.items()}


def traffic_summary(d: str):
    """profiles/traffic.json and profiles/traffic_all_workloads.md from the
    counter passes under d: <key>_fetch and <key>_write for every key of
    TRAFFIC_OPS and for `copy` (rocprofv3 -d directories)."""
    cf = _per_kernel(os.path.join(d, "copy_fetch"), "FETCH_SIZE")
    cw = _per_kernel(os.path.join(d, "copy_write"), "WRITE_SIZE")
    copy_bytes = N_ROWS * V_LEN * 4
    (ck,) = [k for k in cf if "copyBuffer" in k]
    fetch_scale = copy_bytes / (cf[ck][1] * 1024)
    write_scale = copy_bytes / (cw[ck][1] * 1024)
    sha = kernel_source_sha()
    data = {"_scale": {"kernel": ck, "bytes": copy_bytes, "fetch_kib": cf[ck][1],
                       "write_kib": cw[ck][1], "fetch_scale": fetch_scale,
                       "write_scale": write_scale, "source_sha": sha}}
    rows = []
    for key, w, op, arg in TRAFFIC_OPS:
        fk = _per_kernel(os.path.join(d, key + "_fetch"), "FETCH_SIZE")
        wk = _per_kernel(os.path.join(d, key + "_write"), "WRITE_SIZE")
        kernels = [k for k in fk if k.startswith("osm::")]
        calls = TRAFFIC_CALLS
        per = []
        for k in kernels:
            n, fkib, ns = fk[k]
            wkib = wk.get(k, (0, 0.0, 0))[1]
            per.append({"kernel": k, "dispatches_per_call": n / calls,
                        "fetch_kib": fkib, "write_kib": wkib,
                        "read_bytes": fkib * 1024 * fetch_scale,
                        "write_bytes": wkib * 1024 * write_scale, "us": ns / 1e3})
        rd = sum(p["read_bytes"] * p["dispatches_per_call"] for p in per)
        wr = sum(p["write_bytes"] * p["dispatches_per_call"] for p in per)
        us = sum(p["us"] * p["dispatches_per_call"] for p in per)
        alg = traffic_algorithmic_bytes(TRAFFIC_WORKLOADS[w], op, arg)
        data[key] = {"workload": w, "op": op, "arg": arg, "kernels": per,
                     "read_bytes": rd, "write_bytes": wr, "bytes_per_launch": rd + wr,
                     "algorithmic_bytes": alg, "us_under_counters": us, "source_sha": sha}
        rows.append((key, per, rd, wr, alg, us))
    with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as f:
        json.dump(data, f, indent=1)
    cmd = ("rocprofv3 --pmc {C} -d <out>/{key}_{c} -o run -f csv -- "
           "python3 bench.py --traffic-probe {key}")
    lines = [
        "# HBM traffic per call, every workload (rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE)", "",
        "Each operation runs alone in its own process, {} calls; one counter per pass:".format(
            TRAFFIC_CALLS), "",
        "```",
        cmd.format(C="FETCH_SIZE", c="fetch", key="<key>"),
        cmd.format(C="WRITE_SIZE", c="write", key="<key>"),
        "python3 bench.py --traffic-summary <out>",
        "```", "",
        f"`<key>` is `copy` and each key below. Kernel sources hash: `{sha}`.", "",
        f"Scale: a plain {copy_bytes / 1e6:.0f} MB copy (`{ck}`) reads FETCH_SIZE = "
        f"{cf[ck][1]:.0f} KiB and WRITE_SIZE = {cw[ck][1]:.0f} KiB per dispatch, so bytes = "
        f"FETCH_SIZE x 1024 x {fetch_scale:.4f} and WRITE_SIZE x 1024 x {write_scale:.4f}.",
        "FETCH_SIZE counts what the L2 caches fetch over the fabric: reads served by the "
        "256 MB last-level cache (MALL) count too, so `read` is an upper bound on HBM reads.",
        "",
        "Per call (medians over the calls' dispatches); `us` is the dispatch time while the "
        "counters were collected (indicative only):", "",
        "| key | kernels (dispatches per call) | read B | write B | algorithmic B | "
        "(read+write)/alg | us | alg GB/s | fabric GB/s |",
        "|---|---|---|---|---|---|---|---|---|"]
    for key, per, rd, wr, alg, us in rows:
        ks = "<br>".join(f"`{p['kernel']}` ({p['dispatches_per_call']:g})" for p in per)
        lines.append(f"| {key} | {ks} | {rd:.4g} | {wr:.4g} | {alg:.4g} | {(rd + wr) / alg:.3f} | "
                     f"{us:.1f} | {alg / us / 1e3:.0f} | {(rd + wr) / us / 1e3:.0f} |")
    with open(os.path.join(ROOT, "profiles", "traffic_all_workloads.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    log("wrote profiles/traffic.json and profiles/traffic_all_workloads.md")


def sweep_summary(path: str):
    """profiles/sweep_all_workloads.md from the JSON records of `--sweep`."""
    recs = [json.loads(l) for l in open(path) if l.strip()]
    by = {}
    for r in recs:
        by.setdefault(r["workload"], {})[r["op"]] = r
    named = [w for w in by if not w.startswith("sweep_") and not w.startswith("proj_")]
    L = ["# All workload shapes, the V sweeps and the K sweep (bench.py --sweep)", "",
         "Commands (repository root, GPU host): `python bench.py --sweep <file>`, then "
         "`python bench.py --sweep-summary <file>`.", "",
         "Each entry is the median over 10 batches of back-to-back calls through the Python "
         "binding, each batch queued behind a ~4 ms spin kernel so that the events bracket GPU "
         "time, not the host's call rate. GB/s are algorithmic: softmax naive/online 12 B/elem "
         "(binary32) or 6 (bfloat16), safe 16 or 8, resident 8 or 4; fused top-k 4 or 2 B/elem "
         "+ 8 B per output pair. Peak = 8000 GB/s.", "",
         "## Workload shapes", "",
         "| workload | op | plan | us | GB/s | % of 8 TB/s |", "|---|---|---|---|---|---|"]
    for w in named:
        for op, r in by[w].items():
            if op.endswith("_cold") or "GBps" not in r or op.startswith("topk_") and \
                    not op.startswith("topk_fused"):
                continue
            L.append(f"| {w} | {op} | {r.get('plan', '')} | {r['us']} | {r['GBps']} | "
                     f"{r['GBps'] / PEAK_HBM_GBS * 100:.1f} |")
    L += ["", "## Cold caches", "",
          "Inputs that fit in the 256 MB last-level cache, timed again with a 512 MB buffer "
          "read (torch sum: ordinary loads, so it evicts without dirty lines) before each call "
          "(events around the call alone, calls queued behind a spin kernel; median of 20). "
          "Warm = the back-to-back figure; an isolated call also carries ~3 us of dispatch "
          "that back-to-back calls hide.", "",
          "| workload | online softmax warm us | cold us | cold GB/s (% of 8 TB/s) | "
          "fused top-5 warm us | cold us | cold GB/s (%) |", "|---|---|---|---|---|---|---|"]
    for w, ops in by.items():
        if "softmax_online_cold" not in ops:
            continue
        sc, tc = ops["softmax_online_cold"], ops.get("topk_fused_k5_cold")
        tw = ops.get("topk_fused_k5", ops.get("topk_online_fused_k5", {}))
        L.append(f"| {w} | {ops['softmax_online']['us']} | {sc['us']} | {sc['GBps']} "
                 f"({sc['GBps'] / PEAK_HBM_GBS * 100:.1f}) | {tw.get('us', '')} | "
                 f"{tc['us'] if tc else ''} | "
                 + (f"{tc['GBps']} ({tc['GBps'] / PEAK_HBM_GBS * 100:.1f}) |" if tc else " |"))
    L += ["", "## Softmax + top-k algorithms (Section 5.2's comparison), K = 5", "",
          "Times in us; ratio = safe unfused / online fused (the paper's Fig. 3 and 4 quantity).",
          "", "| workload | V | online fused | safe fused | online unfused | safe unfused | "
          "ratio | top-k plan |", "|---|---|---|---|---|---|---|---|"]
    for w, ops in by.items():
        if "topk_ratios_k5" not in ops:
            continue
        t = {a: ops[f"topk_{a}_k5"]["us"] for a in
             ("online_fused", "safe_fused", "online_unfused", "safe_unfused")}
        r = ops["topk_ratios_k5"]
        L.append(f"| {w} | {r['V']} | {t['online_fused']} | {t['safe_fused']} | "
                 f"{t['online_unfused']} | {t['safe_unfused']} | "
                 f"{r['safe_unfused_over_online_fused']} | {r['topk_plan']} |")
    L += ["", "## K sweep (ratio safe unfused / online fused)", "",
          "| workload | K | online fused us | safe unfused us | ratio |", "|---|---|---|---|---|"]
    for w, ops in by.items():
        ks = sorted(int(op[len("topk_ratios_k"):]) for op in ops if op.startswith("topk_ratios_k"))
        if len(ks) < 2:
            continue
        for K in ks:
            L.append(f"| {w} | {K} | {ops[f'topk_online_fused_k{K}']['us']} | "
                     f"{ops[f'topk_safe_unfused_k{K}']['us']} | "
                     f"{ops[f'topk_ratios_k{K}']['safe_unfused_over_online_fused']} |")
    L += ["", "## Softmax V sweeps (elements/s; ratio = safe / online time)", "",
          "resident = the row-resident variant (one load + one store per element), reported "
          "apart.", "", "| workload | V | online us | safe us | naive us | resident us | "
          "online elem/s | safe/online |", "|---|---|---|---|---|---|---|---|"]
    for w, ops in by.items():
        if not w.startswith("sweep_") or "softmax_online" not in ops:
            continue
        o = ops["softmax_online"]
        res = ops.get("softmax_resident", {}).get("us", "")
        L.append(f"| {w} | {o['V']} | {o['us']} | {ops['softmax_safe']['us']} | "
                 f"{ops['softmax_naive']['us']} | {res} | {o['elements_per_s']:.3g} | "
                 f"{ops['softmax_safe']['us'] / o['us']:.3f} |")
    L += ["", "## Projection with softmax + top-5 in its epilogue (bfloat16 h, W; binary32 "
          "accumulation)", "",
          "fused = proj_softmax_topk (logits never written); proj_then_topk = proj_fwd writing "
          "binary32 logits, then the fused top-k over them; library = torch's bfloat16 matmul "
          "(hipBLASLt) then the fused top-k over bfloat16 logits. TF/s = 2 N H V / time; the "
          "bfloat16 dense peak is 2500 TF/s.", "",
          "| N x H x V | fused us | fused TF/s | proj_fwd us (TF/s) | proj_then_topk us | "
          "library_gemm_then_topk us |", "|---|---|---|---|---|---|"]
    for w, ops in by.items():
        if not w.startswith("proj_"):
            continue
        r = ops["proj_softmax_topk_k5"]
        L.append(f"| {r['N']} x {r['H']} x {r['V']} | {r['fused_us']} | {r['fused_TFLOPs']} | "
                 f"{r['proj_only_us']} ({r['proj_only_TFLOPs']}) | {r['proj_then_topk_us']} | "
                 f"{r['library_gemm_then_topk_us']} |")
    with open(os.path.join(ROOT, "profiles", "sweep_all_workloads.md"), "w") as f:
        f.write("\n".join(L) + "\n")
    log("wrote profiles/sweep_all_workloads.md")


def kernel_stats_summary(d: str, out_name: str, command: str):
    """A markdown table of rocprofv3's kernel statistics (--kernel-trace --stats)
    found under d, written to profiles/<out_name>."""
    import csv
    files = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {d}")
    rows = []
    with open(files[0], newline="") as f:
        for r in csv.DictReader(f):
            name = r["Name"].split("(")[0].strip()
            if name.startswith("void "):
                name = name[5:]
            rows.append((name, int(r["Calls"]), float(r["AverageNs"]) / 1e3,
                         float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3,
                         float(r["Percentage"])))
    rows.sort(key=lambda r: -r[5])
    L = [f"# Kernel time (rocprofv3 --kernel-trace --stats)", "", "Command (repository root, GPU "
         "host), then the summary:", "", "```", command,
         f"python3 bench.py --kernel-stats <out> {out_name} '<the command above>'", "```", "",
         f"Kernel sources hash: `{kernel_source_sha()}`",
         "", "| kernel | calls | average us | min us | max us | share % |",
         "|---|---|---|---|---|---|"]
    for name, n, avg, mn, mx, pc in rows[:25]:
        L.append(f"| `{name}` | {n} | {avg:.2f} | {mn:.2f} | {mx:.2f} | {pc:.1f} |")
    # The bench's timed steps: its two step kernels' dispatches after the
    # warm-up ones (the table above averages every call, stand-alone
    # comparisons included).
    m_steps = re.search(r"--steps (\d+)", command)
    m_warm = re.search(r"--warmup (\d+)", command)
    if m_steps and m_warm and glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        steps, warm = int(m_steps.group(1)), int(m_warm.group(1))
        trace = _trace_dispatches(d)
        L += ["", f"Timed steps (dispatches {warm + 1} to {warm + steps} of each step kernel, "
              "from the kernel trace; the bench's own figures are event-timed in its own run):",
              "", "| step kernel | dispatches | average us |", "|---|---|---|"]
        for prefix in STEP_KERNELS:
            ts = [t for n, t in trace if n.startswith(prefix)][warm:warm + steps]
            if ts:
                name = next(n for n, _ in trace if n.startswith(prefix))
                L.append(f"| `{name}` | {len(ts)} | {sum(ts) / len(ts) / 1e3:.2f} |")
    with open(os.path.join(ROOT, "profiles", out_name), "w") as f:
        f.write("\n".join(L) + "\n")
    log(f"wrote profiles/{out_name}")


# The kernels of one bench step (name prefixes as the profiler reports them):
# the online softmax of the 4000 x 32000 binary32 batch and its fused top-5.
STEP_KERNELS = ("osm::softmax_rows<float, 2, 1024, 1024,", "osm::topk_fused<float, 1, 5, 0,")

# Core counters of the fused top-k and of the projection kernels: a kernel
# trace and two counter passes per probe (each pass its own process, within
# the per-block counter limits), summarised by `--counters-summary KIND DIR`
# from DIR/stats, DIR/p0 and DIR/p1.
CORE_COUNTERS = {
    "topk": ("--topk-probe", "topk_fused_counters.md",
             ["SQ_WAVE_CYCLES SQ_BUSY_CU_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_VALU "
              "SQ_INSTS_VALU SQ_INSTS_LDS GRBM_GUI_ACTIVE",
              "SQ_ACTIVE_INST_ANY SQ_INSTS_VMEM_RD SQ_INSTS_SALU SQ_WAVES GRBM_COUNT"]),
    "proj": ("--proj-probe", "proj_4000x4096x128256_bf16.md",
             ["SQ_WAVE_CYCLES SQ_BUSY_CU_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY "
              "SQ_VALU_MFMA_BUSY_CYCLES SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_LDS "
              "GRBM_GUI_ACTIVE",
              "SQ_INSTS_MFMA SQ_INSTS_VALU SQ_INSTS_VMEM_RD TCC_HIT_sum TCC_MISS_sum GRBM_COUNT"]),
}
# the fused top-k probe's cases, in dispatch order, three calls each
TOPK_PROBE_CASES = [("4000x32000 f32", 4000, 32000, 4, 5), ("4000x32000 f32", 4000, 32000, 4, 50),
                    ("32768x128256 bf16", 32768, 128256, 2, 5),
                    ("32768x128256 bf16", 32768, 128256, 2, 50)]


def _trace_dispatches(d: str):
    """(kernel, duration ns) of every dispatch in a kernel trace under d, in
    dispatch order."""
    import csv
    files = glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_trace.csv under {d}")
    out = []
    with open(files[0], newline="") as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"].split("(")[0].strip()
            if name.startswith("void "):
                name = name[5:]
            out.append((int(r["Dispatch_Id"]), name,
                        int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    out.sort()
    return [(n, t) for _, n, t in out]


def _dispatch_counters(d: str, keep):
    """Counter values per dispatch (dict counter -> value) of the kernels
    whose name passes `keep`, in dispatch order."""
    per = {}
    for disp, name, cname, v, s, e in _counter_rows(d):
        if keep(name):
            per.setdefault(int(disp), (name, {}))[1][cname] = v
    return [per[k] for k in sorted(per)]


def counters_summary(kind: str, d: str):
    """profiles/<file> for the core counters of `kind` ('topk' or 'proj')
    from the kernel trace d/stats and the counter passes d/p0, d/p1."""
    probe, out_name, passes = CORE_COUNTERS[kind]
    cmds = [f"rocprofv3 --kernel-trace --stats -f csv -d <out>/stats -o run -- python3 bench.py "
            f"{probe}"]
    cmds += [f"rocprofv3 --pmc {c} -d <out>/p{i} -o run -f csv -- python3 bench.py {probe}"
             for i, c in enumerate(passes)]
    cmds.append(f"python3 bench.py --counters-summary {kind} <out>")
    trace = _trace_dispatches(os.path.join(d, "stats"))
    pcs = [_dispatch_counters(os.path.join(d, f"p{i}"), lambda n: n.startswith("osm::"))
           for i in range(len(passes))]

    def merged(i):  # counters of the i-th library dispatch, over both passes
        c, name = {}, None
        for p in pcs:
            name = p[i][0]
            c.update(p[i][1])
        return name, c

    L = []
    if kind == "topk":
        L += ["# Fused softmax + top-k: kernel time and core counters", "",
              "Commands (repository root, GPU host; each counter pass its own process):", "",
              "```", *cmds, "```", "", f"Kernel sources hash: `{kernel_source_sha()}`", "",
              "Three calls per case, in the order below (one wavefront per row). VALU busy =",
              "SQ_ACTIVE_INST_VALU / (4 SIMDs x SQ_BUSY_CU_CYCLES); waiting = SQ_WAIT_ANY / "
              "SQ_WAVE_CYCLES",
              "(wave cycles spent on a dependency, mostly `s_waitcnt` for loads); VALU and LDS "
              "instructions per",
              "element = wavefront instructions x 64 / elements; time from the kernel trace "
              "(median of the three).", "",
              "| case | K | kernel | us | GB/s | VALU busy | waiting | VALU instr / element | "
              "LDS instr / element |", "|---|---|---|---|---|---|---|---|---|"]
        tk = [t for n, t in trace if n.startswith("osm::topk_fused")]
        for ci, (case, N, V, es, K) in enumerate(TOPK_PROBE_CASES):
            us = median(tk[3 * ci:3 * ci + 3]) / 1e3
            rows = [merged(3 * ci + j) for j in range(3)]
            name = rows[0][0]
            m = {c: median([r[1][c] for r in rows]) for c in rows[0][1]}
            busy = m["SQ_ACTIVE_INST_VALU"] / (4 * m["SQ_BUSY_CU_CYCLES"])
            wait = m["SQ_WAIT_ANY"] / m["SQ_WAVE_CYCLES"]
            L.append(f"| {case} | {K} | `{name}` | {us:.1f} | {N * V * es / us / 1e3:.0f} | "
                     f"{100 * busy:.1f}% | {100 * wait:.1f}% | "
                     f"{m['SQ_INSTS_VALU'] * 64 / (N * V):.2f} | "
                     f"{m['SQ_INSTS_LDS'] * 64 / (N * V):.3f} |")
    else:
        N, H, V = 4000, 4096, 128256
        L += ["# Projection kernels at 4000 x 4096 x 128256 (bfloat16 h, w; binary32 "
              "accumulation)", "",
              "Commands (repository root, GPU host; each counter pass its own process):", "",
              "```", *cmds, "```", "", f"Kernel sources hash: `{kernel_source_sha()}`", "",
              "## Kernel time (3 calls of each entry point, from the kernel trace)", "",
              "| kernel | calls | avg us | min us | max us | TF/s at avg (2NHV) |",
              "|---|---|---|---|---|---|"]
        by = {}
        for n, t in trace:
            if n.startswith("osm::"):
                by.setdefault(n, []).append(t / 1e3)
        for n, ts in by.items():
            avg = sum(ts) / len(ts)
            tf = f"{2.0 * N * H * V / avg / 1e6:.0f}" if n.startswith("osm::proj") else ""
            L.append(f"| `{n}` | {len(ts)} | {avg:.1f} | {min(ts):.1f} | {max(ts):.1f} | {tf} |")
        L += ["", "## Counters per dispatch (medians over the three calls)", "",
              "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES); clock = "
              "GRBM_GUI_ACTIVE / 8 XCDs / kernel time (kernel time from the trace above).", "",
              "| kernel | MFMA busy | clock GHz | LDS bank conflict / LDS active cycles | "
              "waves waiting on counters / wave cycles | L2 hit rate |",
              "|---|---|---|---|---|---|"]
        rows = [merged(i) for i in range(len(pcs[0]))]
        names = []
        for n, _ in rows:
            if n.startswith("osm::proj") and n not in names:
                names.append(n)
        for n in names:
            rs = [c for nn, c in rows if nn == n]
            m = {c: median([r[c] for r in rs]) for c in rs[0]}
            avg_ns = sum(by[n]) / len(by[n]) * 1e3
            mfma = m["SQ_VALU_MFMA_BUSY_CYCLES"] / (4 * m["SQ_BUSY_CU_CYCLES"])
            clk = m["GRBM_GUI_ACTIVE"] / 8 / avg_ns
            bank = m["SQ_LDS_BANK_CONFLICT"] / max(m["SQ_LDS_IDX_ACTIVE"], 1.0)
            wait = m["SQ_WAIT_ANY"] / m["SQ_WAVE_CYCLES"]
            hit = m["TCC_HIT_sum"] / max(m["TCC_HIT_sum"] + m["TCC_MISS_sum"], 1.0)
            L.append(f"| `{n}` | {100 * mfma:.1f}% | {clk:.2f} | {bank:.3f} | {100 * wait:.1f}% "
                     f"| {100 * hit:.1f}% |")
        L += ["", "The clock figure is taken under the profiler (one dispatch at a time).",
              "hipBLASLt's GEMM on the same shape (bfloat16 out) runs at ~1.42 PF/s."]
    with open(os.path.join(ROOT, "profiles", out_name), "w") as f:
        f.write("\n".join(L) + "\n")
    log(f"wrote profiles/{out_name}")


def sweep(path: str):
    """Every workload shape, the paper's V sweeps at batch 4000 and 10, and
    its K sweep: one JSON record per (shape, op) into `path`.  Each record is
    the median over 10 batches of back-to-back calls queued behind a spin
    kernel (enough calls per batch that a batch runs >= ~1 ms), so small
    shapes are measured as GPU time rather than host call rate."""
    import torch
    import paper_1805_02867_amd as osm
    from paper_1805_02867_amd import synth
    stream = torch.cuda.current_stream()
    out = open(path, "w")

    def run(fn, est_us):
        # at most 64 calls per batch: they must all be enqueued within the
        # spin kernel's ~4 ms
        reps = max(1, min(64, int(1000.0 / max(est_us, 1.0))))
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        return median(queued_batches(fn, reps, 10, stream))

    def emit(rec):
        out.write(json.dumps(rec) + "\n")
        out.flush()
        log(json.dumps(rec))

    cases = [  # (name, N, V, dtype, sigma, extra)
        ("softmax_topk_16x1000_f32", 16, 1000, "f32", 1.0, {}),
        ("softmax_4000x32000_f32_shift", 4000, 32000, "f32", 2.0, {"shift_frac": 0.01}),
        ("softmax_10x1e6_f32", 10, 1_000_000, "f32", 3.0, {}),
        ("topk_4000x50000_f32_ties", 4000, 50000, "f32", 2.0, {"tie_frac": 0.01}),
        ("softmax_topk_32768x128256_bf16", 32768, 128256, "bf16", 4.0, {}),
    ]
    for V in (35, 100, 300, 1000, 3000, 4000, 10000, 25000, 100000, 500000):
        cases.append((f"sweep_4000x{V}_f32", 4000, V, "f32", 2.0, {}))
    for V in (1000, 10000, 100000, 1000000, 15000000):
        cases.append((f"sweep_10x{V}_f32", 10, V, "f32", 2.0, {}))
    topk_k = {"softmax_topk_16x1000_f32": (5,), "softmax_4000x32000_f32_shift": (5, 10),
              "topk_4000x50000_f32_ties": (5, 10), "softmax_topk_32768x128256_bf16": (5, 50)}
    algo_cases = {"softmax_4000x32000_f32_shift", "softmax_10x1e6_f32"}
    algo_cases.update(n for n, *_ in cases if n.startswith("sweep_"))
    k_sweep = {"sweep_4000x25000_f32": (5, 10, 15, 30), "softmax_4000x32000_f32_shift":
               (5, 10, 15, 30), "softmax_10x1e6_f32": (5, 10, 15, 30)}
    cases.append(("sweep_4000x25000_f32", 4000, 25000, "f32", 2.0, {}))
    # accesses per element of each softmax + top-k algorithm (Section 4)
    algo_access = {"online_fused": 1, "safe_fused": 2, "online_unfused": 4, "safe_unfused": 5}
    # inputs that fit in the 256 MB last-level cache are also timed cold
    cold_mb = 256
    scratch = torch.zeros(512 * 1024 * 1024 // 4, dtype=torch.float32, device="cuda")
    sink = torch.empty(1024, dtype=torch.float32, device="cuda")
    flush = lambda: torch.sum(scratch, dim=0, out=sink[:1].view(()))
    for name, N, V, dt, sg, extra in cases:
        x = synth.logits(N, V, sigma=sg, seed=0, dtype=dt, device="cuda", **extra)
        es = 2 if dt == "bf16" else 4
        y = torch.empty_like(x)
        est = 12.0 * N * V / 6e3 / 1e3  # us at ~6 TB/s
        modes = [("online", 3), ("safe", 4), ("naive", 3)]
        if V // (16 // es) <= osm.RESIDENT_MAX_VEC:
            modes.append(("resident", 2))
        for mode, acc in modes:
            us = run(lambda m=mode: osm.softmax_fwd(x, y, mode=m), est)
            emit({"workload": name, "op": f"softmax_{mode}", "N": N, "V": V, "dtype": dt,
                  "plan": list(osm.plan(N, V, x.dtype, mode)), "us": round(us, 2),
                  "GBps": round(acc * es * N * V / us / 1e3, 1),
                  "elements_per_s": round(N * V / us * 1e6, 1), "rows_per_s": round(N / us * 1e6, 1)})
        if name in algo_cases:
            for K in k_sweep.get(name, (5,)):
                if K > V:
                    continue
                vals = torch.empty((N, K), dtype=torch.float32, device="cuda")
                idx = torch.empty((N, K), dtype=torch.int32, device="cuda")
                t = {}
                for algo, acc in algo_access.items():
                    t[algo] = run(lambda a=algo: osm.softmax_topk(x, K, vals, idx, algo=a, y=y),
                                  est * acc / 3)
                    emit({"workload": name, "op": f"topk_{algo}_k{K}", "N": N, "V": V,
                          "dtype": dt, "us": round(t[algo], 2),
                          "elements_per_s": round(N * V / t[algo] * 1e6, 1),
                          "accesses_per_element": acc})
                emit({"workload": name, "op": f"topk_ratios_k{K}", "N": N, "V": V, "dtype": dt,
                      "safe_unfused_over_online_fused": round(t["safe_unfused"] / t["online_fused"], 3),
                      "safe_fused_over_online_fused": round(t["safe_fused"] / t["online_fused"], 3),
                      "safe_unfused_over_safe_fused": round(t["safe_unfused"] / t["safe_fused"], 3),
                      "topk_plan": list(osm.topk_plan(N, V, K, x.dtype))})
        del y
        for K in topk_k.get(name, (5,)):
            if K > V:
                continue
            vals = torch.empty((N, K), dtype=torch.float32, device="cuda")
            idx = torch.empty((N, K), dtype=torch.int32, device="cuda")
            us = run(lambda: osm.softmax_topk(x, K, vals, idx), est / 3)
            emit({"workload": name, "op": f"topk_fused_k{K}", "N": N, "V": V, "dtype": dt,
                  "us": round(us, 2), "GBps": round((es * N * V + 8 * N * K) / us / 1e3, 1),
                  "elements_per_s": round(N * V / us * 1e6, 1), "rows_per_s": round(N / us * 1e6, 1)})
        if es * N * V <= cold_mb * 1024 * 1024:
            vals = torch.empty((N, 5), dtype=torch.float32, device="cuda")
            idx = torch.empty((N, 5), dtype=torch.int32, device="cuda")
            y = torch.empty_like(x)
            for op, fn, nbytes in (
                    ("softmax_online_cold", lambda: osm.softmax_fwd(x, y), 3 * es * N * V),
                    ("topk_fused_k5_cold", lambda: osm.softmax_topk(x, 5, vals, idx),
                     es * N * V + 40 * N)):
                if op.startswith("topk") and V < 5:
                    continue
                fn()
                us = median(cold_calls(fn, 20, stream, flush))
                emit({"workload": name, "op": op, "N": N, "V": V, "dtype": dt,
                      "us": round(us, 2), "GBps": round(nbytes / us / 1e3, 1),
                      "elements_per_s": round(N * V / us * 1e6, 1)})
            del y
        del x
        torch.cuda.empty_cache()
    for N, H, V in ((64, 4096, 128256), (512, 4096, 128256), (4000, 1024, 32000),
                    (4000, 4096, 32000), (4000, 4096, 128256)):
        rec = proj_compare(osm, torch, N, H, V, 5, 10, stream)
        emit({"workload": f"proj_{N}x{H}x{V}", "op": "proj_softmax_topk_k5", **rec})
    out.close()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true")
    ap.add_argument("--proj-probe", action="store_true")
    ap.add_argument("--counters-summary", nargs=2, metavar=("KIND", "DIR"),
                    help="write the core-counter summary of KIND (topk or proj) from the "
                         "rocprofv3 outputs DIR/stats, DIR/p0 and DIR/p1")
    ap.add_argument("--topk-probe", action="store_true")
    ap.add_argument("--compare-reps", type=int, default=20)
    ap.add_argument("--traffic-probe", metavar="KEY", help="one operation of one workload "
                    "(or `copy`), for a counter pass")
    ap.add_argument("--traffic-summary", metavar="DIR", help="write profiles/traffic.json "
                    "and profiles/traffic_all_workloads.md from the counter passes under DIR")
    ap.add_argument("--sweep-summary", metavar="FILE", help="write "
                    "profiles/sweep_all_workloads.md from the records of --sweep")
    ap.add_argument("--kernel-stats", nargs=3, metavar=("DIR", "OUT", "COMMAND"),
                    help="write profiles/OUT from the rocprofv3 kernel statistics under DIR")
    ap.add_argument("--sweep", metavar="FILE", help="time every workload shape and the V "
                    "sweeps; one JSON record per line into FILE")
    args = ap.parse_args()
    if args.traffic_summary:
        traffic_summary(args.traffic_summary)
        return
    if args.sweep_summary:
        sweep_summary(args.sweep_summary)
        return
    if args.kernel_stats:
        kernel_stats_summary(*args.kernel_stats)
        return
    if args.counters_summary:
        counters_summary(*args.counters_summary)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(independent rows shard across GPUs with no communication)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_1805_02867_amd as osm
    from paper_1805_02867_amd import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    osm.lib()  # fail loudly if the HIP library is not built
    if args.copy_probe:
        copy_probe()
        return
    if args.proj_probe:
        proj_probe(osm)
        return
    if args.topk_probe:
        topk_probe(osm, synth)
        return
    if args.traffic_probe:
        traffic_probe(args.traffic_probe)
        return
    if args.sweep:
        sweep(args.sweep)
        return

    dev = torch.device("cuda:0")
    N, V, K = N_ROWS, V_LEN, K_TOP
    x = synth.logits(N, V, sigma=SIGMA, seed=0, device=dev, shift_frac=SHIFT_FRAC)
    y = torch.empty_like(x)
    vals = torch.empty((N, K), dtype=torch.float32, device=dev)
    idx = torch.empty((N, K), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    plan = osm.plan(N, V, mode="online")
    log(f"device {torch.cuda.get_device_name(0)}; plan online {plan}")

    def soft():
        osm.softmax_fwd(x, y, mode="online")

    def topk():
        osm.softmax_topk(x, K, vals, idx)

    for _ in range(args.warmup):
        soft()
        topk()
    torch.cuda.synchronize()

    # timed region: exactly `steps` steps, events around every launch
    ev_s = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps)]
    ev_t = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        ev_s[i][0].record(stream)
        soft()
        ev_s[i][1].record(stream)
        ev_t[i][0].record(stream)
        topk()
        ev_t[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_soft = [a.elapsed_time(b) for a, b in ev_s]
    ms_topk = [a.elapsed_time(b) for a, b in ev_t]
    log(f"{args.steps} steps in {wall:.3f} s")

    bytes_soft = 12.0 * N * V
    bytes_topk = 4.0 * N * V + 8.0 * N * K
    step_ms = wall * 1e3 / args.steps
    value = (bytes_soft + bytes_topk) / (step_ms * 1e-3) / 1e9
    avg_soft = sum(ms_soft) / len(ms_soft)
    avg_topk = sum(ms_topk) / len(ms_topk)
    gbs_soft = bytes_soft / (avg_soft * 1e-3) / 1e9
    gbs_topk = bytes_topk / (avg_topk * 1e-3) / 1e9

    # the paper's comparison: naive and safe on the same batch
    compare = {}
    # (and the row-resident variant, one load + one store: 8 B/element,
    # reported apart from the paper's three modes)
    for mode, nbytes in (("naive", 12.0), ("safe", 16.0), ("online", 12.0), ("resident", 8.0)):
        t = timed_calls(lambda m=mode: osm.softmax_fwd(x, y, mode=m), args.compare_reps, stream)
        compare[mode] = {"median_us": round(median(t) * 1e3, 2),
                         "p10_us": round(pct(t, 0.1) * 1e3, 2),
                         "p90_us": round(pct(t, 0.9) * 1e3, 2),
                         "algorithmic_GBps": round(nbytes * N * V / (median(t) * 1e-3) / 1e9, 1)}
    ratio = compare["safe"]["median_us"] / compare["online"]["median_us"]
    separated = compare["safe"]["p10_us"] > compare["online"]["p90_us"]

    # the paper's softmax + top-k comparison (Section 5.2) on the same batch
    algos = {}
    for algo, acc in (("online_fused", 1), ("safe_fused", 2), ("online_unfused", 4),
                      ("safe_unfused", 5)):
        t = timed_calls(lambda a=algo: osm.softmax_topk(x, K, vals, idx, algo=a, y=y),
                        args.compare_reps, stream)
        algos[algo] = {"median_us": round(median(t) * 1e3, 2),
                       "p10_us": round(pct(t, 0.1) * 1e3, 2),
                       "p90_us": round(pct(t, 0.9) * 1e3, 2),
                       "accesses_per_element": acc}
    med = {a: v["median_us"] for a, v in algos.items()}
    algos["safe_unfused_over_online_fused"] = round(med["safe_unfused"] / med["online_fused"], 3)
    algos["safe_unfused_over_safe_fused"] = round(med["safe_unfused"] / med["safe_fused"], 3)
    algos["safe_fused_over_online_fused"] = round(med["safe_fused"] / med["online_fused"], 3)

    # reference kernels on the same bytes: the library's plain streaming read
    # and copy (16-byte non-temporal, a contiguous span per wavefront), and
    # torch's copy_ and sum.  The ratios are of times: online softmax must move
    # at least what a copy moves (one read, one write per element; its second
    # read may hit in cache), fused top-k at least what a read moves.
    sink = torch.empty(1024, dtype=torch.float32, device=dev)
    tr = timed_calls(lambda: osm.ref_stream("read", x, sink), args.compare_reps, stream)
    tc = timed_calls(lambda: osm.ref_stream("copy", x, y), args.compare_reps, stream)
    ttc = timed_calls(lambda: y.copy_(x), args.compare_reps, stream)
    ttr = timed_calls(lambda: x.sum(), args.compare_reps, stream)
    read_gbs = 4.0 * N * V / (median(tr) * 1e-3) / 1e9
    copy_gbs = 8.0 * N * V / (median(tc) * 1e-3) / 1e9
    reference = {"read_GBps": round(read_gbs, 1), "copy_GBps": round(copy_gbs, 1),
                 "online_softmax_time_over_copy": round(avg_soft / median(tc), 4),
                 "fused_topk_time_over_read": round(avg_topk / median(tr), 4),
                 "torch_copy_GBps": round(8.0 * N * V / (median(ttc) * 1e-3) / 1e9, 1),
                 "torch_sum_GBps": round(4.0 * N * V / (median(ttr) * 1e-3) / 1e9, 1),
                 "kernels": "osm_ref_stream read and copy (16-byte non-temporal, a span per wavefront) "
                            "and torch copy_ / sum, over the same batch"}

    traffic = traffic_entry("softmax_online_4000x32000_f32")
    roofline = {"bound": "hbm", "achieved": round(gbs_soft, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(gbs_soft / PEAK_HBM_GBS, 4),
                "traffic": traffic}

    # projection fused with softmax + top-k (logits never leave the chip)
    # against the same projection writing logits, then the fused top-k
    projection = proj_compare(osm, torch, 4000, 1024, 32000, K, args.compare_reps, stream)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        rows = N  # the whole batch: about 10-15 core-seconds
        xh = x[:rows].cpu().numpy()
        oracle.softmax(xh[:8])  # load the library outside the timing
        t1 = time.perf_counter()
        oracle.softmax(xh)
        oracle.topk(xh, K)
        dt = time.perf_counter() - t1
        cpu_bytes = rows * V * 12.0 + rows * V * 4.0 + rows * K * 8.0
        threads = oracle.threads()
        # the same work on one core, on a smaller sample
        rows1 = 250
        oracle.set_threads(1)
        t1 = time.perf_counter()
        oracle.softmax(xh[:rows1])
        oracle.topk(xh[:rows1], K)
        dt1 = time.perf_counter() - t1
        oracle.set_threads(threads)
        cpu = {"value": round(cpu_bytes / dt / 1e9, 3), "unit": "GB/s",
               "cores": threads, "kind": "oracle",
               "sample": f"{rows} of the {N} rows (the whole batch), one step: softmax "
                         f"(Eq. 2, all rows) + top-5 by full sort, {dt:.2f} s wall",
               "rows_per_s": round(rows / dt, 1), "elements_per_s": round(rows * V / dt, 1),
               "cpu_model": cpu_model(), "nproc": len(os.sched_getaffinity(0)),
               "one_core": {"rows_per_s": round(rows1 / dt1, 1),
                            "elements_per_s": round(rows1 * V / dt1, 1),
                            "sample": f"{rows1} rows, {dt1:.2f} s wall"}}
        log(f"oracle: {dt:.2f} s for {rows} rows on {threads} threads; "
            f"{dt1:.2f} s for {rows1} rows on one")

    out = {
        "metric": "achieved HBM GB/s (% of peak) for online softmax + fused softmax+top-K rows/s",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": WORKLOAD, "N": N, "V": V, "K": K, "global_batch": N,
                   "parallelism": "none (1 GPU)"},
        "online_softmax": {"avg_us": round(avg_soft * 1e3, 2), "GBps": round(gbs_soft, 1),
                           "frac_of_peak": round(gbs_soft / PEAK_HBM_GBS, 4),
                           "rows_per_s": round(N / (avg_soft * 1e-3), 1),
                           "kernel_plan": list(plan)},
        "fused_topk": {"avg_us": round(avg_topk * 1e3, 2), "GBps": round(gbs_topk, 1),
                       "frac_of_peak": round(gbs_topk / PEAK_HBM_GBS, 4),
                       "rows_per_s": round(N / (avg_topk * 1e-3), 1)},
        "modes": compare,
        "safe_over_online": round(ratio, 3),
        "online_faster_than_safe_p10_p90_separated": bool(separated),
        "topk_algorithms": algos,
        "projection_fusion": projection,
        "reference_kernels": reference,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
