#!/usr/bin/env python3
"""Benchmark: one bifurcated decode-attention step per timed step on MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

A step is one bifattn_decode call (context partials, decode partials and the
combine) over one batch of seeded synthetic inputs that are already resident
in HBM (bifattn_decode_scaled for the workloads with 8-bit or 4-bit KV
caches, whose bytes count one or one half per element). Steps rotate over several device copies of the inputs (about 1.2 GB
or more in total) so that no step finds its KV cache in the 256 MB Infinity
Cache left behind by the previous one. The timed region is bracketed by
torch.cuda.synchronize() on both sides.

Prints ONE JSON line: value = algorithmic KV bytes per step (one copy of the
context K/V plus every sample's valid decode K/V, Section 4.3) divided by the
measured time per step, in GB/s. ``roofline`` reports the dominant kernel
against its own roof, its duration measured with HIP events that the
library's launch records with the kernel itself (hipExtLaunchKernel
start/stop events, the span a kernel trace shows), over further passes of the
same steps (kept out of the value loop, where no events are recorded): on
the few-row path the partial launch (context and decode work-groups) against
the 8 TB/s HBM peak; on the many-row path the longer of the many-row context
kernel (against the 2.5 PFLOP/s dense bf16 matrix peak, with the context's
flops) and the decode launch (against HBM, with the decode bytes).
``roofs`` gives the whole step against both peaks. ``extra.call_us`` gives the 10th, 50th and 90th percentiles of
single calls timed with events on the call's stream around each call.
``cpu_baseline`` times the fp64 CPU oracle on the host on the same workload
(all threads; ``single_thread``: one thread over the first samples; the CPU
model). ``ablation`` times the replicated-KV kernel (no bifurcation).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads  # noqa: E402

METRIC = ("decode-step attention µs and achieved HBM GB/s (% of peak), "
          "b=32 m_c=8k MHA")
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 matrix peak of MI355X
MALL_BYTES = 256 << 20
KERNEL_SRC = os.path.join(ROOT, "paper_2403_08845_amd", "csrc", "bifattn_kernels.hip")
TRAFFIC_DIR = os.path.join(ROOT, "profiles")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the kernel source's code: line comments, trailing blanks and
    empty lines removed, so that editing a comment keeps a counter record."""
    code = []
    for line in open(KERNEL_SRC, encoding="utf-8"):
        line = line.split("//", 1)[0].rstrip()
        if line:
            code.append(line)
    return hashlib.sha256("\n".join(code).encode()).hexdigest()[:16]


def measured_traffic(workload: str, kernel: str = "partials"):
    """HBM bytes per launch of a kernel ("partials": the partial launch;
    "ctx_large": the many-row context kernel) from the committed rocprofv3
    counter summary, or None when it is missing or the kernel source changed
    since the counters were taken."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def to_device(x):
    """q as bf16; caches as bf16, or as uint8 codes with fp32 scales."""
    import torch
    kv = x.get("kv", "bf16")
    out = {}
    for k in ("q", "Kc", "Vc", "Kd", "Vd"):
        a = np.ascontiguousarray(x[k])
        if k == "q" or kv == "bf16":
            out[k] = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        else:
            out[k] = torch.from_numpy(a.view(np.uint8)).cuda()
    out["lens"] = torch.from_numpy(np.ascontiguousarray(x["lens"], dtype=np.int32)).cuda()
    for k in ("k_scale", "v_scale"):
        if k in x:
            out[k] = torch.from_numpy(np.ascontiguousarray(x[k], dtype=np.float32)).cuda()
    return out


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(x, w, min_seconds, single_thread=True):
    """The fp64 oracle on the host's cores, repeated over the whole workload
    until min_seconds have elapsed (at least once); then one pass on a single
    thread, over the sample rows the same number of seconds allow."""
    import oracle
    threads = oracle.max_threads()
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.attention(**x, nthreads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    per = el / reps
    B = workloads.kv_bytes(w.g, w.d, w.m_c, x["lens"], w.kv)
    rec = {"value": round(B / per / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
           "sample": f"whole {w.name} step (b={w.b}), fp64, repeated {reps}x over {el:.1f} s; "
                     f"{per * 1e3:.1f} ms per step",
           "cpu_model": cpu_model()}
    if single_thread:
        # Single thread over the first samples: their rows cost about
        # per * threads seconds per step, so take a share that fits.
        nb = max(1, min(w.b, int(w.b * min_seconds / max(per * threads, 1e-9))))
        xs = workloads.first_samples(x, nb)
        t0 = time.perf_counter()
        oracle.attention(**xs, nthreads=1)
        el1 = time.perf_counter() - t0
        B1 = workloads.kv_bytes(w.g, w.d, w.m_c, xs["lens"], w.kv)
        rec["single_thread"] = {"value": round(B1 / el1 / 1e9, 4), "unit": "GB/s",
                                "sample": f"first {nb} of {w.b} samples, one pass, {el1:.1f} s"}
        oracle.attention(**workloads.first_samples(x, 1), nthreads=threads)  # thread count back
    return rec


COPY_BYTES = 1 << 30


def calibrate_copy(reps: int = 5):
    """A copy-equivalent elementwise kernel over COPY_BYTES (torch.neg on
    float32: reads COPY_BYTES, writes COPY_BYTES), the reference for the HBM
    counters: FETCH_SIZE and WRITE_SIZE should each read COPY_BYTES per
    dispatch. A kernel of its own name, so that it is not confused with the
    blit kernels of host uploads."""
    import torch
    a = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(reps):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    del a, b
    log(f"[bench] copy-equivalent kernel over {COPY_BYTES} bytes, {reps} times")


KERNEL_NAMES = {"partials": "partials_kernel", "ctx_large": "ctx_large_kernel",
                "ctx_wide": "ctx_wide_kernel", "standard": "standard_kernel"}


def summarize_profile(stats_dir: str, fetch_dir: str, write_dir: str, workload: str, out_dir: str,
                      warmup: int, steps: int, kernel: str = "partials"):
    """Turn rocprofv3 outputs into the committed summary: the kernel-trace
    statistics, and one kernel's HBM traffic per launch ("partials": the
    partial launch, "ctx_large": the many-row context kernel) from the two
    counter runs, each scaled by what the same counter reads for the plain
    copy of COPY_BYTES."""
    kname = KERNEL_NAMES[kernel]
    import csv
    import glob

    def rows(d, pattern):
        files = glob.glob(os.path.join(d, "**", pattern), recursive=True)
        if not files:
            raise SystemExit(f"no {pattern} under {d}")
        return list(csv.DictReader(open(files[0])))

    stats = rows(stats_dir, "*kernel_stats.csv")
    # The partial kernel's launches in dispatch order: warmup, value loop,
    # event-timed loop, warm loop, ...; average the event-timed ones.
    trace = [r for r in rows(stats_dir, "*kernel_trace.csv") if kname in r["Kernel_Name"]]
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    timed_us = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in trace) / len(trace) / 1e3

    def per_kernel(d, counter):
        acc = {}
        for r in rows(d, "*counter_collection.csv"):
            if r.get("Counter_Name") != counter:
                continue
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return acc

    fetch, write = per_kernel(fetch_dir, "FETCH_SIZE"), per_kernel(write_dir, "WRITE_SIZE")

    def pick(acc, key):
        for name, vals in acc.items():
            if key(name):
                return name, sum(vals) / len(vals), len(vals)
        raise SystemExit(f"kernel not found in counters: {list(acc)}")

    is_copy = lambda n: "neg" in n.lower()
    is_part = lambda n: kname in n
    _, copy_fetch_kib, _ = pick(fetch, is_copy)
    _, copy_write_kib, _ = pick(write, is_copy)
    pname, part_fetch_kib, nf = pick(fetch, is_part)
    _, part_write_kib, nw = pick(write, is_part)
    f_scale = COPY_BYTES / (copy_fetch_kib * 1024.0)
    w_scale = COPY_BYTES / (copy_write_kib * 1024.0)
    fetch_b = part_fetch_kib * 1024.0 * f_scale
    write_b = part_write_kib * 1024.0 * w_scale
    rec = {"workload": workload, "kernel": pname, "kernel_source_sha256_16": kernel_source_hash(),
           "fetch_size_kib_per_dispatch": part_fetch_kib, "write_size_kib_per_dispatch": part_write_kib,
           "dispatches": [nf, nw], "copy_fetch_kib": copy_fetch_kib, "copy_write_kib": copy_write_kib,
           "copy_bytes": COPY_BYTES, "fetch_scale": f_scale, "write_scale": w_scale,
           "hbm_fetch_bytes_per_launch": fetch_b, "hbm_write_bytes_per_launch": write_b,
           "hbm_bytes_per_launch": fetch_b + write_b,
           "trace_avg_us_all_launches": timed_us}
    os.makedirs(out_dir, exist_ok=True)
    json.dump(rec, open(os.path.join(out_dir, f"traffic_{kernel}_{workload}.json"), "w"), indent=1)
    lines = [f"# rocprofv3 kernel statistics, {workload}", "",
             "| kernel | calls | avg us | min us | max us | % time |", "|---|---|---|---|---|---|"]
    for r in stats:
        lines.append(f"| {r['Name'][:90]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f} |")
    lines += ["", f"`{pname}` over all {len(trace)} launches of the run: average {timed_us:.2f} us."]
    lines += ["", f"HBM traffic of `{pname}` per launch (FETCH_SIZE / WRITE_SIZE, scaled by a "
              f"{COPY_BYTES}-byte copy: fetch x{f_scale:.4f}, write x{w_scale:.4f}): "
              f"{fetch_b / 1e6:.2f} MB read, {write_b / 1e6:.2f} MB written."]
    alg = algorithmic_read_bytes(workload, kernel)
    if alg:
        what, nbytes = alg
        lines += ["", f"Algorithmic bytes this kernel must read ({what}): {nbytes / 1e6:.2f} MB; "
                  f"measured read / algorithmic = {fetch_b / nbytes:.3f}."]
    head = [f"# {kname}, {workload}", "",
            "Commands (repository root, one MI355X, after `cd /tmp && export TMPDIR=/tmp`; "
            "the directories hold the raw rocprofv3 output):", "", "```",
            f"rocprofv3 --kernel-trace --stats -d {stats_dir} -o run --output-format csv "
            f"-- python -u bench.py --workload {workload} --steps {steps} --warmup {warmup} "
            f"--no-cpu-baseline --no-ablation",
            f"rocprofv3 --pmc FETCH_SIZE -d {fetch_dir} -o run --output-format csv -- python -u "
            f"bench.py --workload {workload} --steps 5 --warmup 2 --no-cpu-baseline --no-ablation "
            f"--calibrate-copy",
            f"rocprofv3 --pmc WRITE_SIZE -d {write_dir} -o run --output-format csv -- python -u "
            f"bench.py --workload {workload} --steps 5 --warmup 2 --no-cpu-baseline --no-ablation "
            f"--calibrate-copy",
            f"python bench.py --workload {workload} --steps {steps} --warmup {warmup} --kernel {kernel} "
            f"--summarize-profile {stats_dir} {fetch_dir} {write_dir} {out_dir}",
            "```", ""]
    open(os.path.join(out_dir, f"{kernel}_{workload}.md"), "w").write("\n".join(head + lines) + "\n")
    print("\n".join(lines))
    return lines


def algorithmic_read_bytes(workload: str, kernel: str):
    """(description, bytes) of the KV a kernel must read once for the
    workload: the context chunk of every group for the many-row context
    kernels, the valid decode rows for the decode launch of a many-row plan,
    both for the few-row partial launch; None for unknown workloads."""
    w = workloads.WORKLOADS.get(workload)
    if w is None:
        return None
    rb = workloads.row_bytes(w.d, w.kv)
    ctx = 2 * rb * w.g * w.m_c
    if kernel in ("ctx_large", "ctx_wide"):
        return "one copy of the context K and V", ctx
    lens = workloads.make_workload_lens(w)
    dec = 2 * rb * w.g * int(np.sum(lens, dtype=np.int64))
    if w.b * (w.h // w.g) * w.n > 64:
        return "every sample's valid decode K and V", dec
    return "one copy of the context K and V plus every sample's valid decode K and V", ctx + dec


def summarize_stats(stats_dir: str, workload: str, out_dir: str):
    """Kernel-trace statistics of one rocprofv3 run of this script as a
    markdown table (profiles/stats_<workload>.md)."""
    import csv
    import glob
    files = glob.glob(os.path.join(stats_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {stats_dir}")
    lines = [f"| kernel | calls | avg us | min us | max us | % time |", "|---|---|---|---|---|---|"]
    for r in csv.DictReader(open(files[0])):
        lines.append(f"| {r['Name'][:110]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f} |")
    w = workloads.WORKLOADS[workload]
    head = [f"# rocprofv3 kernel statistics, {workload}", "",
            f"b={w.b}, h={w.h}, g={w.g}, d={w.d}, m_c={w.m_c}, m_d={w.m_d_max}, "
            f"new tokens {w.n}, KV {w.kv}, lengths {'ragged' if w.ragged else 'uniform'}.", "",
            "Commands (repository root, one MI355X, after `cd /tmp && export TMPDIR=/tmp`; "
            f"`{stats_dir}` holds the raw output):", "", "```",
            f"rocprofv3 --kernel-trace --stats -d {stats_dir} -o run --output-format csv "
            f"-- python -u bench.py --workload {workload} --steps 100 --no-cpu-baseline --no-ablation",
            f"python bench.py --workload {workload} --summarize-stats {stats_dir} {out_dir}",
            "```", "", "Every launch of the run (warmup, timed loop, event-timed loop, per-call loop, warm loop).", ""]
    os.makedirs(out_dir, exist_ok=True)
    text = "\n".join(head + lines) + "\n"
    open(os.path.join(out_dir, f"stats_{workload}.md"), "w").write(text)
    print(text)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=workloads.HEADLINE, choices=workloads.WORKLOAD_ORDER)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ablation", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="first run the 1 GiB copy-equivalent kernel that scales HBM counters")
    ap.add_argument("--summarize-profile", nargs=4, metavar=("STATS", "FETCH", "WRITE", "OUT"),
                    help="summarize rocprofv3 outputs of the workload into OUT")
    ap.add_argument("--kernel", default="partials", choices=sorted(KERNEL_NAMES),
                    help="kernel whose counters --summarize-profile records")
    ap.add_argument("--summarize-stats", nargs=2, metavar=("STATS", "OUT"),
                    help="write the kernel statistics of a rocprofv3 run of the workload into OUT")
    args = ap.parse_args()
    if args.summarize_stats:
        summarize_stats(args.summarize_stats[0], args.workload, args.summarize_stats[1])
        return
    if args.summarize_profile:
        summarize_profile(*args.summarize_profile[:3], args.workload, args.summarize_profile[3],
                          args.warmup, args.steps, args.kernel)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the bifurcated decode step runs on a single MI355X "
              "(the sample axis and the KV groups are the axes a multi-GPU layout would split); "
              "--gpus must be 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2403_08845_amd as bif

    if args.calibrate_copy:
        calibrate_copy()
    w = workloads.WORKLOADS[args.workload]
    log(f"[bench] generating {w.name}")
    x = workloads.make_workload_inputs(w)
    B_kv = workloads.kv_bytes(w.g, w.d, w.m_c, x["lens"], w.kv)
    flops = workloads.attention_flops(w.h, w.d, w.b, w.m_c, x["lens"], n=w.n)
    torch.cuda.set_device(0)
    dev0 = to_device(x)
    # Rotate over device copies so each step's KV is cold in the Infinity Cache.
    copies = min(512, max(3, -(-4 * MALL_BYTES // B_kv)))
    devs = [dev0] + [{k: v.clone() for k, v in dev0.items()} for _ in range(copies - 1)]
    out = torch.empty(tuple(x["q"].shape), dtype=torch.float32, device="cuda")
    plan = bif.Plan(w.b, w.h, w.g, w.d, w.m_c, w.m_d_max, n=w.n, kv=w.kv)
    info = plan.info()
    log(f"[bench] plan {info}, {copies} input copies")

    def step(k):
        d = devs[k % copies]
        if w.kv == "bf16":
            bif.bifattn_decode(plan, d["q"], d["Kc"], d["Vc"], d["Kd"], d["Vd"], d["lens"], out)
        else:
            bif.bifattn_decode_scaled(plan, d["q"], d["Kc"], d["Vc"], d["Kd"], d["Vd"], d["lens"],
                                      d["k_scale"], d["v_scale"], out)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    assert bif.bifattn_plan_status(plan) == bif.OK
    log(f"[bench] warmup done ({args.warmup} steps)")

    # Timed region (value, ms_per_step): plain back-to-back steps.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(k)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps
    # Kernel timing (roofline): the same steps again, the library's launch
    # recording start/stop events with the selected kernel in every step.
    def timed_pass(kernel):
        bif.bifattn_plan_set_timing(plan, kernel, args.steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for k in range(args.steps):
            step(k)
        torch.cuda.synchronize()
        loop_us = (time.perf_counter() - t0) * 1e6 / args.steps
        n_timed, ms = bif.bifattn_plan_read_timing(plan)
        bif.bifattn_plan_set_timing(plan, kernel, 0)
        assert n_timed == args.steps
        return ms * 1e3 / n_timed, loop_us

    part_us, evt_loop_us = timed_pass(bif.KERNEL_PARTIALS)
    many_rows = w.b * (w.h // w.g) * w.n > 64 and info["path"] == bif.PATHS["bifurcated"]
    ctx_us = dec_us = None
    if many_rows:
        ctx_us, _ = timed_pass(bif.KERNEL_CONTEXT)
        if w.m_d_max > 0:
            dec_us, _ = timed_pass(bif.KERNEL_DECODE)
    log(f"[bench] timed {args.steps} steps: {ms_per_step * 1e3:.2f} us/step, "
        f"partial section {part_us:.2f} us, context kernel {ctx_us} us, decode launch {dec_us} us "
        f"(event loop {evt_loop_us:.2f} us/step)")

    # Per-call latency distribution: events on the call's stream around each
    # call (the whole call: partial and combine launches).
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for k in range(args.steps):
        starts[k].record()
        step(k)
        ends[k].record()
    torch.cuda.synchronize()
    call_us = np.sort([a.elapsed_time(b) * 1e3 for a, b in zip(starts, ends)])
    call_stats = {q: round(float(np.percentile(call_us, pct)), 3)
                  for q, pct in (("p10", 10), ("median", 50), ("p90", 90))}

    # Warm variant (same inputs every step: KV partly served by the Infinity Cache).
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(0)
    torch.cuda.synchronize()
    warm_us = (time.perf_counter() - t0) * 1e6 / args.steps

    extra = {"warm_us_per_step": round(warm_us, 3), "event_loop_us_per_step": round(evt_loop_us, 3),
             "call_us": call_stats,
             "plan": info, "input_copies": copies,
             "kv_bytes_per_step": B_kv, "flops_per_step": flops}

    ablation = None
    if not args.no_ablation:
        # Replicated cache built on the device: every sample's own copy of the context.
        rows = w.m_c + w.m_d_max
        rep_bytes = 2 * w.b * w.g * rows * workloads.row_bytes(w.d, w.kv)
        if rep_bytes < 40e9:
            K = torch.cat([dev0["Kc"].unsqueeze(0).expand(w.b, -1, -1, -1), dev0["Kd"]], dim=2).contiguous()
            V = torch.cat([dev0["Vc"].unsqueeze(0).expand(w.b, -1, -1, -1), dev0["Vd"]], dim=2).contiguous()
            ref_out = out.clone()
            ks, vs = dev0.get("k_scale"), dev0.get("v_scale")
            bif.bifattn_decode_replicated_scaled(plan, dev0["q"], K, V, dev0["lens"], ks, vs, out)
            torch.cuda.synchronize()
            rep_steps = max(5, args.steps // 10)
            t0 = time.perf_counter()
            for _ in range(rep_steps):
                bif.bifattn_decode_replicated_scaled(plan, dev0["q"], K, V, dev0["lens"], ks, vs,
                                                     out)
            torch.cuda.synchronize()
            rep_us = (time.perf_counter() - t0) * 1e6 / rep_steps
            B_rep = workloads.replicated_kv_bytes(w.b, w.g, w.d, w.m_c, x["lens"], w.kv)
            step(0)
            torch.cuda.synchronize()
            ablation = {"kernel": "bifattn_decode_replicated", "us_per_step": round(rep_us, 3),
                        "kv_bytes_per_step": B_rep,
                        "GBps": round(B_rep / (rep_us * 1e-6) / 1e9, 1),
                        "speedup_of_bifurcation": round(rep_us / (ms_per_step * 1e3), 3)}
            del K, V, ref_out
    plan.close()

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle")
        cpu = cpu_baseline(x, w, args.cpu_seconds)

    value = B_kv / (ms_per_step * 1e-3) / 1e9
    ctx_bytes = 2 * workloads.row_bytes(w.d, w.kv) * w.g * w.m_c
    dec_bytes = B_kv - ctx_bytes
    ctx_flops = 4 * w.h * w.n * w.d * w.b * w.m_c
    if many_rows and (dec_us is None or ctx_us >= dec_us):
        # The many-row context kernel: a contraction over b*p*n rows per group.
        tflops = ctx_flops / (ctx_us * 1e-6) / 1e12
        ck = "ctx_wide" if info.get("ctx_kernel") == 2 else "ctx_large"
        roofline = {"kernel": f"{KERNEL_NAMES[ck]} (many-row context partials)", "bound": "mfma",
                    "achieved": round(tflops, 1), "peak": MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tflops / MFMA_PEAK_TFLOPS, 4),
                    "traffic": measured_traffic(w.name, ck),
                    "avg_launch_us": round(ctx_us, 3), "flops_per_launch": ctx_flops,
                    "bytes_per_launch": ctx_bytes}
    elif many_rows:
        gbs = dec_bytes / (dec_us * 1e-6) / 1e9
        roofline = {"kernel": "partials_kernel (decode partials)", "bound": "hbm",
                    "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4),
                    "traffic": measured_traffic(w.name, "partials"),
                    "avg_launch_us": round(dec_us, 3), "bytes_per_launch": dec_bytes}
    else:
        # One launch: the few-row partial kernel, or the standard kernel where
        # the plan takes the standard path.
        standard = info["path"] == bif.PATHS["standard"]
        kname = "standard" if standard else "partials"
        what = "whole attention, rows written directly" if standard else "context + decode partials"
        gbs = B_kv / (part_us * 1e-6) / 1e9
        roofline = {"kernel": f"{KERNEL_NAMES[kname]} ({what})", "bound": "hbm",
                    "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4),
                    "traffic": measured_traffic(w.name, kname),
                    "avg_launch_us": round(part_us, 3), "bytes_per_launch": B_kv}
    step_s = ms_per_step * 1e-3
    roofs = {"hbm_frac_step": round(B_kv / step_s / 1e9 / HBM_PEAK_GBS, 4),
             "mfma_frac_step": round(flops / step_s / 1e12 / MFMA_PEAK_TFLOPS, 4),
             "hbm_time_us": round(B_kv / (HBM_PEAK_GBS * 1e9) * 1e6, 3),
             "mfma_time_us": round(flops / (MFMA_PEAK_TFLOPS * 1e12) * 1e6, 3)}
    extra["kernel_us"] = {"partial_section": round(part_us, 3),
                          "context": None if ctx_us is None else round(ctx_us, 3),
                          "decode": None if dec_us is None else round(dec_us, 3)}
    rec = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "us_per_step": round(ms_per_step * 1e3, 3),
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # bf16 caches: bf16 products, fp32 accumulation; 8-bit caches: the
        # codes, widened exactly to bf16 for the same products.
        "dtype": w.kv,
        "data": "synthetic",
        "config": {"workload": w.name, "b": w.b, "h": w.h, "g": w.g, "d": w.d, "m_c": w.m_c,
                   "m_d": w.m_d_max, "new_tokens": w.n, "kv_cache": w.kv,
                   "decode_lens": "ragged" if w.ragged else "uniform",
                   "parallelism": "single GPU"},
        "roofline": roofline,
        "roofs": roofs,
        "cpu_baseline": cpu,
        "ablation": ablation,
        "extra": extra,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
