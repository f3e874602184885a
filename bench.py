"""Benchmark of the head-aware compressed-KV decode path on one MI355X.

One step = one whole image generation of the Lumina-mGPT-768-shaped workload
(batch 8, 32 layers x 32 heads, head_dim 128, 128 conditional tokens, 48x49
visual tokens, rho = 1/8, update period one row): prefill of every layer, then
for each of the 2352 visual steps and each layer the append (+ periodic
sliding-window / Stratified-Token-Eviction update), the head grouping and
budget assignment at step 299, and decode attention.  Inputs are synthetic,
seeded, and resident in HBM before timing starts.

Prints one JSON line.  `value` is visual tokens generated per second over the
whole job (batch x 2352 per step); `roofline` rates the decode-attention
kernel (the dominant one) against MI355X's 8 TB/s HBM peak with algorithmic
bytes; `cpu_baseline` times the fp64 CPU oracle on a bounded sample;
`all_layer_launch` (layouts of 256 to 1024 heads) times, outside the timed
region, the last step's attention as one launch per layer and as one launch
for all layers, which shows the per-launch share of the roofline gap;
`roofline.plain_read` is the same-size plain read in one launch on the same
box (the ceiling for one launch per layer) and the kernel's share of it.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
# the oracle's host threads: at most the GPU machine's CPU share for one GPU
CPU_THREADS_CAP = 16
METRIC = "compressed-KV decode attention tokens/s and achieved HBM GB/s (% peak), 768px shape"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--rho", default=None, help="budget ratio, e.g. 1/6 (default: the workload's)")
    p.add_argument("--workload", default="lumina_mgpt_768",
                   help="lumina_mgpt_768 (default), janus_pro_7b, lumina_mgpt_1024, "
                        "stress_768_b64_p1 or tiny")
    p.add_argument("--attn-strategy", default="varlen", choices=["varlen", "padded", "grouped"],
                   help="attention over heads of unequal length: per-head lengths (default), "
                        "every head padded to the layer's longest with a mask, or one launch "
                        "per head group")
    p.add_argument("--score-mode", default="mean_logit", choices=["mean_logit", "attn_sum"],
                   help="eviction score of global heads: Eq. 6's mean raw logit (default) or the "
                        "summed attention weights of the past-P queries")
    p.add_argument("--method", default="headkv", choices=["headkv", "uniform", "full"],
                   help="headkv (default); uniform: every head labelled global, budget rho*N "
                        "for all (the line-based baseline's uniform allocation); full: every "
                        "budget N, no eviction (full cache)")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="approximate CPU work of the oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    # every launch timed with events costs a few microseconds of the whole
    # job's time, so only every n-th step is timed; by default n is the
    # smallest stride from 64 up that is prime to the workload's update period
    # (64 at periods 49 and 65, 65 at period 24), so that the sampled steps
    # include update steps as well as the others
    p.add_argument("--timing-every", type=int, default=None,
                   help="time the launches of every n-th step (default: see timing_stride)")
    p.add_argument("--copy-probe", action="store_true",
                   help="only run a plain 512 MiB device copy five times (calibrates the HBM "
                        "byte counters of a profiler run) and exit")
    p.add_argument("--label-stability", default=None, metavar="THR,THR,...",
                   help="print, as one JSON line, how the head labels found when grouping at the "
                        "first threshold (visual tokens) change when grouping runs at the later "
                        "ones, on the GPU, and exit")
    p.add_argument("--all-layer-launch", action="store_true",
                   help="after one generation, time the attention of the last step over every "
                        "layer as one launch (headkv_decode_attn_layers) and as one launch per "
                        "layer, print one JSON line and exit (a kernel-efficiency bound: a decoder "
                        "cannot launch its layers together)")
    p.add_argument("--traffic-record", nargs=4, metavar="DIR",
                   help="write the attention kernel's traffic record from four rocprofv3 --pmc "
                        "output folders (kernel FETCH_SIZE, kernel WRITE_SIZE, copy probe "
                        "FETCH_SIZE, copy probe WRITE_SIZE) and exit; no GPU needed")
    p.add_argument("--kernel-trace-record", metavar="DIR",
                   help="write the attention kernel's per-phase duration record from a "
                        "rocprofv3 --kernel-trace output folder of the default run and exit; "
                        "no GPU needed")
    p.add_argument("--no-per-config", action="store_true",
                   help="skip the per_config field (one generation each of Lumina-768 at "
                        "rho 1/6 and 1/4, Janus-Pro-7B, Lumina-1024 and the stress shape)")
    p.add_argument("--traffic-kernel", default="k_attn<128, true, 1024, false, 8>",
                   help="kernel name the traffic record is taken for")
    p.add_argument("--traffic-out", default=None,
                   help="path of the traffic record (default: the headline kernel's under profiles/)")
    p.add_argument("--traffic-workload", default="lumina_mgpt_768_shape b8 rho=1/8",
                   help="workload label of the traffic record")
    p.add_argument("--counter-summary", nargs=2, metavar=("DIR", "KERNEL"),
                   help="print the mean per dispatch of every counter of a rocprofv3 --pmc "
                        "output folder for one kernel and exit; no GPU needed")
    return p.parse_args()


# sources of the attention kernel: the profiler's records stay valid while
# these and the flags they are compiled with are unchanged
ATTN_SOURCES = ("paper_2605_20600_amd/csrc/attn_kernels.hip",
                "paper_2605_20600_amd/csrc/attn_block.h",
                "paper_2605_20600_amd/csrc/device_common.h",
                "paper_2605_20600_amd/csrc/layout.h")
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "k_attn_lumina768_b8_rho1-8_traffic.json")


def attn_source_sha256() -> str:
    import hashlib
    from paper_2605_20600_amd import build as lib_build
    h = hashlib.sha256()
    for rel in ATTN_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    flags = lib_build.HIPCC_FLAGS + lib_build.SOURCE_FLAGS.get("attn_kernels.hip", [])
    h.update(" ".join(flags).encode())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per dispatch of the attention kernel from the profiler's byte
    counters (profiles/), or None once the kernel sources differ from the ones
    the counters were taken with."""
    try:
        rec = json.load(open(TRAFFIC_RECORD))
    except OSError:
        return None
    ok = rec.get("attn_source_sha256") == attn_source_sha256()
    return rec["traffic_bytes_per_dispatch"] if ok else None


def counter_mean(run_dir: str, kernel_substr: str, counter: str | None = None):
    """Mean value per dispatch of a counter of a rocprofv3 --pmc run (its
    counter_collection.csv), over the dispatches of the named kernel; without
    `counter`, the run must hold one counter."""
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    total, n = 0.0, 0
    with open(files[0]) as fh:
        for row in csv.DictReader(fh):
            if kernel_substr not in row.get("Kernel_Name", ""):
                continue
            if counter is not None and row.get("Counter_Name") != counter:
                continue
            total += float(row["Counter_Value"])
            n += 1
    if n == 0:
        raise SystemExit(f"no dispatch of {kernel_substr!r} in {files[0]}")
    return total / n, n


def counter_summary(run_dir: str, kernel_substr: str):
    """Mean per dispatch of every counter of a rocprofv3 --pmc run, over the
    dispatches of the named kernel, as one JSON line."""
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {run_dir}")
    names = set()
    with open(files[0]) as fh:
        for row in csv.DictReader(fh):
            if kernel_substr in row.get("Kernel_Name", ""):
                names.add(row["Counter_Name"])
    out = {"kernel": kernel_substr, "run": os.path.basename(os.path.normpath(run_dir))}
    for c in sorted(names):
        out[c], out["dispatches"] = counter_mean(run_dir, kernel_substr, c)
    print(json.dumps(out))


def write_traffic_record(dirs, kernel: str, out_path: str = TRAFFIC_RECORD,
                         workload: str = "lumina_mgpt_768_shape b8 rho=1/8"):
    """Writes a traffic record from four rocprofv3 --pmc runs: FETCH_SIZE and
    WRITE_SIZE of the kernel, then of the copy probe (whose bytes are known),
    which scale the counters to bytes."""
    fetch, n = counter_mean(dirs[0], kernel)
    write, _ = counter_mean(dirs[1], kernel)
    copy_fetch, _ = counter_mean(dirs[2], "copyBuffer")  # the runtime's copy kernel
    copy_write, _ = counter_mean(dirs[3], "copyBuffer")
    probe = 512 << 20
    fs, ws = probe / (copy_fetch * 1024), probe / (copy_write * 1024)
    rec = {
        "kernel": kernel,
        "workload": workload,
        "attn_source_sha256": attn_source_sha256(),
        "dispatches_sampled": n,
        "fetch_kib_per_dispatch": fetch,
        "write_kib_per_dispatch": write,
        "copy_probe_bytes": probe,
        "copy_fetch_kib": copy_fetch,
        "copy_write_kib": copy_write,
        "fetch_scale": fs,
        "write_scale": ws,
        "traffic_bytes_per_dispatch": fetch * 1024 * fs + write * 1024 * ws,
    }
    with open(out_path, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec))


KTRACE_RECORD = os.path.join(ROOT, "profiles", "k_attn_lumina768_b8_rho1-8_rocprof.json")


def write_kernel_trace_record(run_dir: str, layers: int = 32):
    """Per-phase durations of the decode kernels from the kernel_trace.csv of
    a rocprofv3 --kernel-trace run of this benchmark's default workload.  The
    dispatches are taken in start order: a prefill attention starts a
    generation in the full-cache phase, and the grouping step's `layers`-th
    head scoring starts its compressed phase.  The fused append + attention
    launches of each phase, and the update steps' append + update + attention
    launches, are summarised separately; the attention launches of the grouping
    step itself and of the after-run comparisons (no append) are left out.
    Written to profiles/ with the attention sources' SHA-256."""
    import csv
    import glob
    import re
    import statistics
    files = glob.glob(os.path.join(run_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_trace.csv under {run_dir}")
    rows = []
    with open(files[0]) as fh:
        for r in csv.DictReader(fh):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]))
    rows.sort()
    attn = re.compile(r"k_attn<(\d+), (true|false), (\d+), (true|false), (\d+)>")
    buckets = {"compressed_fused": [], "full_cache_fused": [], "update_attn": []}
    spans = {}
    phase, scores = None, 0
    for t0, t1, name in rows:
        if "k_prefill_attn" in name:
            phase, scores = "full_cache", 0
            continue
        if "k_score" in name:
            scores += 1
            if scores == layers:
                phase = "compressed"
            continue
        m = attn.search(name)
        key = None
        if m and m.group(2) == "true" and phase is not None:
            key = phase + "_fused"
        elif "k_update_attn<" in name and phase == "compressed":
            key = "update_attn"
        if key is None:
            continue
        buckets[key].append((t0, t1))
        if key != "full_cache_fused":
            lo, hi, n = spans.get(phase, (t0, t1, 0))
            spans[phase] = (min(lo, t0), max(hi, t1), n + 1)
    rec = {"workload": "lumina_mgpt_768_shape b8 rho=1/8 (bench.py default)",
           "attn_source_sha256": attn_source_sha256(), "layers": layers,
           "trace": os.path.basename(files[0])}
    for key, v in buckets.items():
        d = [t1 - t0 for t0, t1 in v]
        rec[key] = None if not d else {
            "calls": len(d), "avg_ns": statistics.mean(d), "median_ns": statistics.median(d),
            "min_ns": min(d), "max_ns": max(d)}
    if "compressed" in spans:
        lo, hi, n = spans["compressed"]
        busy = sum(t1 - t0 for k in ("compressed_fused", "update_attn") for t0, t1 in buckets[k])
        rec["compressed_phase"] = {"launches": n, "span_ns": hi - lo,
                                   "kernel_ns": busy, "gap_ns_per_launch": (hi - lo - busy) / n}
    with open(KTRACE_RECORD, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec))


def rocprof_roofline(alg_bytes: float):
    """The headline kernel's profiler-measured fraction of the HBM peak: the
    compressed phase's average fused-launch duration from the committed
    kernel-trace record, if that was taken with the current kernel sources."""
    try:
        rec = json.load(open(KTRACE_RECORD))
    except OSError:
        return {"frac_rocprof": None}
    c = rec.get("compressed_fused")
    if rec.get("attn_source_sha256") != attn_source_sha256() or not c:
        return {"frac_rocprof": None,
                "rocprof_note": "kernel-trace record taken with other attention sources"}
    us = c["avg_ns"] * 1e-3
    return {"frac_rocprof": alg_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS,
            "avg_launch_us_rocprof": us, "launches_rocprof": c["calls"],
            "rocprof_record": os.path.relpath(KTRACE_RECORD, ROOT)}


# The headline attention launch reads 48.5 MB of algorithmic bytes: 46 MiB.
PLAIN_READ_MIB = 46


def plain_read_ceiling(mib: int):
    """The one-launch streaming ceiling on this machine: the stream probe (built
    with the library) reads `mib` MiB in one launch of 256 x 1024 threads,
    640 times, each launch timed by its own start/stop events as the
    attention's are.  Run as a child process before this process touches the
    GPU; the kernel's share of the ceiling is added once the attention is
    measured."""
    import re
    import subprocess
    probe = os.path.join(ROOT, "paper_2605_20600_amd", "stream_probe")
    if not os.path.exists(probe):
        return None
    try:
        res = subprocess.run([probe, str(mib), "640"], capture_output=True, text=True,
                             timeout=120, check=True)
    except (subprocess.SubprocessError, OSError) as e:
        return {"error": str(e)[:200]}
    m = re.search(rf"read {mib} MB, 256 x 1024 threads\s+([0-9.]+) us per launch back to back,"
                  r"\s+([0-9.]+) us per launch from its own events", res.stdout)
    if not m:
        return {"error": "unexpected probe output"}
    b2b, own = float(m.group(1)), float(m.group(2))
    frac = mib * 2**20 / (own * 1e-6) / 1e9 / HBM_PEAK_GBPS
    return {"probe": f"stream_probe {mib} 640", "bytes": mib * 2**20,
            "us_events": own, "us_back_to_back": b2b, "frac_events": frac}


def cpu_baseline(wl, seconds_target: float):
    """The fp64 oracle through grouping, budgets and whole generations of
    sampled (layer, batch row) slices, one head per host thread (the C code
    runs without the GIL).  Inputs are generated before timing."""
    import numpy as np
    import torch
    import oracle
    from paper_2605_20600_amd import synth

    threads = min(CPU_THREADS_CAP, os.cpu_count() or 1)
    t_g = wl.group_threshold - 1
    ov = synth.budget_override(wl)

    def prepare(layer, b):
        return [synth.head_inputs(wl, layer, b, h) for h in range(wl.heads)]

    def run_slice(layer, b, inputs, pool):
        labels = []
        for (q, k, v, kc, vc) in inputs:
            g = oracle.group_head(q[t_g], torch.cat([kc, k[: t_g + 1]]), wl.tau, wl.local_window)
            labels.append(g["is_local"])
        bud = oracle.budgets(wl.budget_mode, labels, wl.num_visual, wl.row_len, wl.recent_len,
                             wl.rho, None if ov is None else ov[layer, b])

        def one(h):
            q, k, v, kc, vc = inputs[h]
            oracle.run_head(q, k, v, kc, vc, t_g, wl.period, bool(labels[h]), int(bud[h]),
                            wl.recent_len, wl.r_s)
        list(pool.map(one, range(wl.heads)))

    from concurrent.futures import ThreadPoolExecutor
    slices = [((7 * i) % wl.layers, (3 * i) % wl.batch) for i in range(wl.layers * wl.batch)]
    with ThreadPoolExecutor(max_workers=threads) as pool:
        first = prepare(*slices[0])
        t0 = time.perf_counter()
        run_slice(*slices[0], first, pool)
        per_slice = time.perf_counter() - t0
        # seconds_target is CPU time: wall per slice x threads busy
        n_slices = max(1, min(len(slices), int(seconds_target / max(per_slice * threads, 1e-9))))
        prepared = [first] + [prepare(*x) for x in slices[1:n_slices]]
        t0 = time.perf_counter()
        for x, inp in zip(slices[:n_slices], prepared):
            run_slice(*x, inp, pool)
        wall = time.perf_counter() - t0
    # the same oracle on one thread: the first slice again
    with ThreadPoolExecutor(max_workers=1) as pool1:
        t0 = time.perf_counter()
        run_slice(*slices[0], first, pool1)
        wall1 = time.perf_counter() - t0
    heads = n_slices * wl.heads
    # a visual token of the workload = one step of all layers x heads of one batch row
    tokens = heads * wl.num_visual / (wl.layers * wl.heads)
    tokens1 = wl.heads * wl.num_visual / (wl.layers * wl.heads)
    return {"value": tokens / wall, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "threads_cap": CPU_THREADS_CAP, "cpu_count": os.cpu_count(),
            "sample": (f"{n_slices} (layer, batch row) slices = {heads} heads through grouping, "
                       f"budgets and all {wl.num_visual} steps, fp64, {wall:.2f} s wall on "
                       f"{threads} threads; scaled to all {wl.layers}x{wl.heads} heads per token"),
            "single_thread": {"value": tokens1 / wall1, "unit": "tokens/s", "cores": 1,
                              "sample": f"one slice ({wl.heads} heads), {wall1:.2f} s on one thread"}}


def label_stability(wl, thresholds):
    """Labels of every (layer, batch row, head) when grouping runs at each of
    the thresholds, compared with those at the first: the synthetic analogue
    of the paper's grouping-accuracy table (Sec. 5.4).  L->G: heads local at
    the first threshold and global later; G->L: the reverse."""
    import numpy as np
    from paper_2605_20600_amd.runner import DeviceInputs, grouping_labels
    inp = DeviceInputs(wl.with_(group_threshold=max(thresholds)))
    ref = None
    rows = []
    for thr in thresholds:
        lab = grouping_labels(wl.with_(group_threshold=thr), inp)
        x = np.stack([lab[l].cpu().numpy() for l in sorted(lab)]).astype(np.int64)
        if ref is None:
            ref = x
        loc, glo = ref == 1, ref == 0
        rows.append({"threshold": thr, "local_fraction": float(x.mean()),
                     "agreement": float((x == ref).mean()),
                     "L->G": float(((x == 0) & loc).sum() / max(loc.sum(), 1)),
                     "G->L": float(((x == 1) & glo).sum() / max(glo.sum(), 1))})
        print(f"# threshold {thr}: {rows[-1]}", file=sys.stderr, flush=True)
    print(json.dumps({"workload": wl.name + "_shape", "heads": int(ref.size),
                      "reference_threshold": thresholds[0], "rows": rows}), flush=True)


def compare_layer_launches(wl, sess, inp, reps: int = 20):
    """Attention of the session's last step over all layers: one launch per
    layer (as a decoder runs it) vs one launch for all layers, same results;
    times from events on the launch stream, per layer."""
    import torch
    from paper_2605_20600_amd import binding as B
    L = wl.layers
    q = [inp.q[l][wl.num_visual - 1] for l in range(L)]
    o1 = [torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32, device="cuda")
          for _ in range(L)]
    o2 = [torch.empty_like(x) for x in o1]
    st = sess.stream()

    def per_layer():
        for l in range(L):
            B.headkv_decode_attn(sess.h, l, q[l].data_ptr(), o1[l].data_ptr(), st)

    def together():
        B.headkv_decode_attn_layers(sess.h, 0, L, [x.data_ptr() for x in q],
                                    [x.data_ptr() for x in o2], st)

    res = {}
    for name, fn in (("per_layer", per_layer), ("all_layers", together)):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / reps / L * 1e3  # us per layer
    same = max(float((a - b).abs().max()) for a, b in zip(o1, o2))
    C, d = wl.prefix_len, wl.head_dim
    tokens = 0
    for l in range(L):
        _, count = sess.export_retained(l)
        tokens += int(count.sum()) + C * wl.batch * wl.heads
    per_layer_bytes = (tokens * 2 * d * 2 + L * wl.batch * wl.heads * (2 * d + 4 * d)) / L
    gbps = lambda us: per_layer_bytes / (us * 1e-6) / 1e9
    return {"step": wl.num_visual - 1, "layers": L, "alg_bytes_per_layer": per_layer_bytes,
            "max_abs_diff": same,
            "per_layer_launch_us": res["per_layer"], "per_layer_launch_gbps": gbps(res["per_layer"]),
            "all_layers_launch_us_per_layer": res["all_layers"],
            "all_layers_launch_gbps": gbps(res["all_layers"]),
            "all_layers_launch_frac": gbps(res["all_layers"]) / HBM_PEAK_GBPS}


def all_layer_launch(wl):
    """--all-layer-launch: a fresh session through one generation, then the
    comparison of compare_layer_launches as one JSON line."""
    import torch
    from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation_native
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    outs = {l: torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32, device="cuda")
            for l in range(wl.layers)}
    run_generation_native(sess, inp, outs)
    line = {"workload": wl.name + "_shape", **compare_layer_launches(wl, sess, inp)}
    print(json.dumps(line), flush=True)


KIND_NAMES = ["k_attn<d, append> (headkv_decode_step, compressed cache)",
              "k_attn<d> (after an update)",
              "k_update<d> (append + periodic update)",
              "k_prefill_attn<d> (prefix store + causal attention, headkv_prefill_attn)",
              "k_attn<d, append> (headkv_decode_step, full cache before grouping)",
              "k_update_attn<d> (append + periodic update + attention, one launch)"]


def timing_stride(requested, period: int) -> int:
    """The stride of the timed steps: as requested, else the smallest from 64
    up that is prime to the update period (a stride sharing a factor with it
    can miss every update step: 64 and 24 at Janus and LlamaGen, whose update
    steps are all odd)."""
    if requested:
        return requested
    s = 64
    while math.gcd(s, period) != 1:
        s += 1
    return s


def launches_per_generation(wl, fused_update: bool):
    """Launches of each timed kind in one generation (all layers): the
    library times only every n-th step's launches, so the kinds' shares of a
    generation's kernel time are their average durations times these counts."""
    t_g, P, N, L = wl.group_threshold - 1, wl.period, wl.num_visual, wl.layers
    upd = sum(1 for t in range(t_g + 1, N) if (t - t_g) % P == 0)
    comp = (N - 1 - t_g) - upd
    return {0: comp * L, 1: 0 if fused_update else upd * L, 2: 0 if fused_update else upd * L,
            3: L if wl.prefix_len > 0 else 0, 4: t_g * L, 5: upd * L if fused_update else 0}


def run_workload(wl, args, steps: int, warmup: int, labels_mode: str = "headkv",
                 strategy: str = "varlen", compare_launches: bool = False, say=print):
    """Whole generations of one workload with the step loop in the library:
    warm-up, then `steps` timed generations.  Returns the per-kind kernel
    statistics, the whole-job rate and (optionally) the per-layer vs
    all-layer launch comparison."""
    import torch
    from paper_2605_20600_amd import binding as B
    from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation_native
    t0 = time.perf_counter()
    inp = DeviceInputs(wl)
    torch.cuda.synchronize()
    say(f"# {wl.name} inputs: {inp.nbytes() / 1e9:.2f} GB on device in "
        f"{time.perf_counter() - t0:.1f} s")
    labels = None
    if labels_mode == "full":
        for l in inp.layers:
            inp.override[l] = torch.full((wl.batch * wl.heads,), wl.num_visual, dtype=torch.int32,
                                         device="cuda")
    elif labels_mode == "uniform":
        labels = {l: torch.zeros(wl.batch * wl.heads, dtype=torch.uint8, device="cuda")
                  for l in inp.layers}
    sess = new_session(wl, attn_strategy=B.ATTN_STRATEGIES[strategy])
    outs = {l: torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32, device="cuda")
            for l in inp.layers}
    pre_out = {l: torch.empty((wl.batch, wl.heads, wl.prefix_len, wl.head_dim),
                              dtype=torch.float32, device="cuda") for l in inp.layers}
    for i in range(warmup):
        run_generation_native(sess, inp, outs, label_override=labels, prefill_out=pre_out)
        torch.cuda.synchronize()
        say(f"# {wl.name} warmup {i + 1}/{warmup} done")
    # timed region: whole generations, the step loop in the library.  Every
    # `timing_every`-th step's launches are timed with HIP events that take
    # the kernel's own start and end timestamps (every prefill launch too)
    te = timing_stride(args.timing_every, wl.period)
    per_gen = ((wl.num_visual + te - 1) // te * 2 + 1) * wl.layers
    B.headkv_timing_reserve(sess.h, per_gen * steps)
    B.headkv_timing_collect(sess.h)              # discard warm-up records
    torch.cuda.synchronize()
    # events between the generations, on the stream they run on, give each
    # generation's own time
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t_start = time.perf_counter()
    marks[0].record()
    for i in range(steps):
        run_generation_native(sess, inp, outs, timing_every=te,
                              label_override=labels, prefill_out=pre_out)
        marks[i + 1].record()
        say(f"# {wl.name} step {i + 1}/{steps} issued")
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    step_ms = [marks[i].elapsed_time(marks[i + 1]) for i in range(steps)]
    per_kind, dropped = B.headkv_timing_collect(sess.h)
    fused_update = per_kind[5][1] > 0
    counts = launches_per_generation(wl, fused_update)
    kinds = {}
    for k, (name, (kms, kn, kb)) in enumerate(zip(KIND_NAMES, per_kind)):
        if kn:
            avg_us = kms / kn * 1e3
            kinds[name] = {"launches_timed": kn, "avg_us": avg_us, "alg_bytes_per_launch": kb / kn,
                           "achieved_gbps": kb / kn / (avg_us * 1e-6) / 1e9,
                           "launches_per_generation": counts[k],
                           "est_ms_per_generation": avg_us * counts[k] * 1e-3}
    C, d = wl.prefix_len, wl.head_dim
    if KIND_NAMES[3] in kinds:
        k = kinds[KIND_NAMES[3]]
        k["causal_flops_per_launch"] = wl.batch * wl.heads * 4 * d * C * (C + 1) / 2
        k["achieved_tflops"] = k["causal_flops_per_launch"] / (k["avg_us"] * 1e-6) / 1e12
    total = sum(v["est_ms_per_generation"] for v in kinds.values())
    for v in kinds.values():
        v["share_of_generation_kernel_time"] = v["est_ms_per_generation"] / total
    dominant = max(kinds, key=lambda k: kinds[k]["est_ms_per_generation"])
    for k, v in kinds.items():
        say(f"# {wl.name} {k}: {v['launches_timed']} timed launches, avg {v['avg_us']:.2f} us, "
            f"{v['alg_bytes_per_launch'] / 1e6:.2f} MB algorithmic -> {v['achieved_gbps']:.0f} GB/s, "
            f"~{v['share_of_generation_kernel_time']:.1%} of a generation's kernel time")
    layers_cmp = None
    if compare_launches and 256 <= wl.batch * wl.heads <= 1024:
        layers_cmp = compare_layer_launches(wl, sess, inp)
        say(f"# last step, per layer: {layers_cmp['per_layer_launch_us']:.2f} us per launch, "
            f"{layers_cmp['all_layers_launch_us_per_layer']:.2f} us per layer in one launch")
    res = {"tokens_per_s": wl.batch * wl.num_visual * steps / elapsed,
           "elapsed_s": elapsed, "step_ms": step_ms, "kinds": kinds, "dominant": dominant,
           "dropped": dropped, "layers_cmp": layers_cmp}
    sess.close()
    del inp, outs, pre_out, sess
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


# workloads of the per_config field: the other budget ratios of the headline
# shape and the other shapes, one warm-up and one timed generation each
PER_CONFIG = (("lumina_mgpt_768", (1, 6)), ("lumina_mgpt_768", (1, 4)), ("janus_pro_7b", None),
              ("lumina_mgpt_1024", None), ("stress_768_b64_p1", None))


def per_config(args, say):
    from paper_2605_20600_amd import workloads as W
    out = []
    for name, rho in PER_CONFIG:
        wl = W.ALL[name] if rho is None else W.ALL[name].with_(rho=rho)
        r = run_workload(wl, args, steps=1, warmup=1, say=say)
        dom = r["kinds"][r["dominant"]]
        out.append({"workload": wl.name + "_shape", "batch": wl.batch,
                    "rho": f"{wl.rho[0]}/{wl.rho[1]}",
                    "budget_mode": ["paper", "override", "layer_total"][wl.budget_mode],
                    "tokens_per_s": r["tokens_per_s"], "ms_per_generation": r["step_ms"][0],
                    "kernel": r["dominant"].replace("<d", f"<{wl.head_dim}"),
                    "avg_launch_us": dom["avg_us"], "alg_bytes_per_launch": dom["alg_bytes_per_launch"],
                    "achieved_gbps": dom["achieved_gbps"],
                    "frac": dom["achieved_gbps"] / HBM_PEAK_GBPS,
                    "launches_timed": dom["launches_timed"]})
        say(f"# per_config {out[-1]}")
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the decode path "
              "shards by batch row or head with no communication, see DESIGN.md", file=sys.stderr)
        sys.exit(2)
    if args.traffic_record:
        write_traffic_record(args.traffic_record, args.traffic_kernel,
                             args.traffic_out or TRAFFIC_RECORD, args.traffic_workload)
        return
    if args.counter_summary:
        counter_summary(*args.counter_summary)
        return
    if args.kernel_trace_record:
        write_kernel_trace_record(args.kernel_trace_record)
        return
    # the headline run measures the plain-read ceiling first, as a child
    # process, before this one touches the GPU
    ceiling = None
    if (args.workload == "lumina_mgpt_768" and args.rho in (None, "1/8") and not args.copy_probe
            and args.method == "headkv" and args.attn_strategy == "varlen"
            and args.score_mode == "mean_logit" and not args.label_stability
            and not args.all_layer_launch):
        ceiling = plain_read_ceiling(PLAIN_READ_MIB)
    import torch
    if args.copy_probe:
        src = torch.empty(512 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print("# copy probe: 5 copies of 536870912 bytes", file=sys.stderr, flush=True)
        return
    from paper_2605_20600_amd import workloads as W
    from paper_2605_20600_amd import binding as B

    say = lambda m: print(m, file=sys.stderr, flush=True)
    wl = W.ALL[args.workload]
    if args.label_stability:
        label_stability(wl, [int(x) for x in args.label_stability.split(",")])
        return
    if args.all_layer_launch:
        all_layer_launch(wl)
        return
    if args.rho is not None:
        wl = wl.with_(rho=tuple(int(x) for x in args.rho.split("/")))
    if args.method == "full":
        wl = wl.with_(budget_mode=W.BUDGET_OVERRIDE)
    if args.score_mode == "attn_sum":
        wl = wl.with_(score_mode=B.HEADKV_SCORE_ATTN_SUM)
    rho_s = f"{wl.rho[0]}/{wl.rho[1]}"
    torch.cuda.set_device(torch.cuda.current_device())
    headline = (wl.name == "lumina_mgpt_768" and rho_s == "1/8" and args.method == "headkv"
                and args.attn_strategy == "varlen" and args.score_mode == "mean_logit")
    r = run_workload(wl, args, args.steps, args.warmup, labels_mode=args.method,
                     strategy=args.attn_strategy,
                     compare_launches=args.method == "headkv" and args.attn_strategy == "varlen",
                     say=say)
    print(f"# {r['dropped']} launches untimed", file=sys.stderr, flush=True)
    kinds, dominant = r["kinds"], r["dominant"]
    dom = kinds[dominant]
    achieved = dom["achieved_gbps"]

    cfgs = None
    if headline and not args.no_per_config:
        cfgs = per_config(args, say)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_seconds)

    roof = {
        "bound": "hbm",
        "achieved": achieved,
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": achieved / HBM_PEAK_GBPS,
        "traffic": (measured_traffic() if headline and dominant == KIND_NAMES[0] else None),
        "kernel": dominant.replace("<d", f"<{wl.head_dim}"),
        "frac_events": achieved / HBM_PEAK_GBPS,
        "timed_every_nth_step": timing_stride(args.timing_every, wl.period),
        "launches": dom["launches_timed"],
        "avg_launch_us": dom["avg_us"],
        "alg_bytes_per_launch": dom["alg_bytes_per_launch"],
    }
    if headline and dominant == KIND_NAMES[0]:
        roof.update(rocprof_roofline(dom["alg_bytes_per_launch"]))
        if ceiling and "frac_events" in ceiling:
            ceiling["kernel_share"] = roof["frac_events"] / ceiling["frac_events"]
        roof["plain_read"] = ceiling
    line = {
        "metric": METRIC,
        "value": r["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["elapsed_s"] / args.steps * 1e3,
        "ms_per_step_each": r["step_ms"],
        "ms_per_step_median": sorted(r["step_ms"])[len(r["step_ms"]) // 2],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": wl.name + "_shape",
            "step": (f"one whole generation: prefill, {wl.num_visual} visual steps x "
                     f"{wl.layers} layers of append/update + grouping at step "
                     f"{wl.group_threshold - 1} + decode attention"),
            "batch": wl.batch, "layers": wl.layers, "heads": wl.heads,
            "head_dim": wl.head_dim, "prefix_tokens": wl.prefix_len,
            "visual_tokens": wl.num_visual, "rho": rho_s,
            "budget_mode": ["paper", "override", "layer_total"][wl.budget_mode],
            "method": args.method, "attn_strategy": args.attn_strategy,
            "score_mode": args.score_mode,
            "period": wl.period,
            "group_threshold": wl.group_threshold, "recent_window": wl.recent_len,
            "kv_storage": "bf16", "accumulate": "fp32 (attention), fp64 (grouping, eviction)",
        },
        "roofline": roof,
        "cpu_baseline": cpu,
        "per_config": cfgs,
        "all_layer_launch": r["layers_cmp"],
        "kernels": {k.replace("<d", f"<{wl.head_dim}"): v for k, v in kinds.items()},
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
