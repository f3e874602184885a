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
bytes; `cpu_baseline` times the fp64 CPU oracle on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "compressed-KV decode attention tokens/s and achieved HBM GB/s (% peak), 768px shape"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--rho", default="1/8")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="approximate CPU work of the oracle sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--timing-every", type=int, default=16,
                   help="time the attention launch of every n-th step")
    p.add_argument("--copy-probe", action="store_true",
                   help="only run a plain 512 MiB device copy five times (calibrates the HBM "
                        "byte counters of a profiler run) and exit")
    return p.parse_args()


def measured_traffic():
    """HBM bytes per dispatch of the attention kernel from the profiler's byte
    counters (profiles/), or None once the kernel source differs from the one
    the counters were taken with."""
    import hashlib
    rec_path = os.path.join(ROOT, "profiles", "k_attn_lumina768_b8_rho1-8_traffic.json")
    src = os.path.join(ROOT, "paper_2605_20600_amd", "csrc", "kernels.hip")
    try:
        rec = json.load(open(rec_path))
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    return rec["traffic_bytes_per_dispatch"] if rec.get("kernels_hip_sha256") == sha else None


def cpu_baseline(wl, seconds_target: float):
    """The fp64 oracle through whole generations of a sample of heads, one head
    per host thread (the C code runs without the GIL)."""
    import numpy as np
    import torch
    import oracle
    from paper_2605_20600_amd import synth

    threads = min(16, os.cpu_count() or 1)
    t_g = wl.group_threshold - 1
    # calibrate on one head: grouping + the whole generation
    q, k, v, kc, vc = synth.head_inputs(wl, 0, 0, 0)
    t0 = time.perf_counter()
    oracle.group_head(q[t_g], torch.cat([kc, k[: t_g + 1]]), wl.tau, wl.local_window)
    oracle.run_head(q, k, v, kc, vc, t_g, wl.period, False,
                    wl.num_visual * wl.rho[0] // wl.rho[1], wl.recent_len)
    per_head = time.perf_counter() - t0
    n_heads = max(threads, int(round(seconds_target / per_head / threads)) * threads)
    heads = [(l % wl.layers, (l // wl.layers) % wl.batch, (7 * l) % wl.heads) for l in range(n_heads)]
    inputs = [synth.head_inputs(wl, *x) for x in heads]
    amp = synth.amplitudes(wl)
    budgets = {True: wl.recent_len, False: wl.num_visual * wl.rho[0] // wl.rho[1]}
    lock = threading.Lock()
    todo = list(range(n_heads))

    def work():
        while True:
            with lock:
                if not todo:
                    return
                i = todo.pop()
            q, k, v, kc, vc = inputs[i]
            g = oracle.group_head(q[t_g], torch.cat([kc, k[: t_g + 1]]), wl.tau, wl.local_window)
            loc = bool(g["is_local"])
            oracle.run_head(q, k, v, kc, vc, t_g, wl.period, loc, budgets[loc], wl.recent_len)

    t0 = time.perf_counter()
    ths = [threading.Thread(target=work) for _ in range(threads)]
    for th in ths:
        th.start()
    for th in ths:
        th.join()
    wall = time.perf_counter() - t0
    # a visual token of the workload = one step of all layers x heads of one batch row
    tokens = n_heads * wl.num_visual / (wl.layers * wl.heads)
    local = sum(int(amp[l, b, h] == 3.0) for (l, b, h) in heads)
    return {"value": tokens / wall, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"{n_heads} (layer, batch, head) heads ({local} planted local) through "
                       f"grouping + all {wl.num_visual} steps, fp64, {wall:.2f} s wall on "
                       f"{threads} threads; scaled to all {wl.layers}x{wl.heads} heads per token")}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the decode path "
              "shards by batch row or head with no communication, see DESIGN.md", file=sys.stderr)
        sys.exit(2)
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
    from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation_native

    rho = tuple(int(x) for x in args.rho.split("/"))
    wl = W.LUMINA768.with_(rho=rho)
    dev = torch.cuda.current_device()
    torch.cuda.set_device(dev)
    t0 = time.perf_counter()
    inp = DeviceInputs(wl)
    torch.cuda.synchronize()
    print(f"# inputs: {inp.nbytes() / 1e9:.2f} GB on device in {time.perf_counter() - t0:.1f} s",
          file=sys.stderr, flush=True)
    sess = new_session(wl)
    outs = {l: torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32, device="cuda")
            for l in inp.layers}

    for i in range(args.warmup):
        run_generation_native(sess, inp, outs)
        torch.cuda.synchronize()
        print(f"# warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)

    # timed region: K whole generations, the step loop in the library.  Every
    # `timing_every`-th step's fused append + attention launch (one kernel) is
    # timed with HIP events that take the kernel's own start and end.
    per_gen = (wl.num_visual + args.timing_every - 1) // args.timing_every * wl.layers
    B.headkv_timing_reserve(sess.h, per_gen * args.steps)
    B.headkv_timing_collect(sess.h)              # discard warm-up records
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        run_generation_native(sess, inp, outs, timing_every=args.timing_every)
        print(f"# step {i + 1}/{args.steps} issued", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    kern_ms, n_launch, bytes_sum, dropped = B.headkv_timing_collect(sess.h)
    avg_us = kern_ms / n_launch * 1e3
    avg_bytes = bytes_sum / n_launch
    achieved = avg_bytes / (avg_us * 1e-6) / 1e9
    tokens = wl.batch * wl.num_visual * args.steps
    ms_per_step = elapsed / args.steps * 1e3
    print(f"# attention: {n_launch} timed launches ({dropped} untimed), avg {avg_us:.2f} us, "
          f"{avg_bytes / 1e6:.2f} MB algorithmic -> {achieved:.0f} GB/s", file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_seconds)

    line = {
        "metric": METRIC,
        "value": tokens / elapsed,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "lumina_mgpt_768_shape",
            "step": "one whole generation: prefill, 2352 visual steps x 32 layers of "
                    "append/update + grouping at step 299 + decode attention",
            "batch": wl.batch, "layers": wl.layers, "heads": wl.heads,
            "head_dim": wl.head_dim, "prefix_tokens": wl.prefix_len,
            "visual_tokens": wl.num_visual, "rho": args.rho, "period": wl.period,
            "group_threshold": wl.group_threshold, "recent_window": wl.recent_len,
            "kv_storage": "bf16", "accumulate": "fp32 (attention), fp64 (grouping, eviction)",
        },
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": measured_traffic() if args.rho == "1/8" else None,
            "kernel": "k_attn<128, append> (headkv_decode_step)",
            "timed_every_nth_step": args.timing_every,
            "launches": n_launch,
            "avg_launch_us": avg_us,
            "alg_bytes_per_launch": avg_bytes,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
