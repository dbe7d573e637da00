#!/usr/bin/env python3
"""Benchmark of the GSPN 4-direction line scan on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
the forward scan and, for workloads with a backward, the adjoint scan that
produces dx, dw, dlam and du.  Inputs are generated on the device (seeded)
before the timed region; nothing is copied over PCIe inside it.

Prints one JSON line with the throughput in propagated pixel-channel-directions
per second (B*C*H*W*n per step / seconds), the roofline position of the
dominant kernel (algorithmic HBM bytes / its average duration, timed with
events on the stream it runs on) and the float64 CPU oracle timed on a bounded
sample of the same workload.  The timed steps run back to back (warm: inputs
smaller than the 256 MB last-level cache may partly hit in it); "cold" adds
single steps each preceded by a 1 GiB read that evicts that cache.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--algo auto|resident|stream|two_pass]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "propagated pixel-channel-directions/sec and % of HBM roofline, fwd and fwd+bwd"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak
DEFAULT_WORKLOAD = "cls28_bf16_fb"  # the workload whose step covers forward and backward
ALGOS = {"auto": 0, "resident": 1, "stream": 2, "resident_generic": 3, "two_pass": 4}
KERNEL_SRC = os.path.join(ROOT, "paper_2501_12381_amd", "csrc")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in sorted(os.listdir(KERNEL_SRC)):
        if f.endswith((".hip", ".hpp")):
            h.update(f.encode())
            h.update(open(os.path.join(KERNEL_SRC, f), "rb").read())
    return h.hexdigest()[:16]


def alg_bytes(wl, which: str) -> int:
    """Algorithmic HBM bytes of one call: every ABI tensor read once, written once."""
    s = 4 if wl.dtype == "f32" else 2
    npc = wl.B * wl.C * wl.H * wl.W
    n = wl.n_dirs
    if which == "fwd":
        return npc * (4 + 3 * n) * s  # x, lam, u, w in; y out
    return npc * (7 + 6 * n) * s  # dy, x, lam, u, w in; dx, dlam, du, dw out


def traffic_for(workload: str, kernel: str):
    """Counter-measured HBM bytes per launch, if a profile of the current kernels exists."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    k = d.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


def cpu_baseline(wl, target_s: float = 12.0) -> dict:
    """The float64 oracle on a sample of planes of the same workload (host cores)."""
    import oracle as O
    from paper_2501_12381_amd import synth

    import torch

    def run(planes):
        sub = wl.with_shape(B=1, C=planes)
        t = synth.make_inputs(sub, "cpu", with_dy=wl.backward)
        a = {k: v.to(torch.float64).numpy() for k, v in t.items()}
        t0 = time.perf_counter()
        O.scan_fwd(a["x"], a["w"], a["lam"], a["u"], wl.mask)
        if wl.backward:
            O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], wl.mask)
        return time.perf_counter() - t0

    # calibrate on a few planes, then size the sample for about target_s seconds
    # (repeating the whole workload when it is shorter than that)
    probe = min(8, wl.planes)
    dt = run(probe)
    sample_planes = max(1, min(wl.planes, int(probe * target_s / max(dt, 1e-3))))
    dt = run(sample_planes)
    reps, total = 1, dt
    while total < target_s * 0.8 and reps < 30:
        total += run(sample_planes)
        reps += 1
    pcd = sample_planes * wl.H * wl.W * wl.n_dirs * reps
    return {"value": pcd / total, "unit": "PCD/s", "cores": 1, "kind": "oracle",
            "sample": f"{sample_planes} of {wl.planes} planes of {wl.name} "
                      f"({'fwd+bwd' if wl.backward else 'fwd'}) x {reps} run(s), float64 NumPy, "
                      f"single process, {total:.1f} s"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--algo", default="auto", choices=sorted(ALGOS), help="forward kernel family")
    ap.add_argument("--bwd-algo", default="auto", choices=sorted(ALGOS), help="backward kernel family")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cold-reps", type=int, default=5,
                    help="extra single steps, each after a 1 GiB read that evicts the last-level cache "
                         "(reported as 'cold' beside the timed, warm steps; 0 = skip)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="also run the reference copy kernel on this many MiB (for counter runs)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the scan shards over (b, c) planes with no "
              "communication, so a multi-GPU run would add nothing this benchmark measures; "
              "run with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    from paper_2501_12381_amd import ops, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    wl = synth.WORKLOADS[args.workload]
    algo = ALGOS[args.algo]
    bwd_algo = ALGOS[args.bwd_algo]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    inp = synth.make_inputs(wl, dev, with_dy=wl.backward)
    torch.cuda.synchronize()
    x, w, lam, u = inp["x"], inp["w"], inp["lam"], inp["u"]
    y = torch.empty_like(x)

    def fwd_call():
        ops.gspn_scan_fwd(x, w, lam, u, wl.mask, algo=algo, y=y)

    def bwd_call():
        ops.gspn_scan_bwd(inp["dy"], x, w, lam, u, wl.mask, algo=bwd_algo)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        fwd_call()
        if ev is not None:
            ev[1].record()
        if wl.backward:
            bwd_call()
            if ev is not None:
                ev[2].record()

    if args.copy_calibration_mb:
        nb = args.copy_calibration_mb << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev)
        dst = torch.empty(nb, dtype=torch.uint8, device=dev)
        ops.gspn_copy_calibration(src, dst)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: K steps back to back, events only around the whole run
    # (an event recorded between the calls costs the stream a few
    # microseconds, ~10% of a 100 us step)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for _ in range(args.steps):
        step()
    t_end.record()
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps
    # per-call durations for the roofline: the same K steps again, with events
    # around each call on the stream the kernels run on (each call then also
    # carries one event's cost; calls of one kind back to back would instead
    # change what the last-level cache holds when they start)
    if wl.backward:
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        for k in range(args.steps):
            step(evs[k])
        torch.cuda.synchronize()
        fwd_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
        bwd_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    else:
        fwd_ms, bwd_ms = ms_step, 0.0  # one call per step: the timed run itself

    # cold steps: a 1 GiB read between steps (outside the events) evicts the
    # inputs from the 256 MB last-level cache, so each step reads them from HBM.
    # The flush reads (a reduction), so the lines it leaves are clean and the
    # step pays no write-back for them; medians over the repetitions
    cold = None
    if args.cold_reps > 0:
        flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        sink = torch.empty((), dtype=torch.float32, device=dev)
        torch.sum(flush, dim=0, out=sink)
        torch.cuda.synchronize()
        cev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.cold_reps)]
        for k in range(args.cold_reps):
            torch.sum(flush, dim=0, out=sink)
            step(cev[k])
        torch.cuda.synchronize()
        del flush, sink

        def median(v):
            v = sorted(v)
            return v[len(v) // 2] if len(v) % 2 else 0.5 * (v[len(v) // 2 - 1] + v[len(v) // 2])
        c_fwd = median([e[0].elapsed_time(e[1]) for e in cev])
        c_bwd = median([e[1].elapsed_time(e[2]) for e in cev]) if wl.backward else 0.0
        c_dom = c_bwd if wl.backward and bwd_ms > fwd_ms else c_fwd
        d_name = "bwd" if wl.backward and bwd_ms > fwd_ms else "fwd"
        cold = {"reps": args.cold_reps, "flush_bytes": 1 << 30, "fwd_us": c_fwd * 1e3,
                "bwd_us": c_bwd * 1e3 if wl.backward else None, "step_us": (c_fwd + c_bwd) * 1e3,
                "dominant_frac": alg_bytes(wl, d_name) / (c_dom / 1e3) / (HBM_PEAK_GBS * 1e9)}

    pcd = wl.B * wl.C * wl.H * wl.W * wl.n_dirs
    value = pcd / (ms_step / 1e3)
    dom = "bwd" if wl.backward and bwd_ms > fwd_ms else "fwd"
    dom_ms = bwd_ms if dom == "bwd" else fwd_ms
    kname = {"fwd": "gspn_scan_fwd", "bwd": "gspn_scan_bwd"}[dom]
    achieved = alg_bytes(wl, dom) / (dom_ms / 1e3) / 1e9
    traffic = traffic_for(wl.name, kname)
    print(f"[bench] {wl.name} algo={args.algo}: step {ms_step * 1e3:.1f} us, fwd {fwd_ms * 1e3:.1f} us "
          f"({alg_bytes(wl, 'fwd') / (fwd_ms / 1e3) / 1e9:.0f} GB/s alg)"
          + (f", bwd {bwd_ms * 1e3:.1f} us ({alg_bytes(wl, 'bwd') / (bwd_ms / 1e3) / 1e9:.0f} GB/s alg)"
             if wl.backward else "")
          + (f"; cold fwd {cold['fwd_us']:.1f} us" + (f", bwd {cold['bwd_us']:.1f} us" if wl.backward else "")
             if cold else ""), file=sys.stderr, flush=True)

    cpu = None if args.no_cpu_baseline else cpu_baseline(wl)
    step_bytes = alg_bytes(wl, "fwd") + (alg_bytes(wl, "bwd") if wl.backward else 0)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "PCD/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "C": wl.C, "H": wl.H, "W": wl.W,
                   "mask": wl.mask, "directions": wl.n_dirs,
                   "pass": "fwd+bwd" if wl.backward else "fwd", "algo": args.algo,
                   "bwd_algo": args.bwd_algo if wl.backward else None,
                   "step_alg_bytes": step_bytes,
                   "step_roofline_frac": step_bytes / (ms_step / 1e3) / (HBM_PEAK_GBS * 1e9)},
        "roofline": {"bound": "hbm", "kernel": kname, "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "avg_launch_us": dom_ms * 1e3, "alg_bytes_per_launch": alg_bytes(wl, dom)},
        "cpu_baseline": cpu,
        "cold": cold,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
