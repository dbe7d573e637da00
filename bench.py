#!/usr/bin/env python3
"""Benchmark of the GSPN 4-direction line scan on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
the forward scan and, for workloads with a backward, the adjoint scan that
produces dx, dw, dlam and du (as in training, the forward keeps its states in
the workspace for the backward where the kernel family supports it).  Inputs
are generated on the device (seeded) before the timed region; nothing is
copied over PCIe inside it.

The headline line measures the largest single-GPU workload: the 4-direction
bf16 forward on 1 x 320 x 2048 x 2048 planes (an image latent of about 16K
pixels a side).  Beside it, `extra` holds the other measured workloads (the
28 x 28 classification-stage forward+backward, the 128 x 128 diffusion-latent
forward, the 56 x 56 fp32 forward, forward+backward at both latent sizes, and
forward+backward at 28 x 28 and 128 x 128 with the paper's Eq. 6 logits
normalised inside the call), each with its own roofline entries.

Prints one JSON line with the throughput in propagated pixel-channel-directions
per second (B*C*H*W*n per step / seconds), the roofline position of the
dominant call (algorithmic HBM bytes / its average duration, timed with events
on the stream it runs on), the bandwidth of a plain device copy measured in the
same run (the achievable ceiling), and the float64 CPU oracle timed on a
bounded sample of the same workload over the host's cores.  The timed steps
run back to back (warm: inputs smaller than the 256 MB last-level cache may
partly hit in it); "cold" adds single steps each preceded by a 1 GiB read that
evicts that cache.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--algo auto|resident|stream|two_pass]
                    [--no-extras] [--no-cpu-baseline]
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
DEFAULT_WORKLOAD = "lat2048_bf16"  # the largest workload that fits one GPU
EXTRA_WORKLOADS = ("cls28_bf16_fb", "lat128_bf16", "cls56_f32", "lat128_bf16_fb", "lat2048_bf16_fb",
                   "cls28_bf16_lg_fb", "lat128_bf16_lg_fb")
ALGOS = {"auto": 0, "resident": 1, "stream": 2, "resident_generic": 3, "two_pass": 4}
KERNEL_SRC = os.path.join(ROOT, "paper_2501_12381_amd", "csrc")
CPU_WORKERS_MAX = 16  # the host-core share of one GPU on the benchmark machines


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


# ---------------------------------------------------------------------------
# CPU baseline: the float64 oracle over the host's cores
# ---------------------------------------------------------------------------
def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_worker(args):
    """Runs in a forked worker: draw `planes` planes, wait for the others, time the oracle."""
    wl, planes, seed, barrier = args
    import oracle as O
    from paper_2501_12381_amd import synth

    a = synth.numpy_planes(wl, planes, seed)
    barrier.wait()
    t0 = time.perf_counter()
    O.scan_fwd(a["x"], a["w"], a["lam"], a["u"], wl.mask)
    if wl.backward:
        O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], wl.mask)
    return t0, time.perf_counter()


def cpu_baseline(wl, target_s: float = 6.0) -> dict:
    """The float64 oracle on a sample of planes of the same workload, one plane
    set per host core (forked worker processes, started before this process
    touches the GPU)."""
    import multiprocessing as mp

    cores = min(CPU_WORKERS_MAX, len(os.sched_getaffinity(0)))
    ctx = mp.get_context("fork")
    with ctx.Manager() as mgr:
        # one plane on one core calibrates the sample size
        with ctx.Pool(1) as pool:
            t0, t1 = pool.apply(_oracle_worker, ((wl, 1, 0, mgr.Barrier(1)),))
        t_plane = t1 - t0
        per = max(1, min(max(1, wl.planes // cores), int(target_s / max(t_plane, 1e-4))))
        bar = mgr.Barrier(cores)
        with ctx.Pool(cores) as pool:
            res = pool.map(_oracle_worker, [(wl, per, 1 + i, bar) for i in range(cores)])
    wall = max(e for _, e in res) - min(s for s, _ in res)
    pcd = cores * per * wl.H * wl.W * wl.n_dirs
    return {"value": pcd / wall, "unit": "PCD/s", "cores": cores, "kind": "oracle",
            "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "single_core_value": wl.H * wl.W * wl.n_dirs / t_plane,
            "sample": f"{cores} processes x {per} plane(s) of {wl.H}x{wl.W} ({wl.name}, "
                      f"{'fwd+bwd' if wl.backward else 'fwd'}; {cores * per} of {wl.planes} planes), "
                      f"float64 NumPy, {wall:.1f} s wall"}


# ---------------------------------------------------------------------------
# GPU measurement of one workload
# ---------------------------------------------------------------------------
def median(v):
    v = sorted(v)
    return v[len(v) // 2] if len(v) % 2 else 0.5 * (v[len(v) // 2 - 1] + v[len(v) // 2])


def roofline_entry(wl, which: str, ms: float) -> dict:
    kname = {"fwd": "gspn_scan_fwd", "bwd": "gspn_scan_bwd"}[which]
    achieved = alg_bytes(wl, which) / (ms / 1e3) / 1e9
    return {"bound": "hbm", "kernel": kname, "achieved": achieved, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic_for(wl.name, kname), "avg_launch_us": ms * 1e3,
            "alg_bytes_per_launch": alg_bytes(wl, which)}


def measure(wl, algo: int, bwd_algo: int, steps: int, warmup: int, cold_reps: int, dev) -> dict:
    import torch

    from paper_2501_12381_amd import ops, synth

    inp = synth.make_inputs(wl, dev, with_dy=wl.backward)
    torch.cuda.synchronize()
    x, w, lam, u = inp["x"], inp["w"], inp["lam"], inp["u"]
    y = torch.empty_like(x)
    # a training step keeps the forward's states for the backward (the kernel
    # families that keep a plane on chip ignore the option); one workspace
    # serves both calls
    save = wl.backward and algo == bwd_algo
    ws = ops.scan_workspace(x, wl.mask, algo=algo, save_state=True, logits=wl.logits) if save else None
    kept = None
    if save:
        from paper_2501_12381_amd import lib as L
        sizes = [L.gspn_scan_fwd_workspace_bytes(wl.B, wl.C, wl.H, wl.W, wl.mask, ops._dtype_code(x),
                                                 flags=f | (L.GSPN_FLAG_W_LOGITS if wl.logits else 0), algo=algo)
                 for f in (0, L.GSPN_FLAG_SAVE_STATE)]
        kept = "kept for the backward" if sizes[1] > sizes[0] else "recomputed by the backward (on chip)"

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        ops.gspn_scan_fwd(x, w, lam, u, wl.mask, algo=algo, y=y, logits=wl.logits, workspace=ws, save_state=save)
        if ev is not None:
            ev[1].record()
        if wl.backward:
            ops.gspn_scan_bwd(inp["dy"], x, w, lam, u, wl.mask, algo=bwd_algo, logits=wl.logits, workspace=ws,
                              save_state=save)
            if ev is not None:
                ev[2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: K steps back to back, events only around the whole run
    # (an event recorded between the calls costs the stream a few microseconds)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record()
    for _ in range(steps):
        step()
    t_end.record()
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / steps
    # per-call durations: the same K steps again with events around each call
    # on the launch stream (calls of one kind back to back would change what
    # the last-level cache holds when they start)
    if wl.backward:
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        for k in range(steps):
            step(evs[k])
        torch.cuda.synchronize()
        fwd_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / steps
        bwd_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / steps
    else:
        fwd_ms, bwd_ms = ms_step, 0.0  # one call per step: the timed run itself

    # cold steps: a 1 GiB read between steps (outside the events) evicts the
    # inputs from the last-level cache; the flush reads, so it leaves no dirty
    # lines whose write-back the step would pay for
    cold = None
    if cold_reps > 0:
        flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        sink = torch.empty((), dtype=torch.float32, device=dev)
        torch.sum(flush, dim=0, out=sink)
        torch.cuda.synchronize()
        cev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(cold_reps)]
        for k in range(cold_reps):
            torch.sum(flush, dim=0, out=sink)
            step(cev[k])
        torch.cuda.synchronize()
        del flush, sink
        c_fwd = median([e[0].elapsed_time(e[1]) for e in cev])
        c_bwd = median([e[1].elapsed_time(e[2]) for e in cev]) if wl.backward else 0.0
        cold = {"reps": cold_reps, "flush_bytes": 1 << 30, "fwd_us": c_fwd * 1e3,
                "fwd_frac": alg_bytes(wl, "fwd") / (c_fwd / 1e3) / (HBM_PEAK_GBS * 1e9),
                "bwd_us": c_bwd * 1e3 if wl.backward else None,
                "bwd_frac": alg_bytes(wl, "bwd") / (c_bwd / 1e3) / (HBM_PEAK_GBS * 1e9)
                if wl.backward else None,
                "step_us": (c_fwd + c_bwd) * 1e3}
    del inp, x, w, lam, u, y, ws
    torch.cuda.empty_cache()

    dom = "bwd" if wl.backward and bwd_ms > fwd_ms else "fwd"
    step_bytes = alg_bytes(wl, "fwd") + (alg_bytes(wl, "bwd") if wl.backward else 0)
    r = {"workload": wl.name, "B": wl.B, "C": wl.C, "H": wl.H, "W": wl.W, "mask": wl.mask,
         "directions": wl.n_dirs, "dtype": wl.dtype, "pass": "fwd+bwd" if wl.backward else "fwd",
         "weights": "eq6_logits" if wl.logits else "normalised",
         "forward_state": kept,
         "ms_per_step": ms_step, "value": wl.B * wl.C * wl.H * wl.W * wl.n_dirs / (ms_step / 1e3),
         "step_alg_bytes": step_bytes,
         "step_roofline_frac": step_bytes / (ms_step / 1e3) / (HBM_PEAK_GBS * 1e9),
         "fwd_us": fwd_ms * 1e3, "bwd_us": bwd_ms * 1e3 if wl.backward else None,
         "dominant": dom, "roofline": roofline_entry(wl, dom, bwd_ms if dom == "bwd" else fwd_ms),
         "cold": cold}
    if wl.backward:
        r["roofline_fwd"] = roofline_entry(wl, "fwd", fwd_ms)
        r["roofline_bwd"] = roofline_entry(wl, "bwd", bwd_ms)
    print(f"[bench] {wl.name}: step {ms_step * 1e3:.1f} us, fwd {fwd_ms * 1e3:.1f} us "
          f"({alg_bytes(wl, 'fwd') / (fwd_ms / 1e3) / 1e9:.0f} GB/s alg)"
          + (f", bwd {bwd_ms * 1e3:.1f} us ({alg_bytes(wl, 'bwd') / (bwd_ms / 1e3) / 1e9:.0f} GB/s alg)"
             if wl.backward else "")
          + (f"; cold fwd {cold['fwd_us']:.1f} us" + (f", bwd {cold['bwd_us']:.1f} us" if wl.backward else "")
             if cold else ""), file=sys.stderr, flush=True)
    return r


def copy_ceiling(dev, nbytes: int = 2 << 30, reps: int = 10) -> dict:
    """Bandwidth of the library's plain copy kernel (bytes read + written per second)."""
    import torch

    from paper_2501_12381_amd import ops

    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    src.fill_(1)
    ops.gspn_copy_calibration(src, dst)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        ops.gspn_copy_calibration(src, dst)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    torch.cuda.empty_cache()
    gbs = 2 * nbytes / (ms / 1e3) / 1e9
    return {"bytes_each_way": nbytes, "us": ms * 1e3, "GB_s": gbs, "frac_of_peak": gbs / HBM_PEAK_GBS}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--algo", default="auto", choices=sorted(ALGOS), help="forward kernel family")
    ap.add_argument("--bwd-algo", default="auto", choices=sorted(ALGOS), help="backward kernel family")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="measure the selected workload only")
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

    from paper_2501_12381_amd import synth

    wl = synth.WORKLOADS[args.workload]
    # the CPU leg forks its workers before this process touches the GPU
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl)
        print(f"[bench] cpu oracle: {cpu['value']:.3e} PCD/s on {cpu['cores']} cores ({cpu['sample']})",
              file=sys.stderr, flush=True)

    import torch

    from paper_2501_12381_amd import ops

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    algo, bwd_algo = ALGOS[args.algo], ALGOS[args.bwd_algo]

    if args.copy_calibration_mb:
        nb = args.copy_calibration_mb << 20
        src = torch.empty(nb, dtype=torch.uint8, device=dev)
        dst = torch.empty(nb, dtype=torch.uint8, device=dev)
        ops.gspn_copy_calibration(src, dst)
        torch.cuda.synchronize()
        del src, dst

    head = measure(wl, algo, bwd_algo, args.steps, args.warmup, args.cold_reps, dev)
    extra = {}
    if not args.no_extras:
        for name in EXTRA_WORKLOADS:
            if name != wl.name:
                extra[name] = measure(synth.WORKLOADS[name], 0, 0, args.steps, args.warmup,
                                      args.cold_reps, dev)
    ceiling = None if args.no_extras else copy_ceiling(dev)

    rl = dict(head["roofline"])
    if ceiling:
        rl["copy_ceiling_GB_s"] = ceiling["GB_s"]
        rl["frac_of_copy_ceiling"] = rl["achieved"] / ceiling["GB_s"]
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "PCD/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "C": wl.C, "H": wl.H, "W": wl.W,
                   "mask": wl.mask, "directions": wl.n_dirs, "pass": head["pass"],
                   "algo": args.algo, "bwd_algo": args.bwd_algo if wl.backward else None,
                   "step_alg_bytes": head["step_alg_bytes"],
                   "step_roofline_frac": head["step_roofline_frac"],
                   "fwd_us": head["fwd_us"], "bwd_us": head["bwd_us"]},
        "roofline": rl,
        "cpu_baseline": cpu,
        "cold": head["cold"],
        "copy_ceiling": ceiling,
        "extra": extra,
    }
    if wl.backward:
        out["roofline_fwd"], out["roofline_bwd"] = head["roofline_fwd"], head["roofline_bwd"]
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
