#!/usr/bin/env python3
"""Benchmark of the active-set batched Sinkhorn hot path on one MI355X.

One step = one complete solve of the mixture workload window (W=64 lanes,
n=m=1024 points in d=8, Dirichlet(1) marginals, eps=0.05, two-sided L1
tolerance 1e-3, audit after every cycle, active mode): ingest, packed f/g
half-steps, fused row screen, two-sided check, retirement, physical compaction
and output emission -- with the inputs already resident in HBM.

Prints one JSON line:
  value       candidate-update slots per second (sum_t l_t per solve / solve time)
  ms_per_step end-to-end batch time of one solve
  roofline    the update kernel (the dominant kernel): algorithmic x.y flops
              (2 d per valid (i, j) term) / summed HIP-event duration of its
              launches inside the timed region, against the fp32 matrix peak
  cpu_baseline the float64 oracle on a bounded sample, on this host's cores
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_FP32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0


def _cores():
    try:
        return len(os.sched_getaffinity(0))
    except Exception:
        return os.cpu_count() or 1


def measured_traffic():
    """HBM bytes per update launch from the committed FETCH_SIZE / WRITE_SIZE
    summary, or None once the kernel source has changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "k_update_mfma_c2_traffic.md")
    src = os.path.join(ROOT, "paper_2607_24741_amd", "csrc", "ds_kernels.hip")
    try:
        fields = dict(line.split(": ", 1) for line in open(path).read().splitlines()
                      if line.startswith(("kernel_source_sha256: ", "traffic_bytes_per_launch: ")))
        cur = hashlib.sha256(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    if fields.get("kernel_source_sha256") != cur:
        return None
    return float(fields["traffic_bytes_per_launch"])


def cpu_baseline(w, tol, cycles=600, lanes=None):
    """Oracle as it stands (test infrastructure, float64, not tuned) on a
    bounded sample: the first `lanes` lanes of the window, each run for a fixed
    `cycles` cycles with the two-sided audit after every cycle (the same work
    per slot as the solver), one process per core."""
    import numpy as np
    import oracle
    n_proc = min(16, _cores())
    lanes = n_proc if lanes is None else lanes
    sel = list(range(min(lanes, w.W)))
    t0 = time.perf_counter()
    oracle.solve(w.X, w.Y, w.a, w.b, w.eps, 1e-30, n=w.n, m=w.m, max_iter=cycles, lanes=sel,
                 processes=n_proc)
    dt = time.perf_counter() - t0
    slots = cycles * len(sel)
    return {"value": slots / dt, "unit": "slots/s", "cores": n_proc, "kind": "oracle",
            "sample": f"{len(sel)} lanes of the same window, {cycles} cycles each with a two-sided "
                      f"audit after every cycle (float64 numpy, {n_proc} worker processes, "
                      f"{dt:.1f} s wall)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--tol", type=float, default=1e-3)
    ap.add_argument("--mode", default="active", choices=["active", "static", "logical"])
    ap.add_argument("--config", default="c2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: lanes are independent problems and the "
              "path has no cross-GPU step; run one process per GPU instead "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2607_24741_amd as ds
    from paper_2607_24741_amd import workloads as wl

    dev = torch.device("cuda:0")
    w = wl.make(args.config)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    X, Y, a, b, eps, n, m = (t(w.X), t(w.Y), t(w.a), t(w.b), t(w.eps), t(w.n), t(w.m))
    need = ds.workspace_bytes(w.W, w.X.shape[1], w.Y.shape[1], w.d, tol=args.tol,
                              max_iter=w.max_iter, mode=args.mode)
    ws = torch.empty(need + 256, dtype=torch.uint8, device=dev)

    def step(flags):
        r = ds.solve(X, Y, a, b, eps, args.tol, n=n, m=m, max_iter=w.max_iter, mode=args.mode,
                     flags=flags, return_stats=True, workspace=ws)
        return r

    for _ in range(args.warmup):
        step(0)
    torch.cuda.synchronize()
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        last = step(ds.F_TIMING)
        stats.append(last[-1])
    torch.cuda.synchronize()
    T = time.perf_counter() - t0
    status = last[4].cpu().numpy()
    slots = sum(s.slots_update for s in stats)
    pairs = sum(s.pair_evals + s.check_pair_evals for s in stats)
    # roofline: the timed (sampled) launches of the update kernel -- both
    # launches of every 32nd cycle, bracketed by HIP events on the solve's stream
    tpairs = sum(s.timed_pair_evals for s in stats)
    ms_upd = sum(s.ms_update for s in stats)
    launches = sum(s.update_launches for s in stats)
    achieved = 2.0 * w.d * tpairs / (ms_upd * 1e-3) / 1e12
    rec = {
        "metric": "candidate-update slots/sec (end-to-end batch solve at tol 1e-3)",
        "value": slots / T,
        "unit": "slots/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * T / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded generator shaped like the paper's Packer19 window; no dataset)",
        "config": {"workload": wl.DESCRIPTIONS[args.config], "name": args.config, "W": w.W,
                   "n": int(w.X.shape[1]), "m": int(w.Y.shape[1]), "d": w.d, "tol": args.tol,
                   "audit_every": 1, "mode": args.mode, "max_iter": w.max_iter},
        "slots_per_step": slots // args.steps,
        "pair_evals_per_step": pairs // args.steps,
        "l_max": stats[-1].l_max,
        "lanes_converged": int((status == 0).sum()),
        "lanes_max_iter": int((status == 1).sum()),
        "compactions": stats[-1].compactions,
        "timed_update_launches_per_step": launches // args.steps,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": MFMA_FP32_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / MFMA_FP32_PEAK_TFLOPS,
                     "traffic": measured_traffic(),
                     "kernel": "k_update_mfma (f- and g-half-steps)",
                     "avg_launch_us": 1e3 * ms_upd / max(1, launches),
                     "algorithmic": "2*d flops per valid (i,j) term evaluated by the timed launches",
                     "timed_pair_evals": tpairs, "timed_ms": ms_upd},
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, args.tol)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
