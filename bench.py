#!/usr/bin/env python3
"""Benchmark of the active-set batched Sinkhorn hot path on one MI355X.

One step = one complete solve of the largest workload window, the
LiDAR-shaped heterogeneous batch (W=1024 lanes, n_t, m_t ~ U{256..8192} padded
to 8192, d=3, Dirichlet(0.5) marginals, eps_t ~ logU(0.005, 0.1), two-sided L1
tolerance 1e-3, audit after every cycle, active mode, default float64 state):
ingest, packed f/g half-steps, fused row screen, two-sided check, retirement,
physical compaction and output emission -- with the inputs already resident in
HBM. The headline runs as one sub-batch (one stream), so that every update
launch has the chip to itself and its duration is the kernel's own. Other
windows (`--config c1..c5`), `--fast32`, `--materialize` and `--streams` are
available for study.

Prints one JSON line:
  value        candidate-update slots per second (sum_t l_t per solve / solve time)
  ms_per_step  end-to-end batch time of one solve
  roofline     the update kernel (the dominant kernel): algorithmic work of the
               timed launches (every 32nd cycle's two launches and the final
               audit, timed by events attached to the kernel dispatches) over
               their summed duration. Matrix-free small d: the vector-unit
               model t_pe = max((d + 4) / R_v, 1 / R_e) per (i, j) term, with
               R_v = 3.93e13 lane operations/s (256 CUs x 4 SIMDs x 16 lanes x
               2.4 GHz: the float64 and non-packed float32 issue rate) and
               R_e = 1.97e13 exponentials/s (8 lanes/clk per SIMD); `achieved`
               counts each lane operation as one multiply-add (2 flops) against
               the float64 vector peak 78.6 TFLOP/s, so `frac` is the model's
               fraction. Materialised cost: HBM, 4 bytes per term.
  mixture_modes      the mixture window's static and logical modes over its active
               mode, all three at one sub-batch
  mixture_tol_sweep  the mixture window's end-to-end batch time at each swept tol
  cpu_baseline the float64 oracle on a bounded sample, on this host's cores

`--study` instead measures the execution surface of eq:time-accounting on the
window's lanes (one JSON line): the width-cost curve c(A) of a fixed-work cycle,
the static/active ratio per physical width W (windows cut from the same lanes,
the width sweep of tab:width-regime) and the grouping intervention of
tab:m3-grouping (one fixed lane multiset grouped by depth, against depth,
and at random).
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# float64 vector peak (and non-packed float32: this build generates no packed
# float32 instructions): 256 CUs x 4 SIMDs x 16 lanes x 2 flops (FMA) x 2.4 GHz
VALU_PEAK_TFLOPS = 78.6
# The vector-unit model of a small-d matrix-free half-step, t_pe = max((d + 4)
# / R_v, 1 / R_e) per (i, j) term: d multiply-adds of the dot product plus the
# scale, maximum, shift and add, at R_v = 3.93e13 lane operations/s, and one
# exponential at 256 CUs x 4 SIMDs x 8 lanes/clk x 2.4 GHz of transcendental
# issue (the published quarter rate, 9.8e12/s, is below what gfx950 was
# measured to sustain, 1.83e13/s, so it would inflate the fraction).
VECTOR_LANE_OPS_PEAK = VALU_PEAK_TFLOPS * 1e12 / 2.0
MAT_MAX_POINTS = 16384   # points per side the materialised-cost kernels stage
EXP_PEAK = 256 * 4 * 8 * 2.4e9


def _cores():
    try:
        return len(os.sched_getaffinity(0))
    except Exception:
        return os.cpu_count() or 1


LIBRARY_SOURCES = ("ds_kernels.hip", "ds_host.cpp", "ds_internal.h")


def source_code_hash(texts):
    """sha256 of the library's code with comments and blank lines taken out
    (each line cut at `//`, stripped, empty lines dropped; the sources hold no
    `//` inside string literals), so that a comment edit keeps a profile valid
    and any code edit does not."""
    import hashlib
    h = hashlib.sha256()
    for text in texts:
        for line in text.splitlines():
            code = line.split("//", 1)[0].strip()
            if code:
                h.update(code.encode() + b"\n")
        h.update(b"\0")
    return h.hexdigest()


def measured_traffic(name):
    """HBM bytes per update launch from the committed FETCH_SIZE / WRITE_SIZE
    summary `profiles/<name>`, or None once the library's code (kernels and the
    host runtime that picks their layouts and sub-batches) has changed since it
    was taken."""
    path = os.path.join(ROOT, "profiles", name)
    csrc = os.path.join(ROOT, "paper_2607_24741_amd", "csrc")
    try:
        fields = dict(line.split(": ", 1) for line in open(path).read().splitlines()
                      if line.startswith(("kernel_code_sha256: ", "traffic_bytes_per_launch: ")))
        cur = source_code_hash(open(os.path.join(csrc, n)).read() for n in LIBRARY_SOURCES)
    except OSError:
        return None
    if fields.get("kernel_code_sha256") != cur:
        return None
    return float(fields["traffic_bytes_per_launch"])


def study(args):
    """Width-cost curve, width sweep and grouping intervention (see the module
    docstring). One sub-batch throughout, so that width effects are not mixed
    with concurrency; every time is a synchronised wall time of one solve."""
    import numpy as np
    import torch
    import paper_2607_24741_amd as ds
    from paper_2607_24741_amd import workloads as wl

    dev = torch.device("cuda:0")
    w = wl.make(args.config)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    D = dict(X=t(w.X), Y=t(w.Y), a=t(w.a), b=t(w.b), eps=t(w.eps), n=t(w.n), m=t(w.m))

    def run(idx, mode, tol, max_iter):
        ix = torch.tensor(idx, device=dev, dtype=torch.long)
        sel = {k: v.index_select(0, ix).contiguous() for k, v in D.items()}
        def once():
            return ds.solve(sel["X"], sel["Y"], sel["a"], sel["b"], sel["eps"], tol, n=sel["n"],
                            m=sel["m"], max_iter=max_iter, mode=mode, streams=1)
        once()   # warm (workspace allocation, first-touch)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r = once()
        torch.cuda.synchronize()
        return 1e3 * (time.perf_counter() - t0), r[2].cpu().numpy()

    W = w.W
    widths = [k for k in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024) if k <= W]
    # (a) width-cost curve: K fixed cycles (unreachable tolerance) at width A
    K = 64
    curve = []
    for A in widths:
        ms, _ = run(list(range(A)), "static", 1e-30, K)
        curve.append({"A": A, "ms_per_cycle": ms / K, "us_per_lane_cycle": 1e3 * ms / K / A})
        print(f"[study] {args.config} width-cost A={A}: {ms / K:.3f} ms per cycle", file=sys.stderr,
              flush=True)
    # (b) width sweep: windows of W lanes cut from the window (at most 8 per
    # width, evenly spaced), static time over active time
    sweep = []
    for Wd in widths:
        starts = list(range(0, W - Wd + 1, Wd))
        if len(starts) > 8:
            starts = [starts[int(q)] for q in np.linspace(0, len(starts) - 1, 8).round()]
        ratios = []
        for s0 in starts:
            idx = list(range(s0, s0 + Wd))
            ta, _ = run(idx, "active", args.tol, w.max_iter)
            ts, _ = run(idx, "static", args.tol, w.max_iter)
            ratios.append(ts / ta)
        r = np.array(ratios)
        print(f"[study] {args.config} width {Wd}: static/active median {np.median(r):.3f} over "
              f"{len(r)} windows", file=sys.stderr, flush=True)
        sweep.append({"W": Wd, "windows": len(r), "static_over_active_median": float(np.median(r)),
                      "min": float(r.min()), "max": float(r.max()), "wins": int((r > 1).sum())})
    # eq:active-gate: the smallest width from which active execution wins --
    # static over active above 1.02 (the spread of repeated equal-work solves
    # at W = 1) in the median over the windows -- at every larger width measured
    above = [q["W"] for q in sweep if q["static_over_active_median"] > 1.02]
    gate = None
    for q in reversed(sweep):
        if q["static_over_active_median"] > 1.02:
            gate = q["W"]
        else:
            break
    # (c) grouping intervention: one lane multiset (the first 128 lanes at
    # most) in windows of G lanes
    G = min(16, W)
    Wg = min(W, 128)
    _, depth = run(list(range(Wg)), "active", args.tol, w.max_iter)
    order = np.argsort(depth, kind="stable")
    nwin = Wg // G
    groupings = {"homogeneous": [order[q * G:(q + 1) * G] for q in range(nwin)],
                 "heterogeneous": [order[q::nwin][:G] for q in range(nwin)]}
    for rs in (1, 2, 3):
        perm = np.random.default_rng(rs).permutation(Wg)
        groupings[f"random {rs}"] = [perm[q * G:(q + 1) * G] for q in range(nwin)]
    grouping = []
    for name, wins in groupings.items():
        hd, pad, act, stat, ta_sum, ts_sum = [], [], 0, 0, 0.0, 0.0
        for idx in wins:
            dd = depth[idx].astype(np.float64)
            hd.append(dd.std() / dd.mean())
            pad.append(len(dd) * dd.max() / dd.sum() - 1.0)
            act += dd.sum()
            stat += len(dd) * dd.max()
            ta, _ = run([int(i) for i in idx], "active", args.tol, w.max_iter)
            ts, _ = run([int(i) for i in idx], "static", args.tol, w.max_iter)
            ta_sum += ta
            ts_sum += ts
        print(f"[study] {args.config} grouping {name}: static/active {ts_sum / ta_sum:.3f}",
              file=sys.stderr, flush=True)
        grouping.append({"grouping": name, "H_D": float(np.mean(hd)), "padding": float(np.mean(pad)),
                         "active_slots": float(act / stat), "static_over_active": ts_sum / ta_sum})
    rec = {"study": "execution surface", "config": {"workload": wl.DESCRIPTIONS[args.config],
                                                    "name": args.config, "tol": args.tol,
                                                    "sub_batches": 1, "window_for_grouping": G},
           "width_cost_curve": {"fixed_cycles": K, "points": curve},
           "width_sweep": sweep, "active_wins_from_W": gate, "widths_active_wins": above,
           "grouping_lanes": Wg, "grouping": grouping}
    print(json.dumps(rec), flush=True)


def cpu_baseline(w, tol):
    """Oracle as it stands (test infrastructure, float64, not tuned) on a
    bounded sample of the window, each lane run for a fixed number of cycles
    with the two-sided audit after every cycle (the same work per slot as the
    solver), one process per core (at most 16). Mixed-size windows take 16
    lanes at evenly spaced ranks of n_t m_t for 12 cycles; uniform ones their
    first 16 lanes for 600 cycles."""
    import numpy as np
    import oracle
    host = _cores()
    n_proc = min(16, host)
    area = w.n.astype(np.int64) * w.m
    if len(set(area.tolist())) > 1:
        order = np.argsort(area, kind="stable")
        sel = [int(t) for t in order[np.linspace(0, w.W - 1, min(16, w.W)).round().astype(int)]]
        cycles, what = 12, "lanes at evenly spaced ranks of n_t m_t"
    else:
        sel, cycles, what = list(range(min(16, w.W))), 600, "first lanes"
    t0 = time.perf_counter()
    oracle.solve(w.X, w.Y, w.a, w.b, w.eps, 1e-30, n=w.n, m=w.m, max_iter=cycles, lanes=sel,
                 processes=n_proc)
    dt = time.perf_counter() - t0
    slots = cycles * len(sel)
    pairs = 2.0 * cycles * float(area[sel].sum())
    return {"value": slots / dt, "unit": "slots/s", "cores": n_proc, "host_cores": host,
            "kind": "oracle", "pair_evals_per_s": pairs / dt,
            "sample": f"{len(sel)} {what} of the same window, {cycles} cycles each with a "
                      f"two-sided audit after every cycle (float64 numpy, {n_proc} worker "
                      f"processes on a host with {host} cores, {dt:.1f} s wall)"}


def roofline(w, args, stats, T, traffic_summary):
    """The dominant kernel's roofline record (see the module docstring)."""
    tpairs = sum(s.timed_pair_evals for s in stats)
    ms_upd = sum(s.ms_update for s in stats)
    launches = sum(s.update_launches for s in stats)
    kept_pairs = sum(s.pair_evals for s in stats)
    # d > 32: the library materialises the cost unless asked not to or a side
    # has more points than its materialised kernels stage (16384)
    mfree = w.d > 32 and not args.materialize and (
        args.matrix_free or max(int(w.X.shape[1]), int(w.Y.shape[1])) > MAT_MAX_POINTS)
    mat = args.materialize or (w.d > 32 and not mfree)
    rec = {}
    if mfree:
        # the contraction on the matrix cores: 2 d flops per term, fp32 peak
        per_pair, unit, peak, bound = 2.0 * w.d, "TFLOP/s", 157.3, "mfma"
        algo = "2 d flops of the x~.y~ contraction per valid (i,j) term"
        kname = "k_update_mfma_k (f- and g-half-steps)"
        scale = 1e12
    elif mat:
        per_pair, unit, peak, bound = 4.0, "GB/s", HBM_PEAK_GBS, "hbm"
        algo = "4 bytes of materialised cost per valid (i,j) term"
        kname = "k_mat_rows (f-half over Q, g-half over its transpose)"
        scale = 1e9
    else:
        # FMA-equivalent flops of the vector-unit model: 2 (d + 4) per term
        per_pair, unit, peak, bound = 2.0 * (w.d + 4), "TFLOP/s", VALU_PEAK_TFLOPS, "alu"
        algo = ("(d + 4) lane operations per valid (i,j) term (the vector-unit model), "
                "counted as multiply-adds (2 flops each)")
        f64 = not (args.fast32 or args.force_valu) and w.d <= 16
        kname = ("k_update_f64 (float64 state)" if f64 else
                 "k_update_valu (float32 state)" if args.force_valu else
                 "k_update_mfma (float32 state)") + " (f- and g-half-steps)"
        scale = 1e12
        rec["exp_bound_frac"] = (1.0 / EXP_PEAK) / ((w.d + 4) / VECTOR_LANE_OPS_PEAK)
    achieved = per_pair * tpairs / (ms_upd * 1e-3) / scale
    out = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
           "frac": achieved / peak, "traffic": measured_traffic(traffic_summary),
           "kernel": kname, "avg_launch_us": 1e3 * ms_upd / max(1, launches),
           "algorithmic": algo + ", lanes running at each launch's cycle",
           "timed_pair_evals": tpairs, "timed_ms": ms_upd, "timed_launches": launches,
           "device_frac_lb": per_pair * kept_pairs / T / scale / peak}
    out.update(rec)
    return out


def algorithmic_bytes(w, last, f64, st):
    """HBM bytes an update launch must move, on average over the step's
    launches (float64 state only): a lane's half-step with r rows and c columns
    reads the rows' records, lse and log masses and the columns' records and
    potentials, and writes the rows' new lse and potentials --
    r (8 dp + 32) + c (8 dp + 8) bytes, dp = d rounded up to even -- so a cycle
    moves (n + m)(16 dp + 40) bytes per running lane."""
    import numpy as np
    if not f64:
        return {}
    depth = last[2].cpu().numpy().astype(np.int64)
    dp = w.d + (w.d & 1)
    per_cycle = (w.n.astype(np.int64) + w.m) * (16 * dp + 40)
    launches = 2 * st.l_max
    return {"hbm_bytes_per_launch_algorithmic": float((depth * per_cycle).sum()) / max(1, launches)}


def h_terms(w, stats, last, T, steps):
    """Where the step's time goes besides the kept half-steps (eq:time-accounting):
    the verifier's (i, j) work (the column check of screen-positive lanes runs in
    the g-half launches; the final audit's passes), the fused screen's overhead
    (a retired lane's discarded f-half and the g-half that shared its check's
    launch), both as shares of the arithmetic work, and the compaction launches
    (scan + gather, timed with events) as a share of the wall time. The rest of
    the wall time beyond the kernels -- launch gaps and host control -- is read
    from the kernel-trace profile (summed kernel time against the solve time)."""
    import numpy as np
    depth = last[2].cpu().numpy().astype(np.int64)
    status = last[4].cpu().numpy()
    area = w.n.astype(np.int64) * w.m
    st = stats[-1]
    kept = st.pair_evals
    check = st.check_pair_evals
    retired = (status == 0) & (depth < w.max_iter)
    extra = int(2 * area[retired].sum())     # the two extra half-steps of each retired lane
    total = kept + check + extra
    ms_compact = sum(s.ms_compact for s in stats) / steps
    return {"kept_update_pairs": kept, "check_pairs": check, "screen_extra_pairs": extra,
            "check_work_share": check / total, "screen_work_share": extra / total,
            "extra_halfsteps": st.halfsteps_executed - 2 * st.slots_update,
            "compaction_ms": ms_compact, "compaction_share": ms_compact / (1e3 * T / steps),
            "compactions": st.compactions}


def mixture_extras(args, flags):
    """The mixture window (W=64, n=m=1024, d=8): its execution modes at one
    sub-batch each (static packing runs every lane to the common boundary,
    logical masking keeps the full width) and its end-to-end batch time at
    each tolerance of the sweep (automatic sub-batches)."""
    import numpy as np
    import torch
    import paper_2607_24741_amd as ds
    from paper_2607_24741_amd import workloads as wl
    dev = torch.device("cuda:0")
    w = wl.make("c2")
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    X, Y, a, b, eps, n, m = (t(w.X), t(w.Y), t(w.a), t(w.b), t(w.eps), t(w.n), t(w.m))

    def once(mode, tol, streams):
        kw = dict(n=n, m=m, max_iter=w.max_iter, mode=mode, flags=flags, streams=streams,
                  return_stats=True)
        ds.solve(X, Y, a, b, eps, tol, **kw)   # warm
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        r = ds.solve(X, Y, a, b, eps, tol, **kw)
        torch.cuda.synchronize()
        return time.perf_counter() - t1, r

    modes = {}
    ta, _ = once("active", 1e-3, 1)
    modes["active_ms"] = 1e3 * ta
    for mname in ("static", "logical"):
        dt, _ = once(mname, 1e-3, 1)
        modes[mname + "_ms"] = 1e3 * dt
        modes[mname + "_over_active"] = dt / ta
    modes["sub_batches"] = 1
    sweep = []
    for tol in wl.TOL_SWEEP:
        dt, r = once("active", tol, 0)
        st = r[-1]
        sweep.append({"tol": tol, "ms": 1e3 * dt, "slots_per_s": st.slots_update / dt,
                      "slots": st.slots_update, "l_max": st.l_max, "sub_batches": st.sub_batches,
                      "lanes_max_iter": int((r[4].cpu().numpy() == 1).sum())})
    return modes, sweep


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--tol", type=float, default=1e-3)
    ap.add_argument("--mode", default="active", choices=["active", "static", "logical"])
    ap.add_argument("--config", default="c5")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--study", action="store_true",
                    help="measure the width-cost curve, width sweep and grouping instead")
    ap.add_argument("--streams", type=int, default=1,
                    help="concurrent sub-batches (0: the library's automatic choice)")
    ap.add_argument("--fast32", action="store_true", help="float32 state (DS_F_FAST32)")
    ap.add_argument("--force-valu", action="store_true",
                    help="float32 state on the vector-ALU kernels (DS_F_FORCE_VALU)")
    ap.add_argument("--materialize", action="store_true", help="materialised cost (DS_F_MATERIALIZE)")
    ap.add_argument("--matrix-free", action="store_true",
                    help="d > 32: K-looped matrix-core half-step (DS_F_MATRIX_FREE)")
    ap.add_argument("--guard", action="store_true", help="guarded release (DS_F_GUARD)")
    ap.add_argument("--points", type=int, default=None,
                    help="override the window's points per side (n = m); the same recipe")
    ap.add_argument("--no-tol-sweep", action="store_true",
                    help="skip the mixture window's modes and tolerance sweep")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: lanes are independent problems and the "
              "path has no cross-GPU step; run one process per GPU instead "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    if args.study:
        study(args)
        return

    import numpy as np
    import torch
    import paper_2607_24741_amd as ds
    from paper_2607_24741_amd import workloads as wl

    dev = torch.device("cuda:0")
    w = wl.make(args.config) if args.points is None else wl.make(args.config, n=args.points,
                                                                  m=args.points)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    X, Y, a, b, eps, n, m = (t(w.X), t(w.Y), t(w.a), t(w.b), t(w.eps), t(w.n), t(w.m))
    base_flags = ((ds.F_FAST32 if args.fast32 else 0) | (ds.F_FORCE_VALU if args.force_valu else 0)
                  | (ds.F_MATERIALIZE if args.materialize else 0) | (ds.F_GUARD if args.guard else 0)
                  | (ds.F_MATRIX_FREE if args.matrix_free else 0))
    need = ds.workspace_bytes(w.W, w.X.shape[1], w.Y.shape[1], w.d, tol=args.tol,
                              max_iter=w.max_iter, mode=args.mode, flags=base_flags,
                              streams=args.streams)
    ws = torch.empty(need + 256, dtype=torch.uint8, device=dev)

    def step(flags):
        return ds.solve(X, Y, a, b, eps, args.tol, n=n, m=m, max_iter=w.max_iter, mode=args.mode,
                        flags=flags | base_flags, streams=args.streams, return_stats=True,
                        workspace=ws)

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
    f64 = not (args.fast32 or args.force_valu or args.materialize) and w.d <= 16
    traffic_summary = f"k_update_{'f64' if f64 else 'mfma'}_{args.config}_traffic.md"
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
        "dtype": "f64" if f64 else "f32",
        "guarded_release": bool(args.guard),
        "data": "synthetic (seeded generator shaped like the paper's workload; no dataset)",
        "config": {"workload": wl.DESCRIPTIONS[args.config], "name": args.config, "W": w.W,
                   "n": int(w.X.shape[1]), "m": int(w.Y.shape[1]), "d": w.d, "tol": args.tol,
                   "audit_every": 1, "mode": args.mode, "max_iter": w.max_iter,
                   "sub_batches": stats[-1].sub_batches,
                   "points_override": args.points},
        "slots_per_step": slots // args.steps,
        "pair_evals_per_step": pairs // args.steps,
        "l_max": stats[-1].l_max,
        "lanes_converged": int((status == 0).sum()),
        "lanes_max_iter": int((status == 1).sum()),
        "compactions": stats[-1].compactions,
        "timed_update_launches_per_step": sum(s.update_launches for s in stats) // args.steps,
        "roofline": dict(roofline(w, args, stats, T, traffic_summary),
                         **algorithmic_bytes(w, last, f64, stats[-1])),
        "h_terms": h_terms(w, stats, last, T, args.steps),
    }
    if args.guard:
        # lane-audits whose row marginal was verified in float64 (the outward
        # bound excluded the rest), rejections, and the checks' (i, j) terms
        rec["guard"] = {"lane_audits": int(sum(int(x) for x in last[2].cpu().numpy())),
                        "row_verifications": stats[-1].screen_positive,
                        "rejected": stats[-1].check_failures,
                        "check_pair_evals": stats[-1].check_pair_evals}
    if not args.no_tol_sweep:
        rec["mixture_modes"], rec["mixture_tol_sweep"] = mixture_extras(args, base_flags)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, args.tol)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
