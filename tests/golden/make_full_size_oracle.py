"""Write the float64 oracle's results on full-size benchmark windows.

Usage: python tests/golden/make_full_size_oracle.py [c2] [c4] [c5] [--procs N]

Calls only ``oracle/`` (and the seeded generators of
``paper_2607_24741_amd/workloads.py``, which hold no arithmetic of the method).
For every selected lane it stores the completion depth, status, residuals, the
completion order of the selection, the potentials of the returned state
(float32), and the oracle's residuals at the audits l-2 .. l+2 around the
completion depth l (the two audits past l come from continuing the returned
state with its own g as a proposal, which continues the trajectory exactly), so
that a GPU depth one or two audits away from the oracle's can be checked
against the 1e-6 exemption band without re-running the oracle.

Windows and lane samples (tol 1e-3, max_iter 5000, audit after every cycle):
  c2  all 64 lanes of the mixture window (n = m = 1024, d = 8);
  c4  lanes 0 and 5 of the feature window (n = m = 4096, d = 512);
  c5  12 lanes of the LiDAR-shaped window spanning its size range: among the
      lanes whose estimated oracle time n m (5 / eps) 4e-8 s is at most 600 s,
      the ones at 12 evenly spaced ranks of n m (the six smallest lanes are
      compared by the GPU test itself).
"""

from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_24741_amd import workloads as wl  # noqa: E402

TOL = 1e-3
MAX_ITER = 5000
HERE = os.path.dirname(os.path.abspath(__file__))


def c5_sample(w):
    area = w.n.astype(np.int64) * w.m
    est = area * 4e-8 * 5.0 / w.eps.astype(np.float64)
    ok = np.nonzero(est <= 600.0)[0]
    ok = ok[np.argsort(area[ok], kind="stable")]
    return [int(t) for t in ok[np.linspace(0, len(ok) - 1, 12).round().astype(int)]]


def lanes_for(name, w):
    if name == "c2":
        return list(range(w.W))
    if name == "c4":
        return [0, 5]
    return c5_sample(w)


def _continue(args):
    """Residuals at the two audits after the returned state (proposal = its g)."""
    x, y, a, b, eps, g = args
    r = oracle.solve_lane(x, y, a, b, eps, 0.0, max_iter=2, history=True, g0=g)
    return [max(rr, rc) for _, rr, rc in r["history"]]


def run(name, procs):
    w = wl.make(name)
    lanes = lanes_for(name, w)
    t0 = time.time()
    o = oracle.solve(w.X, w.Y, w.a, w.b, w.eps, TOL, n=w.n, m=w.m, max_iter=MAX_ITER,
                     history=True, lanes=lanes, processes=procs)
    jobs = []
    for t in lanes:
        nt, mt = int(w.n[t]), int(w.m[t])
        jobs.append((w.X[t, :nt], w.Y[t, :mt], w.a[t, :nt], w.b[t, :mt], float(w.eps[t]),
                     o["g"][t, :mt]))
    conv = [int(o["status"][t]) == oracle.CONVERGED for t in lanes]
    import multiprocessing as mp
    todo = [j for j, c in zip(jobs, conv) if c]
    with mp.get_context("fork").Pool(procs, initializer=oracle.sinkhorn._single_thread) as pool:
        after = pool.map(_continue, todo, chunksize=1)
    r_near = np.full((len(lanes), 5), np.nan)
    it = iter(after)
    for q, t in enumerate(lanes):
        hist = {k: max(rr, rc) for k, rr, rc in o["history"][t]}
        ell = int(o["depth"][t])
        for j, k in enumerate(range(ell - 2, ell + 1)):
            r_near[q, j] = hist.get(k, np.nan)
        if conv[q]:
            r_near[q, 3:] = next(it)
    order = [int(t) for t in o["order"] if t in set(lanes)]
    out = os.path.join(HERE, f"full_size_{name}.npz")
    np.savez_compressed(
        out, lanes=np.array(lanes, np.int64), depth=o["depth"][lanes], status=o["status"][lanes],
        residual=o["residual"][lanes], row_residual=o["row_residual"][lanes],
        col_residual=o["col_residual"][lanes], order=np.array(order, np.int64),
        f=o["f"][lanes].astype(np.float32), g=o["g"][lanes].astype(np.float32), r_near=r_near,
        tol=TOL, max_iter=MAX_ITER,
        note=np.array(f"oracle (float64) on {name} lanes {lanes}; r_near = residual at audits "
                      f"depth-2 .. depth+2; written by tests/golden/make_full_size_oracle.py"))
    print(f"{name}: {len(lanes)} lanes in {time.time() - t0:.0f} s -> {out}", flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("names", nargs="*", default=["c2", "c4", "c5"])
    ap.add_argument("--procs", type=int, default=max(1, len(os.sched_getaffinity(0))))
    args = ap.parse_args()
    for name in args.names:
        run(name, args.procs)


if __name__ == "__main__":
    main()
