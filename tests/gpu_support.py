"""Helpers for the GPU parity tests: run a seeded workload through the C ABI
and compare with the float64 oracle on the same float32 bytes.

Parity bar (readings of the stated tolerances):
  * potentials: max_i |f_gpu - f_or| / max(||f_or||_inf, ||g_or||_inf, eps) <= 1e-4
    (likewise for g);
  * residuals: |r_gpu - r_or| <= 1e-5 absolute;
  * depths, statuses and completion order exact, except for lanes whose
    residual lies within 1e-6 of tol: a differing depth or status is accepted
    only when the oracle's own residual trajectory is within EXEMPT_BAND of tol
    at every audit where the two decisions differ (every audit at which the
    GPU continued has r_or >= tol - 1e-6, and the audit at which it stopped has
    r_or <= tol + 1e-6); such a lane is then compared at fixed work (the
    oracle's state at the GPU's depth), and every such margin is printed.

The 1e-6 band is the contract of the default path (the float64 state for
d <= 16, the materialised cost above 32). The opt-in float32 kernels
(DS_F_FAST32, DS_F_FORCE_VALU, DS_F_FORCE_MFMA, DS_F_MATERIALIZE at small d)
round the scaled coordinates and potentials to float32, which moves residual
trajectories by 1e-6..1e-5; their tests pass band=FP32_BAND and still count
the lanes outside the 1e-6 band (report["beyond_1e6"]).

Guarded release (DS_F_GUARD) reports, and decides on, the residual of the
float32 potentials it returns rather than of the iterate. Its tests widen the
residual bar and the depth band of each lane by export_rounding_bound(): how
far rounding to those float32 values can move the residual, derived from the
returned values themselves (half an ulp each), the masses and eps.
"""

from __future__ import annotations

import os
import sys

import numpy as np

import oracle

POT_RTOL = 1e-4
RES_ATOL = 1e-5
EXEMPT_BAND = 1e-6
FP32_BAND = 1e-5     # depth-decision band of the opt-in float32 kernels (outside the contract)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def procs():
    try:
        n = len(os.sched_getaffinity(0))
    except Exception:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def to_device(w, device="cuda:0"):
    import torch
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(device)
    g0 = getattr(w, "g0", None)   # optional proposal [W, m_max] float32
    return dict(X=t(w.X), Y=t(w.Y), a=t(w.a), b=t(w.b), eps=t(w.eps), n=t(w.n), m=t(w.m),
                g0=None if g0 is None else t(g0))


def run_gpu(w, tol, *, device="cuda:0", **kw):
    import torch
    import paper_2607_24741_amd as ds
    dv = to_device(w, device)
    out = ds.solve(dv["X"], dv["Y"], dv["a"], dv["b"], dv["eps"], tol, n=dv["n"], m=dv["m"],
                   g0=dv["g0"], return_stats=True, trace_len=kw.pop("trace_len", 20000), **kw)
    f, g, depth, res, status, order, st = out
    torch.cuda.synchronize()
    return dict(f=f.cpu().numpy().astype(np.float64), g=g.cpu().numpy().astype(np.float64),
                depth=depth.cpu().numpy(), residual=res.cpu().numpy().astype(np.float64),
                row_residual=st.row_residual.cpu().numpy().astype(np.float64),
                col_residual=st.col_residual.cpu().numpy().astype(np.float64),
                status=status.cpu().numpy(), order=order.cpu().numpy(), stats=st)


def run_oracle(w, tol, *, lanes=None, **kw):
    return oracle.solve(w.X, w.Y, w.a, w.b, w.eps, tol, n=w.n, m=w.m, history=True,
                        lanes=lanes, processes=procs(), g0=getattr(w, "g0", None), **kw)


def export_rounding_bound(w, g, t):
    """Upper bound on |r(U) - r(f, g)| for lane t, U the float32 potentials the
    GPU returned and (f, g) any state they round from: every |U_i - f_i| is at
    most half an ulp of U_i, each coupling entry then moves by a factor
    exp((df_i + dg_j) / eps), and with |e^x - 1| <= |x| e^|x| the row residual
    moves by at most e^D / eps (sum_i R_i |df_i| + sum_j C_j |dg_j|),
    D = (max |df| + max |dg|) / eps, with sum_i R_i |df_i| <= <a, |df|> + r max|df|
    and C_j <= b_j (1 + 1e-5) (the column marginal after a g-half). The same
    bound holds for the column residual with the roles exchanged."""
    nt, mt = int(w.n[t]), int(w.m[t])
    a, b = w.a[t, :nt].astype(np.float64), w.b[t, :mt].astype(np.float64)
    fu = np.abs(g["f"][t, :nt].astype(np.float32))
    gu = np.abs(g["g"][t, :mt].astype(np.float32))
    hf = np.where(a != 0, np.spacing(fu).astype(np.float64) / 2, 0.0)
    hg = np.where(b != 0, np.spacing(gu).astype(np.float64) / 2, 0.0)
    eps = float(w.eps[t])
    r = float(g["residual"][t]) if np.isfinite(g["residual"][t]) else 1.0
    mx = max(hf.max(initial=0.0), hg.max(initial=0.0))
    side = max((a * hf).sum() + (1 + 1e-5) * (b * hg).sum(), (b * hg).sum() + (1 + 1e-5) * (a * hf).sum())
    return float(np.exp(2 * mx / eps) / eps * (side + r * mx))


def pot_err(fg, fo, gg, go, eps):
    scale = max(np.abs(fo).max(), np.abs(go).max(), eps)
    return max(np.abs(fg - fo).max(), np.abs(gg - go).max()) / scale


def decision_consistent(w, t, tol, depth_gpu, status_gpu, audit_every, band=EXEMPT_BAND):
    """Is the GPU's stop decision for lane t consistent with the oracle's own
    residual trajectory within `band`? Every audit at which the GPU kept going
    must have r_or >= tol - band, and the audit at which it stopped (if it
    converged) must have r_or <= tol + band. Returns (ok, worst margin)."""
    nt, mt = int(w.n[t]), int(w.m[t])
    g0 = getattr(w, "g0", None)
    run = oracle.solve_lane(w.X[t, :nt], w.Y[t, :mt], w.a[t, :nt], w.b[t, :mt], w.eps[t], 0.0,
                            max_iter=depth_gpu, audit_every=audit_every, history=True,
                            g0=None if g0 is None else g0[t, :mt])
    r = {k: max(a, b) for k, a, b in run["history"]}
    worst = 0.0
    for k, rk in r.items():
        if k < depth_gpu:
            worst = max(worst, tol - rk)          # GPU continued: needs rk > tol
    if status_gpu == oracle.CONVERGED:
        worst = max(worst, r[depth_gpu] - tol)    # GPU stopped: needs rk <= tol
    return worst <= band, worst, run


def compare(w, g, o, tol, *, audit_every=1, max_iter=5000, lanes=None, check_order=True,
            res_atol=RES_ATOL, band=EXEMPT_BAND):
    """Assert the parity bar lane by lane; returns a report dict.

    Depth or status mismatches are accepted only when the GPU's decision is
    consistent with the oracle's residual trajectory within `band` (1e-6 on
    the default path); such lanes are compared at fixed work (the oracle's
    state at the GPU's depth) and listed in report["near_threshold"] with
    their margin; report["beyond_1e6"] counts those whose margin exceeds the
    1e-6 band (nonzero only where a test passes the wider FP32_BAND).
    """
    lanes = range(w.W) if lanes is None else lanes
    report = dict(max_pot_err=0.0, max_res_err=0.0, near_threshold=[], beyond_1e6=0)
    per_lane = lambda v, t: float(v[t]) if np.ndim(v) else float(v)
    for t in lanes:
        nt, mt = int(w.n[t]), int(w.m[t])
        dg, do = int(g["depth"][t]), int(o["depth"][t])
        sg, so = int(g["status"][t]), int(o["status"][t])
        ref_f, ref_g, ref_r = o["f"][t, :nt], o["g"][t, :mt], o["residual"][t]
        band_t = per_lane(band, t)
        if dg != do or sg != so:
            ok, margin, fw = decision_consistent(w, t, tol, dg, sg, audit_every, band=band_t)
            report["near_threshold"].append((t, dg, do, margin))
            if margin > EXEMPT_BAND:
                report["beyond_1e6"] += 1
            assert ok, (f"lane {t}: gpu depth/status ({dg},{sg}) vs oracle ({do},{so}): the "
                        f"oracle's residual is {margin:.3e} from tol, outside the {band_t:.2e} band")
            ref_f, ref_g, ref_r = fw["f"], fw["g"], fw["residual"]
        e = pot_err(g["f"][t, :nt], ref_f, g["g"][t, :mt], ref_g, float(w.eps[t]))
        report["max_pot_err"] = max(report["max_pot_err"], e)
        assert e <= POT_RTOL, (t, e)
        if sg != oracle.NONFINITE:
            re_ = abs(g["residual"][t] - ref_r)
            report["max_res_err"] = max(report["max_res_err"], re_)
            assert re_ <= per_lane(res_atol, t), (t, g["residual"][t], ref_r, per_lane(res_atol, t))
        # padded tails are written zero
        assert np.all(g["f"][t, nt:] == 0) and np.all(g["g"][t, mt:] == 0)
    sel = set(lanes)
    got = [int(x) for x in g["order"] if int(x) in sel]
    # the GPU's completion order is its own (depth, lane id) order; it equals
    # the oracle's order whenever no lane sits at the threshold
    assert got == sorted(sel, key=lambda t: (int(g["depth"][t]), t))
    if check_order and not report["near_threshold"]:
        exp = [int(x) for x in o["order"] if int(x) in sel]
        assert got == exp, (got, exp)
    return report
