"""Plain float64 log-domain Sinkhorn, one lane at a time (test infrastructure only).

Notation follows the paper (Sec. 2, Sec. 3): lane t holds points x_i (i < n),
y_j (j < m) in R^d, marginals a, b, regularisation eps. The cost is
C_ij = ||x_i - y_j||^2 and the coupling of potentials (f, g) is
pi_ij = exp((f_i + g_j - C_ij) / eps).

Nothing here is blocked, fused or reordered beyond what the equations state,
apart from computing the dense cost matrix in row chunks to bound memory.
"""

from __future__ import annotations

import numpy as np

CONVERGED = 0
MAX_ITER = 1
NONFINITE = 2

_CHUNK_ELEMS = 1 << 24  # row-chunking of the dense cost construction only


# --------------------------------------------------------------------------- cost
def sq_euclidean_cost(x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """Dense C_ij = sum_k (x_ik - y_jk)^2 (the cost of eq:eot for point clouds).

    For d <= 16 the differences are formed directly. For larger d the identity
    ||x - y||^2 = ||x||^2 + ||y||^2 - 2 <x, y> is used with a library matmul; in
    float64 the cancellation this introduces is ~1e-16 * ||x||^2, far below every
    tolerance used here. Both branches are pinned against each other in tests.
    """
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    n, d = x.shape
    m = y.shape[0]
    if d > 16:
        xx = np.sum(x * x, axis=1)
        yy = np.sum(y * y, axis=1)
        return np.maximum(xx[:, None] + yy[None, :] - 2.0 * (x @ y.T), 0.0)
    C = np.empty((n, m), dtype=np.float64)
    rows = max(1, _CHUNK_ELEMS // max(1, m * d))
    for i0 in range(0, n, rows):
        diff = x[i0:i0 + rows, None, :] - y[None, :, :]
        C[i0:i0 + rows] = np.sum(diff * diff, axis=2)
    return C


# ------------------------------------------------------------------ half-steps
def _lse(z: np.ndarray, axis: int) -> np.ndarray:
    """log sum_axis exp(z), shifted by the max along the axis."""
    zmax = np.max(z, axis=axis, keepdims=True)
    zmax = np.where(np.isfinite(zmax), zmax, 0.0)
    return np.squeeze(zmax, axis) + np.log(np.sum(np.exp(z - zmax), axis=axis))


def f_half_step(C, g, log_a, eps):
    """First leg of eq:sinkhorn-cycle, u <- a / (K v), in log form:
    f_i = eps log a_i - eps log sum_j exp((g_j - C_ij) / eps)."""
    return eps * log_a - eps * _lse((g[None, :] - C) / eps, axis=1)


def g_half_step(C, f, log_b, eps):
    """Second leg of eq:sinkhorn-cycle, v <- b / (K^T u), in log form:
    g_j = eps log b_j - eps log sum_i exp((f_i - C_ij) / eps)."""
    return eps * log_b - eps * _lse((f[:, None] - C) / eps, axis=0)


def coupling(C, f, g, eps):
    """pi_ij = exp((f_i + g_j - C_ij) / eps) = diag(u) K diag(v) (Sec. 2)."""
    return np.exp((f[:, None] + g[None, :] - C) / eps)


def marginal_residuals(C, f, g, a, b, eps):
    """L1 residuals of both marginals, the two terms of eq:release-contract:
    (||pi 1 - a||_1, ||pi^T 1 - b||_1)."""
    P = coupling(C, f, g, eps)
    r_row = float(np.sum(np.abs(np.sum(P, axis=1) - a)))
    r_col = float(np.sum(np.abs(np.sum(P, axis=0) - b)))
    return r_row, r_col


def dual_objective(C, f, g, a, b, eps):
    """Dual of eq:eot: D(f, g) = <f, a> + <g, b> - eps sum_ij pi_ij.

    Each half-step of eq:sinkhorn-cycle maximises D exactly over one block of
    variables, so D is non-decreasing along the iteration (a pinned property).
    """
    return float(f @ a + g @ b - eps * np.sum(coupling(C, f, g, eps)))


# --------------------------------------------------------------------- one lane
def solve_lane(x, y, a, b, eps, tol, *, max_iter=5000, audit_every=1,
               fixed_iters=None, history=False, g0=None):
    """Solve one lane from a proposal (cold by default) and stop on the
    two-sided audit.

    Readings taken:
      * cold proposal f = g = 0 (all formal runs use cold proposals, Sec. 5 /
        tab:workload-configs); f is updated first (eq:sinkhorn-cycle), which
        fixes the gauge (f + c, g - c) of Sec. 4.2 -- no normalisation applied;
      * one iteration = one full cycle (f-half then g-half); max_iter counts
        cycles; the audit runs after cycle k when k % audit_every == 0 or
        k == max_iter, never at k = 0, so depth >= 1;
      * the residual is the max of the two L1 marginal errors, compared with
        an inclusive <= (eq:release-contract), on the caller's a, b as given;
      * depth = first passing audit (Sec. 4.1); the returned state is the
        audited one;
      * a non-finite residual at an audit ends the lane with NONFINITE; a lane
        still failing at max_iter ends with MAX_ITER (no sequential fallback);
      * a zero mass a_i = 0 (b_j = 0) removes that point from the problem and
        its output potential is written 0;
      * ``g0`` (length m) is a proposal (Sec. 2: carried or warm-started dual
        potentials): the iteration starts from g = g0 instead of the cold
        g = 0. Because f is updated first, only the target potential of a
        proposal enters the trajectory.

    ``fixed_iters=k`` runs exactly k cycles with no stopping test and reports
    the residual of the final state (fixed-work parity, Sec. 3.2).

    """
    dt = np.float64
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    eps = float(eps)
    if not (np.isfinite(eps) and eps > 0.0):
        raise ValueError("eps must be finite and > 0")
    n, m = a.shape[0], b.shape[0]
    row_live = a != 0.0
    col_live = b != 0.0
    xs, ys = x[row_live], y[col_live]
    av, bv = a[row_live], b[col_live]

    C = sq_euclidean_cost(xs, ys)
    with np.errstate(divide="ignore", invalid="ignore"):
        log_a = np.log(av).astype(dt)
        log_b = np.log(bv).astype(dt)
    av_t, bv_t = av.astype(dt), bv.astype(dt)
    e = dt(eps)

    f = np.zeros(xs.shape[0], dtype=dt)
    g = np.zeros(ys.shape[0], dtype=dt)
    if g0 is not None:
        g = np.asarray(g0, dtype=np.float64)[col_live].astype(dt)
    hist = []
    status, depth = MAX_ITER, 0
    r_row = r_col = np.nan
    total = fixed_iters if fixed_iters is not None else max_iter
    with np.errstate(over="ignore", invalid="ignore", divide="ignore"):
        for k in range(1, total + 1):
            f = f_half_step(C, g, log_a, e).astype(dt)
            g = g_half_step(C, f, log_b, e).astype(dt)
            if fixed_iters is not None:
                if k == total:
                    r_row, r_col = marginal_residuals(C, f, g, av_t, bv_t, e)
                    depth = k
                    r = max(r_row, r_col)
                    status = CONVERGED if r <= tol else (
                        NONFINITE if not np.isfinite(r) else MAX_ITER)
                continue
            if k % audit_every == 0 or k == max_iter:
                r_row, r_col = marginal_residuals(C, f, g, av_t, bv_t, e)
                r = max(r_row, r_col)
                if history:
                    hist.append((k, r_row, r_col))
                if not (np.isfinite(r_row) and np.isfinite(r_col)):
                    status, depth = NONFINITE, k
                    break
                if r <= tol:
                    status, depth = CONVERGED, k
                    break
                if k == max_iter:
                    status, depth = MAX_ITER, k
    f_out = np.zeros(n, dtype=np.float64)
    g_out = np.zeros(m, dtype=np.float64)
    f_out[row_live] = f
    g_out[col_live] = g
    r_row, r_col = float(r_row), float(r_col)
    residual = max(r_row, r_col) if status != NONFINITE else float("nan")
    out = dict(f=f_out, g=g_out, depth=int(depth), status=int(status),
               residual=residual, row_residual=r_row, col_residual=r_col)
    if history:
        out["history"] = hist
    return out


# ------------------------------------------------------------------------ batch
def _lane_job(args):
    return solve_lane(*args[0], **args[1])


def solve(X, Y, a, b, eps, tol, *, n=None, m=None, max_iter=5000, audit_every=1,
          fixed_iters=None, history=False, lanes=None,
          processes=None, g0=None):
    """Solve a window of W independent lanes (candidate-axis packing).

    eq:pack-commutes (Sec. 3.1): the packed map equals the per-lane maps applied
    independently, so the oracle simply solves each lane on its own. Inputs are
    [W, n_max, d], [W, m_max, d], [W, n_max], [W, m_max], eps [W]; n, m give each
    lane's valid prefix (default: full). ``lanes`` restricts the run to a subset
    of lane indices (outputs of other lanes stay zero / depth 0).
    ``processes`` > 1 spreads lanes over a process pool (largest first).
    ``g0`` [W, m_max] is an optional proposal (initial target potentials).

    Returns f [W, n_max], g [W, m_max] (zero beyond each lane's prefix), depth,
    residual, row_residual, col_residual, status [W], and ``order``: lane
    indices sorted by (depth, lane index) -- the completion order, ties broken
    by ascending lane index (one audit emits its passing lanes in lane order).
    """
    X = np.asarray(X)
    Y = np.asarray(Y)
    a = np.asarray(a)
    b = np.asarray(b)
    W, n_max = a.shape
    m_max = b.shape[1]
    eps = np.broadcast_to(np.asarray(eps, dtype=np.float64), (W,))
    n = np.full(W, n_max, dtype=np.int64) if n is None else np.asarray(n)
    m = np.full(W, m_max, dtype=np.int64) if m is None else np.asarray(m)
    lanes = list(range(W)) if lanes is None else [int(t) for t in lanes]
    kw = dict(max_iter=max_iter, audit_every=audit_every, fixed_iters=fixed_iters,
              history=history)
    jobs = [((X[t, :n[t]], Y[t, :m[t]], a[t, :n[t]], b[t, :m[t]], eps[t], tol),
             dict(kw, g0=None if g0 is None else np.asarray(g0)[t, :m[t]]))
            for t in lanes]
    if processes is not None and processes > 1 and len(jobs) > 1:
        import multiprocessing as mp
        order_big = sorted(range(len(jobs)), key=lambda q: -(n[lanes[q]] * m[lanes[q]]))
        with mp.get_context("fork").Pool(processes, initializer=_single_thread) as pool:
            res_sorted = pool.map(_lane_job, [jobs[q] for q in order_big], chunksize=1)
        results = [None] * len(jobs)
        for q, r in zip(order_big, res_sorted):
            results[q] = r
    else:
        results = [_lane_job(j) for j in jobs]

    out = dict(f=np.zeros((W, n_max)), g=np.zeros((W, m_max)),
               depth=np.zeros(W, dtype=np.int64), status=np.zeros(W, dtype=np.int64),
               residual=np.full(W, np.nan), row_residual=np.full(W, np.nan),
               col_residual=np.full(W, np.nan))
    if history:
        out["history"] = [None] * W
    for t, r in zip(lanes, results):
        out["f"][t, :n[t]] = r["f"]
        out["g"][t, :m[t]] = r["g"]
        for key in ("depth", "status", "residual", "row_residual", "col_residual"):
            out[key][t] = r[key]
        if history:
            out["history"][t] = r["history"]
    out["order"] = np.array(sorted(lanes, key=lambda t: (out["depth"][t], t)), dtype=np.int64)
    return out


def _single_thread():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:  # pragma: no cover - threadpoolctl is optional
        pass


# ------------------------------------------------------------------- accounting
def survival_widths(depths) -> np.ndarray:
    """eq:survival-width: A_k = |{t : l_t >= k}| for k = 1 .. l_max."""
    depths = np.asarray(depths, dtype=np.int64)
    lmax = int(depths.max()) if depths.size else 0
    return np.array([int(np.sum(depths >= k)) for k in range(1, lmax + 1)], dtype=np.int64)


def slot_counts(depths) -> dict:
    """eq:slot-identity and eq:removable-slots (Prop. 1).

    active  = sum_k A_k (physical width summed over packed updates),
    static  = W * l_max,
    removable R = static - sum_t l_t.
    ``active`` is computed from the survival curve, not from sum_t l_t, so that
    the identity sum_k A_k = sum_t l_t is something a test can check.
    """
    depths = np.asarray(depths, dtype=np.int64)
    W = depths.size
    lmax = int(depths.max()) if W else 0
    active = int(np.sum(survival_widths(depths)))
    static = W * lmax
    return dict(active=active, static=static, removable=static - int(np.sum(depths)),
                l_max=lmax, W=W)
