"""Brute-force dense Sinkhorn scaling on tiny inputs (test infrastructure only).

This is eq:sinkhorn-cycle (Sec. 3.1) exactly as printed -- multiplicative
scalings u, v of the Gibbs kernel K = exp(-C / eps), starting from v = 1 -- with
no log-domain stabilisation. It is valid only while K does not underflow
(max C / eps < ~600), i.e. for the tiny cases it is used on. It serves as an
independent route to the same iterates as the log-domain oracle: the two agree
iff the log-domain half-steps are the printed scalings in disguise.
"""

from __future__ import annotations

import numpy as np


def dense_scaling_lane(x, y, a, b, eps, tol, *, max_iter=5000, audit_every=1, v0=None):
    """Returns f = eps log u, g = eps log v, depth, row/col residuals, status.

    Status codes are the oracle's: 0 converged, 1 max-iter. ``v0`` is the
    starting column scaling (a proposal; default v = 1).
    """
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    # C by explicit double loop: the plainest possible statement of the cost
    n, m = x.shape[0], y.shape[0]
    C = np.empty((n, m))
    for i in range(n):
        for j in range(m):
            C[i, j] = float(np.sum((x[i] - y[j]) ** 2))
    if C.max() / eps > 600.0:
        raise ValueError("dense scaling would underflow; use a smaller C/eps")
    K = np.exp(-C / eps)
    v = np.ones(m) if v0 is None else np.asarray(v0, dtype=np.float64).copy()
    u = np.ones(n)
    status, depth = 1, max_iter
    r_row = r_col = np.nan
    for k in range(1, max_iter + 1):
        u = a / (K @ v)
        v = b / (K.T @ u)
        if k % audit_every == 0 or k == max_iter:
            P = u[:, None] * K * v[None, :]
            r_row = float(np.abs(P.sum(axis=1) - a).sum())
            r_col = float(np.abs(P.sum(axis=0) - b).sum())
            if max(r_row, r_col) <= tol:
                status, depth = 0, k
                break
    return dict(f=eps * np.log(u), g=eps * np.log(v), depth=depth, status=status,
                row_residual=r_row, col_residual=r_col, residual=max(r_row, r_col))
