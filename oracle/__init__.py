"""Float64 CPU oracle for batched entropic-OT Sinkhorn with per-lane stopping.

THIS PACKAGE IS TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it. The GPU library
(``paper_2607_24741_amd``) never imports, links or calls anything here, and
nothing here imports the GPU library: the two share no code. The only module
both sides consume is the seeded input generator
(``paper_2607_24741_amd/workloads.py``), which holds none of the method's
arithmetic, and the oracle does not import even that.

What it computes (DrainSinkhorn, arxiv 2607.24741):

* eq:eot (Sec. 2) -- entropic OT between positive unit-mass marginals a, b with
  squared-Euclidean cost; the dual potentials (f, g) define the coupling
  pi_ij = exp((f_i + g_j - C_ij) / eps).
* eq:sinkhorn-cycle (Sec. 3.1) -- one cycle u <- a / (K v), v <- b / (K^T u),
  written here in log form on the potentials f = eps log u, g = eps log v.
* eq:release-contract (Sec. 3.2) -- the two-sided L1 stopping rule
  max(||pi 1 - a||_1, ||pi^T 1 - b||_1) <= tol, evaluated on the audit grid
  (Sec. 4.1: the completion depth is the first passing production audit).
* eq:slot-identity / eq:removable-slots (Sec. 4.1, Prop. 1) -- the slot
  accounting of static versus shrinking active execution.

Each reading of a point the paper leaves open is stated at the function that
takes it.

Parity status: every public function here is pinned by tests in
``tests/test_oracle_pins.py`` against closed forms, brute-force dense scaling,
an independent dual solve, or invariants the paper states. The paper prints no
potentials, plans or residual trajectories for any concrete input, so values on
the paper's own workloads are "parity unpinned" (no such values exist to pin to).
"""

from .sinkhorn import (  # noqa: F401
    CONVERGED,
    MAX_ITER,
    NONFINITE,
    sq_euclidean_cost,
    f_half_step,
    g_half_step,
    marginal_residuals,
    dual_objective,
    solve_lane,
    solve,
    survival_widths,
    slot_counts,
)
from .dense import dense_scaling_lane  # noqa: F401
