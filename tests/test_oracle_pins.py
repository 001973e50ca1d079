"""Pins of the float64 oracle against things other than itself.

Each test ties the oracle to what the paper or plain mathematics fixes:
closed forms, brute-force dense scaling (eq:sinkhorn-cycle as printed), an
independent dual solve, the asymptotic rate of the quotient PF analysis
(Sec. 4.2), the paper's printed slot counts (Sec. 4.1 / Sec. 5), and
invariants. A dropped term, wrong sign, transposed operand or off-by-one on
the audit grid in the oracle fails at least one of them.
"""

import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.sinkhorn import coupling

HERE = os.path.dirname(os.path.abspath(__file__))


def _lane(rng, n, m, d, scale=1.0, dirichlet=True):
    x = rng.standard_normal((n, d)) * scale
    y = rng.standard_normal((m, d)) * scale + 0.3
    if dirichlet:
        a = rng.gamma(1.0, size=n); a /= a.sum()
        b = rng.gamma(1.0, size=m); b /= b.sum()
    else:
        a = np.full(n, 1.0 / n); b = np.full(m, 1.0 / m)
    return x, y, a, b


# ------------------------------------------------------------- half-step pins
def test_half_steps_make_their_marginal_exact():
    """eq:updated-marginal: after each leg the marginal it targets is exact."""
    rng = np.random.default_rng(1)
    x, y, a, b = _lane(rng, 7, 5, 3)
    eps = 0.3
    C = oracle.sq_euclidean_cost(x, y)
    g = rng.standard_normal(5)
    f = oracle.f_half_step(C, g, np.log(a), eps)
    P = coupling(C, f, g, eps)
    assert np.abs(P.sum(1) - a).sum() < 1e-12
    g2 = oracle.g_half_step(C, f, np.log(b), eps)
    P = coupling(C, f, g2, eps)
    assert np.abs(P.sum(0) - b).sum() < 1e-12
    # and the row marginal is *not* exact in general after the g-leg
    assert np.abs(P.sum(1) - a).sum() > 1e-6


def test_dual_ascent_is_monotone():
    """Each half-step maximises D(f, g) over one block: D never decreases."""
    rng = np.random.default_rng(2)
    x, y, a, b = _lane(rng, 9, 6, 2)
    eps = 0.2
    C = oracle.sq_euclidean_cost(x, y)
    f, g = np.zeros(9), np.zeros(6)
    prev = oracle.dual_objective(C, f, g, a, b, eps)
    for _ in range(40):
        f = oracle.f_half_step(C, g, np.log(a), eps)
        cur = oracle.dual_objective(C, f, g, a, b, eps)
        assert cur >= prev - 1e-12
        prev = cur
        g = oracle.g_half_step(C, f, np.log(b), eps)
        cur = oracle.dual_objective(C, f, g, a, b, eps)
        assert cur >= prev - 1e-12
        prev = cur


@pytest.mark.parametrize("n,m,d,eps,audit", [(8, 5, 2, 0.5, 1), (5, 11, 3, 0.8, 3),
                                             (16, 16, 2, 0.4, 1), (1, 6, 2, 0.5, 2),
                                             (6, 1, 2, 0.5, 1)])
def test_matches_brute_force_dense_scaling(n, m, d, eps, audit):
    """Log-domain iterates == multiplicative u, v scaling of eq:sinkhorn-cycle."""
    rng = np.random.default_rng(n * 100 + m)
    x, y, a, b = _lane(rng, n, m, d)
    tol = 1e-6
    ref = oracle.dense_scaling_lane(x, y, a, b, eps, tol, audit_every=audit)
    got = oracle.solve_lane(x, y, a, b, eps, tol, audit_every=audit)
    assert got["depth"] == ref["depth"]
    assert got["depth"] % audit == 0 or got["depth"] == 5000
    assert got["status"] == ref["status"] == oracle.CONVERGED
    scale = max(np.abs(ref["f"]).max(), np.abs(ref["g"]).max(), eps)
    np.testing.assert_allclose(got["f"], ref["f"], rtol=0, atol=1e-10 * scale)
    np.testing.assert_allclose(got["g"], ref["g"], rtol=0, atol=1e-10 * scale)
    assert abs(got["residual"] - ref["residual"]) < 1e-12


def test_brute_force_depth_sequence_over_audit_grid():
    """Depths agree with the dense route for every audit interval 1..5, which
    pins the audit grid (first passing production audit, Sec. 4.1)."""
    rng = np.random.default_rng(7)
    x, y, a, b = _lane(rng, 10, 9, 2)
    for audit in range(1, 6):
        ref = oracle.dense_scaling_lane(x, y, a, b, 0.3, 1e-7, audit_every=audit)
        got = oracle.solve_lane(x, y, a, b, 0.3, 1e-7, audit_every=audit)
        assert got["depth"] == ref["depth"] and got["depth"] % audit == 0


# ------------------------------------------------------------- closed forms
def test_two_point_symmetric_closed_form():
    """a = b = (1/2, 1/2), C = [[0, c], [c, 0]]: with v = 1, K v = (1+q)1 and
    K^T u = 1/2, so the first cycle lands on the fixed point:
    pi_11 = 1 / (2 (1 + exp(-c/eps))), f = -eps log(2 (1 + q)), g = 0."""
    c, eps = 1.7, 0.45
    s = math.sqrt(c)
    x = np.array([[0.0], [s]])
    y = np.array([[0.0], [s]])
    a = b = np.array([0.5, 0.5])
    got = oracle.solve_lane(x, y, a, b, eps, 1e-13)
    q = math.exp(-c / eps)
    assert got["depth"] == 1
    np.testing.assert_allclose(got["f"], [-eps * math.log(2 * (1 + q))] * 2, atol=1e-14)
    np.testing.assert_allclose(got["g"], [0.0, 0.0], atol=1e-14)
    P = coupling(oracle.sq_euclidean_cost(x, y), got["f"], got["g"], eps)
    np.testing.assert_allclose(P[0, 0], 1.0 / (2.0 * (1.0 + q)), rtol=1e-14)
    np.testing.assert_allclose(P[0, 1], q / (2.0 * (1.0 + q)), rtol=1e-14)


@pytest.mark.parametrize("n", [3, 6, 9])
def test_regular_polygon_uniform_converges_in_one_cycle(n):
    """X = Y = vertices of a regular n-gon, uniform weights: K is circulant,
    K 1 = k 1, so one cycle gives pi = K / (n k) exactly."""
    th = 2 * np.pi * np.arange(n) / n
    x = np.stack([np.cos(th), np.sin(th)], 1)
    a = np.full(n, 1.0 / n)
    eps = 0.35
    got = oracle.solve_lane(x, x, a, a, eps, 1e-13)
    assert got["depth"] == 1
    C = oracle.sq_euclidean_cost(x, x)
    K = np.exp(-C / eps)
    expected = K / (n * K.sum(1)[0])
    np.testing.assert_allclose(coupling(C, got["f"], got["g"], eps), expected, rtol=1e-12)


def test_single_source_or_target_point_gives_product_coupling():
    """n = 1 (or m = 1): the only feasible plan is a b^T, reached at depth 1."""
    rng = np.random.default_rng(3)
    for n, m in [(1, 7), (7, 1)]:
        x, y, a, b = _lane(rng, n, m, 2)
        got = oracle.solve_lane(x, y, a, b, 0.1, 1e-13)
        assert got["depth"] == 1
        P = coupling(oracle.sq_euclidean_cost(x, y), got["f"], got["g"], 0.1)
        np.testing.assert_allclose(P, np.outer(a, b), rtol=1e-12, atol=1e-15)


def test_large_eps_tends_to_independent_coupling():
    """eps -> infinity: pi -> a b^T with ||pi - a b^T||_1 = O(C_max / eps)."""
    rng = np.random.default_rng(4)
    x, y, a, b = _lane(rng, 8, 6, 2)
    C = oracle.sq_euclidean_cost(x, y)
    errs = []
    for eps in [1e2 * C.max(), 1e3 * C.max()]:
        got = oracle.solve_lane(x, y, a, b, eps, 1e-14)
        P = coupling(C, got["f"], got["g"], eps)
        errs.append(np.abs(P - np.outer(a, b)).sum())
        assert errs[-1] <= 2.0 * C.max() / eps
    assert 7.0 < errs[0] / errs[1] < 13.0      # first-order in 1/eps


def test_small_eps_tends_to_optimal_assignment():
    """eps -> 0 with uniform weights, n = m: <C, pi_eps> decreases toward the
    optimal assignment cost / n (brute force over permutations), and stays
    within eps (log n + log m) of it (entropy of any coupling is bounded)."""
    rng = np.random.default_rng(5)
    n = 6
    x = 2.0 * rng.standard_normal((n, 2))
    y = x[rng.permutation(n)] + 0.2 * rng.standard_normal((n, 2))
    a = b = np.full(n, 1.0 / n)
    C = oracle.sq_euclidean_cost(x, y)
    best = min(sum(C[i, p[i]] for i in range(n)) for p in itertools.permutations(range(n))) / n
    tol = 1e-6
    slack = C.max() * tol
    prev = np.inf
    for eps in [1.0, 0.3, 0.1, 0.03]:
        got = oracle.solve_lane(x, y, a, b, eps, tol, max_iter=400000)
        assert got["status"] == oracle.CONVERGED
        val = float(np.sum(C * coupling(C, got["f"], got["g"], eps)))
        assert val <= prev + slack
        assert best - slack <= val <= best + eps * 2 * math.log(n) + slack
        prev = val
    assert prev - best < 1e-6


def test_independent_dual_solve_reproduces_fixed_point():
    """The Sinkhorn fixed point maximises D(f, g); a quasi-Newton solve of that
    smooth concave dual (no Sinkhorn steps) gives the same coupling."""
    from scipy.optimize import minimize
    rng = np.random.default_rng(6)
    n, m, eps = 6, 5, 0.4
    x, y, a, b = _lane(rng, n, m, 2)
    C = oracle.sq_euclidean_cost(x, y)

    def negD(z):
        f, g = z[:n], z[n:]
        P = np.exp((f[:, None] + g[None, :] - C) / eps)
        val = -(f @ a + g @ b - eps * P.sum())
        grad = -np.concatenate([a - P.sum(1), b - P.sum(0)])
        return val, grad

    res = minimize(negD, np.zeros(n + m), jac=True, method="L-BFGS-B",
                   options=dict(maxiter=20000, gtol=1e-14, ftol=1e-16))
    P_ref = np.exp((res.x[:n, None] + res.x[None, n:] - C) / eps)
    got = oracle.solve_lane(x, y, a, b, eps, 1e-13, max_iter=100000)
    P = coupling(C, got["f"], got["g"], eps)
    np.testing.assert_allclose(P, P_ref, atol=1e-8)


def test_asymptotic_rate_is_second_singular_value_squared():
    """Sec. 4.2: one cycle linearises to J* = P* P with P = D_a^-1/2 pi* D_b^-1/2;
    on the gauge quotient the slowest mode decays as sigma_2(P)^2 per cycle, so
    r(k+1)/r(k) -> sigma_2^2 (sigma_1 = 1 is the gauge / mass direction)."""
    rng = np.random.default_rng(8)
    n, m, eps = 12, 10, 0.25
    x, y, a, b = _lane(rng, n, m, 2)
    C = oracle.sq_euclidean_cost(x, y)
    star = oracle.solve_lane(x, y, a, b, eps, 1e-15, max_iter=200000)
    Pstar = coupling(C, star["f"], star["g"], eps)
    S = np.linalg.svd(Pstar / np.sqrt(a)[:, None] / np.sqrt(b)[None, :], compute_uv=False)
    assert abs(S[0] - 1.0) < 1e-10
    lam2 = S[1] ** 2
    run = oracle.solve_lane(x, y, a, b, eps, 0.0, max_iter=400, history=True)
    r = np.array([h[1] for h in run["history"]])
    k = int(np.nonzero(r > 1e-11)[0].max())          # last point above the float64 floor
    ratio = r[k] / r[k - 1]
    assert abs(ratio - lam2) < 2e-3 * lam2


# ------------------------------------------------------------- accounting pins
def test_slot_identity_on_random_depths():
    """eq:slot-identity: sum_k A_k = sum_t l_t, static = W l_max, R = 0 iff all
    depths equal (Prop. 2, deterministic form)."""
    rng = np.random.default_rng(9)
    for _ in range(50):
        W = int(rng.integers(1, 40))
        depths = rng.integers(1, 60, size=W)
        sc = oracle.slot_counts(depths)
        assert sc["active"] == int(depths.sum())
        assert sc["static"] == W * int(depths.max())
        assert sc["removable"] == sc["static"] - sc["active"] >= 0
        assert (sc["removable"] == 0) == bool(np.all(depths == depths[0]))
        A = oracle.survival_widths(depths)
        assert A[0] == W and np.all(np.diff(A) <= 0)


def test_slot_counts_match_paper_printed_numbers():
    with open(os.path.join(HERE, "golden", "slot_accounting.json")) as fh:
        cases = json.load(fh)["cases"]
    metro, c80lm, neutral = cases
    # MetroPT-3: W = 16, static 5696 -> l_max = 356; a depth profile on the
    # audit-every-4 grid with sum 3128 (any such profile has these counts)
    lmax = metro["static"] // metro["W"]
    assert lmax * metro["W"] == metro["static"] and lmax % 4 == 0
    depths = np.full(metro["W"], 4)
    depths[0] = lmax
    extra = (metro["active"] - depths.sum()) // 4
    i = 1
    while extra > 0:
        step = min(extra, (lmax - depths[i]) // 4)
        depths[i] += 4 * step
        extra -= step
        i += 1
    sc = oracle.slot_counts(depths)
    assert (sc["static"], sc["active"]) == (metro["static"], metro["active"])
    assert sc["removable"] == metro["static"] - metro["active"]
    # C80-LM: W = 8, 256 static slots (l_max = 32), 100 removed -> 156 active
    lmax = c80lm["static"] // c80lm["W"]
    depths = np.array([32, 32, 16, 16, 16, 16, 16, 12])
    assert depths.max() == lmax
    sc = oracle.slot_counts(depths)
    assert sc["static"] == c80lm["static"] and sc["removable"] == c80lm["removed"]
    # EXP-P19 at tol 1e-2: all lanes pass at update 8 -> nothing removable
    sc = oracle.slot_counts(np.full(neutral["W"], neutral["uniform_depth"]))
    assert sc["removable"] == neutral["removed"]


# ------------------------------------------------------------- invariants
def test_translation_and_permutation_invariance():
    rng = np.random.default_rng(10)
    x, y, a, b = _lane(rng, 9, 7, 3)
    base = oracle.solve_lane(x, y, a, b, 0.3, 1e-6)
    sh = rng.standard_normal(3) * 5
    moved = oracle.solve_lane(x + sh, y + sh, a, b, 0.3, 1e-6)
    assert moved["depth"] == base["depth"]
    np.testing.assert_allclose(moved["f"], base["f"], atol=1e-9)
    np.testing.assert_allclose(moved["g"], base["g"], atol=1e-9)
    p, q = rng.permutation(9), rng.permutation(7)
    perm = oracle.solve_lane(x[p], y[q], a[p], b[q], 0.3, 1e-6)
    assert perm["depth"] == base["depth"]
    np.testing.assert_allclose(perm["f"], base["f"][p], atol=1e-10)
    np.testing.assert_allclose(perm["g"], base["g"][q], atol=1e-10)


def test_batch_results_are_lane_independent_and_ordered():
    """eq:pack-commutes: a lane's result does not depend on its co-lanes; the
    completion order is by (depth, lane index)."""
    rng = np.random.default_rng(11)
    W, n, m, d = 5, 8, 6, 2
    X = rng.standard_normal((W, n, d)).astype(np.float32)
    Y = rng.standard_normal((W, m, d)).astype(np.float32)
    A = np.full((W, n), 1.0 / n, dtype=np.float32)
    B = np.full((W, m), 1.0 / m, dtype=np.float32)
    eps = np.array([0.1, 0.5, 0.1, 0.3, 0.5], dtype=np.float32)
    out = oracle.solve(X, Y, A, B, eps, 1e-5)
    for t in range(W):
        alone = oracle.solve_lane(X[t], Y[t], A[t], B[t], eps[t], 1e-5)
        assert alone["depth"] == out["depth"][t]
        assert np.array_equal(alone["f"], out["f"][t])
    order = list(out["order"])
    assert order == sorted(range(W), key=lambda t: (out["depth"][t], t))
    perm = [3, 0, 4, 1, 2]
    out2 = oracle.solve(X[perm], Y[perm], A[perm], B[perm], eps[perm], 1e-5)
    assert np.array_equal(out2["f"], out["f"][perm])


def test_process_pool_equals_serial_bit_for_bit():
    """The process pool (lanes dispatched largest first, results mapped back
    by lane) returns exactly the serial run's arrays, for every lane and a
    lane subset, with ragged sizes and a proposal: the GPU parity tests call
    the oracle through it."""
    rng = np.random.default_rng(21)
    W, n_max, m_max, d = 7, 14, 11, 3
    X = rng.standard_normal((W, n_max, d)).astype(np.float32)
    Y = (rng.standard_normal((W, m_max, d)) + 0.4).astype(np.float32)
    n = np.array([14, 3, 9, 14, 1, 6, 12], dtype=np.int64)
    m = np.array([11, 8, 1, 5, 11, 7, 2], dtype=np.int64)
    A = np.zeros((W, n_max), np.float32)
    B = np.zeros((W, m_max), np.float32)
    for t in range(W):
        A[t, :n[t]] = rng.dirichlet(np.ones(n[t]))
        B[t, :m[t]] = rng.dirichlet(np.ones(m[t]))
    eps = np.exp(rng.uniform(np.log(0.05), np.log(0.5), size=W)).astype(np.float32)
    g0 = (0.1 * rng.standard_normal((W, m_max))).astype(np.float32)
    for lanes in (None, [5, 0, 3]):
        kw = dict(n=n, m=m, max_iter=400, audit_every=2, history=True, lanes=lanes, g0=g0)
        ser = oracle.solve(X, Y, A, B, eps, 1e-4, **kw)
        par = oracle.solve(X, Y, A, B, eps, 1e-4, processes=4, **kw)
        for key in ("f", "g", "depth", "status", "residual", "row_residual", "col_residual",
                    "order"):
            assert np.array_equal(ser[key], par[key], equal_nan=True), key
        assert ser["history"] == par["history"]
        assert len(set(ser["depth"][ser["depth"] > 0].tolist())) > 1   # lanes really differ


def test_fixed_work_state_matches_stopping_run():
    rng = np.random.default_rng(12)
    x, y, a, b = _lane(rng, 9, 8, 2)
    stop = oracle.solve_lane(x, y, a, b, 0.2, 1e-5)
    fixed = oracle.solve_lane(x, y, a, b, 0.2, 1e-5, fixed_iters=stop["depth"])
    assert np.array_equal(stop["f"], fixed["f"]) and np.array_equal(stop["g"], fixed["g"])
    assert fixed["residual"] == stop["residual"]


def test_column_marginal_is_current_at_every_audit():
    """eq:updated-marginal: the audited state always has r_col ~ 0 in float64;
    only the row marginal carries the residual."""
    rng = np.random.default_rng(13)
    x, y, a, b = _lane(rng, 10, 12, 2)
    run = oracle.solve_lane(x, y, a, b, 0.2, 1e-8, history=True)
    for k, rr, rc in run["history"]:
        assert rc < 1e-13
        assert rr >= 0


# ---------------------------------------------------------------- proposals
def test_cold_proposal_is_the_zero_proposal():
    rng = np.random.default_rng(21)
    x, y, a, b = _lane(rng, 9, 7, 2)
    cold = oracle.solve_lane(x, y, a, b, 0.25, 1e-7)
    zero = oracle.solve_lane(x, y, a, b, 0.25, 1e-7, g0=np.zeros(7))
    for k in ("f", "g"):
        assert np.array_equal(cold[k], zero[k])
    assert cold["depth"] == zero["depth"] and cold["residual"] == zero["residual"]


@pytest.mark.parametrize("audit", [1, 3])
def test_proposal_matches_dense_scaling_from_v0(audit):
    """A proposal g0 is the starting scaling v = exp(g0 / eps) of the printed
    multiplicative iteration (eq:sinkhorn-cycle): same depth, same potentials."""
    rng = np.random.default_rng(22 + audit)
    x, y, a, b = _lane(rng, 8, 11, 2)
    eps, tol = 0.4, 1e-7
    g0 = 0.3 * rng.standard_normal(11)
    ref = oracle.dense_scaling_lane(x, y, a, b, eps, tol, audit_every=audit, v0=np.exp(g0 / eps))
    got = oracle.solve_lane(x, y, a, b, eps, tol, audit_every=audit, g0=g0)
    cold = oracle.solve_lane(x, y, a, b, eps, tol, audit_every=audit)
    assert got["depth"] == ref["depth"] and got["status"] == ref["status"] == oracle.CONVERGED
    scale = max(np.abs(ref["f"]).max(), np.abs(ref["g"]).max(), eps)
    np.testing.assert_allclose(got["f"], ref["f"], rtol=0, atol=1e-10 * scale)
    np.testing.assert_allclose(got["g"], ref["g"], rtol=0, atol=1e-10 * scale)
    # the proposal really changed the trajectory
    assert np.abs(got["f"] - cold["f"]).max() > 1e-9


def test_proposal_continues_the_cold_trajectory():
    """The iteration is a map on g: starting from the cold run's g after k
    cycles reproduces that run from cycle k + 1 on, bit for bit, and the
    stopping depth drops by exactly k (Sec. 2: a carried proposal shortens the
    completion depth)."""
    rng = np.random.default_rng(24)
    x, y, a, b = _lane(rng, 10, 9, 3)
    eps, tol = 0.3, 1e-8
    cold = oracle.solve_lane(x, y, a, b, eps, tol)
    k = cold["depth"] // 3
    assert k >= 2
    mid = oracle.solve_lane(x, y, a, b, eps, tol, fixed_iters=k)
    warm = oracle.solve_lane(x, y, a, b, eps, tol, g0=mid["g"])
    assert warm["depth"] == cold["depth"] - k
    assert np.array_equal(warm["f"], cold["f"]) and np.array_equal(warm["g"], cold["g"])
    assert warm["residual"] == cold["residual"]


def test_proposal_gauge_shift_moves_only_the_potentials():
    """(f, g) -> (f - c, g + c) leaves pi unchanged (Sec. 4.2): a proposal
    shifted by c yields the same depth and residuals and potentials shifted by
    exactly that gauge."""
    rng = np.random.default_rng(25)
    x, y, a, b = _lane(rng, 12, 8, 2)
    eps, tol, c = 0.35, 1e-8, 0.73
    mid = oracle.solve_lane(x, y, a, b, eps, tol, fixed_iters=4)
    base = oracle.solve_lane(x, y, a, b, eps, tol, g0=mid["g"])
    shift = oracle.solve_lane(x, y, a, b, eps, tol, g0=mid["g"] + c)
    assert shift["depth"] == base["depth"]
    np.testing.assert_allclose(shift["f"], base["f"] - c, rtol=0, atol=1e-12)
    np.testing.assert_allclose(shift["g"], base["g"] + c, rtol=0, atol=1e-12)
    assert abs(shift["residual"] - base["residual"]) < 1e-14


def test_batch_proposal_reaches_each_lane():
    rng = np.random.default_rng(26)
    lanes = [_lane(rng, 6, 5, 2) for _ in range(3)]
    X = np.stack([l[0] for l in lanes]); Y = np.stack([l[1] for l in lanes])
    A = np.stack([l[2] for l in lanes]); B = np.stack([l[3] for l in lanes])
    G0 = 0.2 * rng.standard_normal((3, 5))
    out = oracle.solve(X, Y, A, B, [0.3, 0.4, 0.5], 1e-7, g0=G0)
    for t in range(3):
        one = oracle.solve_lane(X[t], Y[t], A[t], B[t], [0.3, 0.4, 0.5][t], 1e-7, g0=G0[t])
        assert np.array_equal(out["f"][t], one["f"]) and out["depth"][t] == one["depth"]


# ------------------------------------------------------------- edge semantics
def test_zero_mass_point_behaves_like_padding():
    rng = np.random.default_rng(14)
    x, y, a, b = _lane(rng, 6, 5, 2)
    a0 = np.concatenate([a[:3], [0.0], a[3:]])
    x0 = np.concatenate([x[:3], [[9.0, 9.0]], x[3:]])
    base = oracle.solve_lane(x, y, a, b, 0.3, 1e-6)
    zero = oracle.solve_lane(x0, y, a0, b, 0.3, 1e-6)
    assert zero["depth"] == base["depth"]
    assert zero["f"][3] == 0.0
    np.testing.assert_array_equal(np.delete(zero["f"], 3), base["f"])


def test_nonfinite_input_ends_lane_at_first_audit():
    rng = np.random.default_rng(15)
    x, y, a, b = _lane(rng, 6, 5, 2)
    x[2, 1] = np.nan
    got = oracle.solve_lane(x, y, a, b, 0.3, 1e-6, audit_every=3)
    assert got["status"] == oracle.NONFINITE and got["depth"] == 3
    assert math.isnan(got["residual"])


def test_max_iter_status_and_depth():
    rng = np.random.default_rng(16)
    x, y, a, b = _lane(rng, 8, 8, 2)
    got = oracle.solve_lane(x, y, a, b, 0.05, 1e-9, max_iter=3)
    assert got["status"] == oracle.MAX_ITER and got["depth"] == 3
    fixed = oracle.solve_lane(x, y, a, b, 0.05, 1e-9, fixed_iters=3)
    assert got["residual"] == fixed["residual"]


def test_cost_direct_and_expanded_forms_agree():
    rng = np.random.default_rng(17)
    x = rng.standard_normal((9, 40)); y = rng.standard_normal((7, 40))
    C = oracle.sq_euclidean_cost(x, y)                      # expanded branch (d > 16)
    ref = np.array([[np.sum((xi - yj) ** 2) for yj in y] for xi in x])
    np.testing.assert_allclose(C, ref, rtol=1e-12)
    C2 = oracle.sq_euclidean_cost(x[:, :16], y[:, :16])    # direct branch
    ref2 = np.array([[np.sum((xi - yj) ** 2) for yj in y[:, :16]] for xi in x[:, :16]])
    np.testing.assert_allclose(C2, ref2, rtol=1e-14)
