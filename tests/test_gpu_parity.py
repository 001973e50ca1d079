"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded float32 inputs, plus the batch properties the paper fixes
(slot identity, bitwise lane independence, mode equivalence, padding
isolation) and edge cases. Every case prints its name before touching the GPU.
"""

import numpy as np
import pytest

import oracle
from paper_2607_24741_amd import workloads as wl
from tests.gpu_support import (EXEMPT_BAND, FP32_BAND, RES_ATOL, compare, export_rounding_bound, log,
                               procs, run_gpu, run_oracle)

pytestmark = pytest.mark.gpu

F_SHADOW, F_FORCE_VALU, F_FORCE_MFMA, F_PRECISE, F_MATERIALIZE, F_GUARD = 1, 4, 8, 16, 32, 64
F_FAST32 = 128
F_MATRIX_FREE = 256
# opt-in float32 kernels: outside the 1e-6 depth contract (see tests/gpu_support.py)
FP32_FLAGS = F_FAST32 | F_FORCE_VALU | F_FORCE_MFMA | F_MATERIALIZE


def band_for(flags, d):
    """Depth-decision band of the iterate: the contract's 1e-6 on the default
    path, FP32_BAND for the opt-in float32 kernels (and for the float32
    matrix-core default of 16 < d <= 32, where no float64-state kernel
    exists). Guarded release adds each lane's export_rounding_bound() (see
    guard_bars)."""
    if flags & FP32_FLAGS:
        return FP32_BAND
    if 16 < d <= 32 and not flags & F_PRECISE:
        return FP32_BAND
    return EXEMPT_BAND


def guard_bars(w, g, flags):
    """Per-lane depth band and residual bar of a guarded run: the iterate's
    own (band_for, RES_ATOL) plus how far rounding to the returned float32
    potentials can move the residual the guard decides on and reports."""
    extra = np.array([export_rounding_bound(w, g, t) for t in range(w.W)])
    log(f"[case] guarded: export rounding bound per lane max {extra.max():.2e} "
        f"median {np.median(extra):.2e}")
    return band_for(flags, w.d) + extra, RES_ATOL + extra


def _case(name, w, tol, flags=0, **kw):
    band = band_for(flags, w.d)
    log(f"[case] {name}: W={w.W} n_max={w.X.shape[1]} m_max={w.Y.shape[1]} d={w.d} tol={tol} "
        f"flags={flags} band={band:.0e} {kw}")
    g = run_gpu(w, tol, flags=flags, **kw)
    o = run_oracle(w, tol, **{k: v for k, v in kw.items() if k in ("max_iter", "audit_every")})
    extra = {}
    if flags & F_GUARD:
        band, extra["res_atol"] = guard_bars(w, g, flags)
    rep = compare(w, g, o, tol, audit_every=kw.get("audit_every", 1), band=band, **extra)
    log(f"[case] {name}: depths {g['depth'].tolist()} max_pot_err={rep['max_pot_err']:.2e} "
        f"max_res_err={rep['max_res_err']:.2e} near_threshold={rep['near_threshold']} "
        f"beyond_1e-6_band={rep['beyond_1e6']}")
    st = g["stats"]
    assert st.slots_update == int(g["depth"].sum())
    assert sum(st.width_trace) == st.slots_update
    return g, o, rep


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU], ids=["default", "fast32", "valu"])
def test_toy_config_full(flags):
    w = wl.make("c1")
    _case("c1", w, 1e-3, flags=flags)


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU], ids=["default", "fast32", "valu"])
def test_mixture_reduced_ragged(flags):
    w = wl.make("c2", W=6, n=200, m=176)
    _case("c2-reduced", w, 1e-2, flags=flags)


def test_telemetry_reduced():
    """MetroPT-shaped case (eps = 0.01, C/eps ~ 3e3) on the default float64
    state: depths, potentials and residuals meet the bar with no lane outside
    the 1e-6 exemption band."""
    w = wl.make("c3", W=4, n=160, m=224)
    g, o, rep = _case("c3-reduced", w, 1e-2, max_iter=4000)
    assert rep["beyond_1e6"] == 0


@pytest.mark.xfail(strict=True, reason=(
    "opt-in float32 state (deterministic, outside the depth contract): at eps=0.01 with "
    "C/eps ~ 3e3 the float32 trajectory drifts from "
    "the float64 one by about one cycle near the threshold (residual slope ~9e-6 per cycle); "
    "the fixed-work residual then differs by 1.01e-5, just over the 1e-5 residual bar"))
def test_telemetry_reduced_fast32():
    w = wl.make("c3", W=4, n=160, m=224)
    _case("c3-reduced-fast32", w, 1e-2, flags=F_FAST32, max_iter=4000)


def test_telemetry_full_size_sampled():
    """Full MetroPT-shaped window (W=256, n=m=512, d=16, eps=0.01, tol 1e-3) in
    its benchmark launch configuration, sampled lanes against the oracle:
    the default float64 state strictly (no lane outside the 1e-6 band), the
    opt-in float32 state within FP32_BAND (its near-threshold lanes are
    printed)."""
    w = wl.make("c3")
    lanes = [1, 2]
    o = run_oracle(w, 1e-3, lanes=lanes)
    for flags in (0, F_FAST32):
        log(f"[case] c3 full size flags={flags}")
        g = run_gpu(w, 1e-3, flags=flags)
        st = g["stats"]
        assert st.slots_update == int(g["depth"].sum())
        assert list(g["order"]) == sorted(range(w.W), key=lambda t: (g["depth"][t], t))
        rep = compare(w, g, o, 1e-3, lanes=lanes, check_order=False, band=band_for(flags, w.d))
        log(f"[case] c3 full flags={flags}: depths {[int(g['depth'][t]) for t in lanes]} "
            f"oracle {[int(o['depth'][t]) for t in lanes]} max_pot_err={rep['max_pot_err']:.2e} "
            f"max_res_err={rep['max_res_err']:.2e} near_threshold={rep['near_threshold']}")
        if flags == 0:
            assert rep["beyond_1e6"] == 0


def test_features_large_d_reduced_ragged():
    """d = 512 (ImageNet-feature-shaped): the materialised cost path, ragged
    sizes in one window."""
    w = wl.make("c4", W=4, n=256, m=240, hetero=(90, 256), pad_value=np.nan)
    _case("c4-reduced", w, 1e-3)


def test_matrix_free_large_d_reduced_ragged():
    """d = 512 on the K-looped matrix-core half-step (DS_F_MATRIX_FREE: the
    cost recomputed per tile instead of materialised): ragged NaN-padded lanes
    against the oracle."""
    w = wl.make("c4", W=4, n=256, m=240, hetero=(90, 256), pad_value=np.nan)
    _case("c4-reduced-matrix-free", w, 1e-3, flags=F_MATRIX_FREE)


def _wide_large_d(n, m, seed, d=40):
    """Two large-d lanes (d = 40 unless given), one with many source points and
    one with many target points (a long column operand for each half-step)."""
    rng = np.random.default_rng(seed)
    W = 2
    n, m = np.array(n, np.int32), np.array(m, np.int32)
    n_max, m_max = int(n.max()), int(m.max())
    X = np.full((W, n_max, d), np.nan, np.float32)
    Y = np.full((W, m_max, d), np.nan, np.float32)
    a = np.full((W, n_max), np.nan, np.float32)
    b = np.full((W, m_max), np.nan, np.float32)
    for t in range(W):
        X[t, :n[t]] = rng.standard_normal((n[t], d)) / np.sqrt(d)
        Y[t, :m[t]] = (rng.standard_normal((m[t], d)) + 0.3) / np.sqrt(d)
        aa = rng.gamma(1.0, size=n[t]); a[t, :n[t]] = aa / aa.sum()
        bb = rng.gamma(1.0, size=m[t]); b[t, :m[t]] = bb / bb.sum()
    eps = np.array([0.1, 0.15], np.float32)
    return wl.Workload("large-d-wide", X, Y, a, b, eps, n, m, 1e-3, 5000)


def test_large_d_beyond_the_materialised_limit():
    """At d > 32 a side with more than 16384 points cannot be materialised:
    the default is then the matrix-free half-step (d = 40, one lane with 16500
    source points and one with 16400 target points)."""
    w = _wide_large_d([16500, 300], [200, 16400], 17)
    _case("large-d beyond 16384 points", w, 1e-3)


@pytest.mark.parametrize("flags", [0, F_MATRIX_FREE], ids=["materialised", "matrix-free"])
def test_large_d_odd_dimension(flags):
    """d = 37 (neither even nor a multiple of the 32-coordinate stages): the
    zero-padded point records of the matrix-free kernel, the clamped loads of
    the cost build and the centre's partial coordinate block, on ragged
    NaN-padded lanes."""
    w = _wide_large_d([300, 170], [130, 260], 23, d=37)
    _case("large-d odd dimension", w, 1e-3, flags=flags)


def test_materialised_cost_long_column_operand():
    """The materialised cost with a column operand beyond 8192 points (staged
    whole in LDS, up to 16384): d = 40, one lane with 12000 source points and
    one with 9000 target points."""
    w = _wide_large_d([12000, 300], [200, 9000], 19)
    _case("materialised, 9000-12000 points a side", w, 1e-3)


@pytest.mark.parametrize("name", ["c2", "c5"])
def test_materialised_cost_small_d(name):
    """The materialised cost on request at small d: parity on the mixture
    window and on NaN-padded heterogeneous lanes."""
    if name == "c2":
        w, kw = wl.make("c2", W=6, n=200, m=176), {}
    else:
        w, kw = wl.make("c5", W=8, n=400, m=360, hetero=(40, 400), pad_value=np.nan), dict(max_iter=3000)
    _case(f"{name}-materialised", w, 1e-2 if name == "c2" else 1e-3, flags=F_MATERIALIZE, **kw)


def test_features_full_size_sampled():
    """Full ImageNet-feature-shaped window (W=32, n=m=4096, d=512) in its
    launch configuration: fixed work (3 cycles) of one lane against the
    oracle, then a real solve at tol 1e-3 whose returned potentials the oracle
    re-evaluates (float64 residual <= tol + 1e-5, equal to the reported one)."""
    w = wl.make("c4")
    log("[case] c4 full size fixed work 3 cycles")
    g = run_gpu(w, 1e-9, max_iter=3)
    t = 5
    fw = oracle.solve_lane(w.X[t], w.Y[t], w.a[t], w.b[t], w.eps[t], 1e-9, fixed_iters=3)
    scale = max(np.abs(fw["f"]).max(), np.abs(fw["g"]).max(), float(w.eps[t]))
    err = max(np.abs(g["f"][t] - fw["f"]).max(), np.abs(g["g"][t] - fw["g"]).max()) / scale
    log(f"  lane {t}: pot err {err:.2e}, res gpu {g['residual'][t]:.6e} or {fw['residual']:.6e}")
    assert err <= 1e-4
    assert abs(g["residual"][t] - fw["residual"]) <= 1e-5
    log("[case] c4 full size tol 1e-3")
    g = run_gpu(w, 1e-3)
    st = g["stats"]
    assert np.all(g["status"] == oracle.CONVERGED)
    assert st.slots_update == int(g["depth"].sum())
    assert list(g["order"]) == sorted(range(w.W), key=lambda q: (g["depth"][q], q))
    C = oracle.sq_euclidean_cost(w.X[t], w.Y[t])
    rr, rc = oracle.marginal_residuals(C, g["f"][t], g["g"][t], w.a[t].astype(np.float64),
                                       w.b[t].astype(np.float64), float(w.eps[t]))
    log(f"  lane {t}: depth {g['depth'][t]} f64 residual of gpu state {max(rr, rc):.6e} "
        f"reported {g['residual'][t]:.6e}")
    assert max(rr, rc) <= 1e-3 + 1e-5
    assert abs(max(rr, rc) - g["residual"][t]) <= 1e-5


def test_lidar_full_size_sampled():
    """Full LiDAR-shaped window (W=1024; n, m uniform on 256..8192, padded to
    8192; d=3; per-lane eps on 0.005..0.1; tol 1e-3) in the library's
    automatic launch configuration (two sub-batches, mixed lane shapes): (i) fixed work, 8
    cycles: the lane nearest 2048 x 2048 points against the oracle's state;
    (ii) a real solve: the six smallest lanes against the oracle (depths,
    potentials, residuals), the largest lane's returned potentials
    re-evaluated in float64 (its residual equals the reported one), and the
    batch properties (statuses, slot identity, width trace, completion order)."""
    w = wl.make("c5")
    area = w.n.astype(np.int64) * w.m
    t_mid = int(np.argmin(np.abs(area - 2048 * 2048)))
    log(f"[case] c5 full size fixed work 8 cycles (lane {t_mid}: {w.n[t_mid]} x {w.m[t_mid]})")
    g = run_gpu(w, 1e-9, max_iter=8)
    assert np.all(g["depth"] == 8) and np.all(g["status"] == oracle.MAX_ITER)
    nt, mt = int(w.n[t_mid]), int(w.m[t_mid])
    fw = oracle.solve_lane(w.X[t_mid, :nt], w.Y[t_mid, :mt], w.a[t_mid, :nt], w.b[t_mid, :mt],
                           w.eps[t_mid], 1e-9, fixed_iters=8)
    scale = max(np.abs(fw["f"]).max(), np.abs(fw["g"]).max(), float(w.eps[t_mid]))
    err = max(np.abs(g["f"][t_mid, :nt] - fw["f"]).max(),
              np.abs(g["g"][t_mid, :mt] - fw["g"]).max()) / scale
    log(f"  lane {t_mid}: pot err {err:.2e}, res gpu {g['residual'][t_mid]:.6e} "
        f"or {fw['residual']:.6e}")
    assert err <= 1e-4
    assert abs(g["residual"][t_mid] - fw["residual"]) <= 1e-5
    log("[case] c5 full size tol 1e-3")
    g = run_gpu(w, 1e-3)
    st = g["stats"]
    assert st.sub_batches == 2
    conv = g["status"] == oracle.CONVERGED
    assert np.all(conv | ((g["status"] == oracle.MAX_ITER) & (g["depth"] == 5000)))
    assert np.all(g["residual"][conv] <= 1e-3)
    assert st.slots_update == int(g["depth"].sum())
    assert list(g["order"]) == sorted(range(w.W), key=lambda t: (g["depth"][t], t))
    small = [int(t) for t in np.argsort(area, kind="stable")[:6]]
    o = run_oracle(w, 1e-3, lanes=small)
    rep = compare(w, g, o, 1e-3, lanes=small, check_order=False, band=band_for(0, w.d))
    log(f"  lanes {small}: depths {[int(g['depth'][t]) for t in small]} oracle "
        f"{[int(o['depth'][t]) for t in small]} max_pot_err={rep['max_pot_err']:.2e} "
        f"max_res_err={rep['max_res_err']:.2e} near_threshold={rep['near_threshold']}")
    t = int(np.argmax(area))
    nt, mt = int(w.n[t]), int(w.m[t])
    C = oracle.sq_euclidean_cost(w.X[t, :nt], w.Y[t, :mt])
    rr, rc = oracle.marginal_residuals(C, g["f"][t, :nt], g["g"][t, :mt],
                                       w.a[t, :nt].astype(np.float64),
                                       w.b[t, :mt].astype(np.float64), float(w.eps[t]))
    log(f"  lane {t} ({nt} x {mt}): depth {g['depth'][t]} status {g['status'][t]} f64 residual "
        f"of gpu state {max(rr, rc):.6e} reported {g['residual'][t]:.6e}")
    assert abs(max(rr, rc) - g["residual"][t]) <= 1e-5
    if conv[t]:
        assert max(rr, rc) <= 1e-3 + 1e-5


@pytest.mark.parametrize("name", ["c1", "c5"])
def test_precise_state_small_cases(name):
    """Float64 state on the toy window and on NaN-padded heterogeneous lanes
    (ingest, compaction and emission of the float64 arrays)."""
    if name == "c1":
        w, kw = wl.make("c1"), {}
    else:
        w, kw = wl.make("c5", W=8, n=400, m=360, hetero=(40, 400), pad_value=np.nan), dict(max_iter=3000)
    g, o, rep = _case(f"{name}-precise", w, 1e-3, flags=F_PRECISE, **kw)
    assert rep["beyond_1e6"] == 0


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU], ids=["default", "fast32", "valu"])
def test_heterogeneous_nan_padded(flags):
    w = wl.make("c5", W=8, n=400, m=360, hetero=(40, 400), pad_value=np.nan)
    _case("c5-hetero", w, 1e-3, flags=flags, max_iter=3000)


def test_audit_grid_every_three():
    w = wl.make("c2", W=4, n=96, m=96)
    g, o, _ = _case("c2-audit3", w, 1e-2, audit_every=3)
    assert np.all(g["depth"] % 3 == 0)


def test_full_size_mixture_fixed_work_and_residual_property():
    """Full c2 shape (W=64, n=m=1024, d=8) in the benchmark's launch config:
    (i) fixed work: 30 cycles with an unreachable tol, sampled lanes against the
    oracle's state after 30 cycles; (ii) a real solve at tol 1e-3: the float64
    residual of the returned potentials of sampled lanes is <= tol (+ fp32
    slack) and matches the reported residual; slot identity holds."""
    w = wl.make("c2")
    log("[case] c2-full fixed work 30 cycles")
    g = run_gpu(w, 1e-9, max_iter=30)
    assert np.all(g["depth"] == 30) and np.all(g["status"] == oracle.MAX_ITER)
    for t in (0, 37):
        fw = oracle.solve_lane(w.X[t], w.Y[t], w.a[t], w.b[t], w.eps[t], 1e-9, fixed_iters=30)
        scale = max(np.abs(fw["f"]).max(), np.abs(fw["g"]).max())
        err = max(np.abs(g["f"][t] - fw["f"]).max(), np.abs(g["g"][t] - fw["g"]).max()) / scale
        log(f"  lane {t}: pot err {err:.2e}, res gpu {g['residual'][t]:.6e} or {fw['residual']:.6e}")
        assert err <= 1e-4
        assert abs(g["residual"][t] - fw["residual"]) <= 1e-5
    log("[case] c2-full tol 1e-3")
    g = run_gpu(w, 1e-3)
    st = g["stats"]
    conv = g["status"] == oracle.CONVERGED
    # lanes that need more than max_iter cycles stop at the cap, still failing
    assert np.all(conv | ((g["status"] == oracle.MAX_ITER) & (g["depth"] == 5000)))
    assert np.all(g["residual"][conv] <= 1e-3) and np.all(g["residual"][~conv] > 1e-3)
    assert st.slots_update == int(g["depth"].sum())
    A = np.array(st.width_trace)
    assert A[0] == 64 and np.all(np.diff(A) <= 0) and A.sum() == g["depth"].sum()
    assert list(g["order"]) == sorted(range(64), key=lambda t: (g["depth"][t], t))
    for t in [int(x) for x in np.nonzero(conv)[0][[0, -1]]]:
        C = oracle.sq_euclidean_cost(w.X[t], w.Y[t])
        rr, rc = oracle.marginal_residuals(C, g["f"][t], g["g"][t], w.a[t].astype(np.float64),
                                           w.b[t].astype(np.float64), float(w.eps[t]))
        log(f"  lane {t}: depth {g['depth'][t]} f64 residual of gpu state {max(rr, rc):.6e} "
            f"reported {g['residual'][t]:.6e}")
        assert max(rr, rc) <= 1e-3 + 1e-5
        assert abs(max(rr, rc) - g["residual"][t]) <= 1e-5


def _static_at_lmax(w, gs, fixed, pot_bar):
    for t in range(w.W):
        scale = max(np.abs(fixed["f"][t]).max(), np.abs(fixed["g"][t]).max(), float(w.eps[t]))
        err = max(np.abs(gs["f"][t] - fixed["f"][t]).max(),
                  np.abs(gs["g"][t] - fixed["g"][t]).max()) / scale
        if pot_bar is not None:
            assert err <= pot_bar, (t, err)
        assert abs(gs["residual"][t] - fixed["residual"][t]) <= 1e-5
        assert gs["residual"][t] <= 1e-3 + 1e-5


def test_modes_agree_and_account_slots():
    """Logical masking returns exactly the active outputs (compaction does no
    arithmetic); static packing records the same first passing depths and
    returns every lane's state at the common final boundary l_max: bit for bit
    the state a fixed-work run of l_max cycles returns, and (float64 state)
    the oracle's at l_max (float64 state; the float32 state is compared
    through its residual only: near a fixed point every cycle repeats nearly
    the same rounding errors, which add up along the slowest-contracting
    direction -- lane 4 of this window, eps 0.133, depth 103, residual still
    3e-5 at cycle 1022, drifts by up to 1.9e-4 relative over 919 extra
    cycles while its residual stays within 2e-7 of the oracle's)."""
    w = wl.make("c1")
    log("[case] modes on c1")
    ga = run_gpu(w, 1e-3, mode="active")
    gl = run_gpu(w, 1e-3, mode="logical")
    gs = run_gpu(w, 1e-3, mode="static")
    for k in ("f", "g", "depth", "residual", "status", "order"):
        assert np.array_equal(ga[k], gl[k]), k
    assert np.array_equal(ga["depth"], gs["depth"])
    assert np.array_equal(ga["order"], gs["order"])
    lmax = int(ga["depth"].max())
    assert ga["stats"].slots_update == int(ga["depth"].sum())
    assert gl["stats"].slots_update == w.W * lmax
    assert gs["stats"].slots_update == w.W * lmax
    sc = oracle.slot_counts(ga["depth"])
    assert sc["active"] == ga["stats"].slots_update and sc["static"] == gs["stats"].slots_update
    log(f"[case] modes on c1: fixed work {lmax} cycles")
    gf = run_gpu(w, 1e-30, max_iter=lmax)
    for k in ("f", "g", "residual"):
        assert np.array_equal(gs[k], gf[k]), k
    fixed = oracle.solve(w.X, w.Y, w.a, w.b, w.eps, 1e-3, n=w.n, m=w.m, fixed_iters=lmax)
    _static_at_lmax(w, gs, fixed, 1e-4)
    log("[case] modes on c1: static, float32 state")
    gp = run_gpu(w, 1e-3, mode="static", flags=F_FAST32)
    lp = int(gp["depth"].max())
    if lp != lmax:
        fixed = oracle.solve(w.X, w.Y, w.a, w.b, w.eps, 1e-3, n=w.n, m=w.m, fixed_iters=lp)
    _static_at_lmax(w, gp, fixed, None)


def test_bitwise_lane_independence_and_determinism():
    w = wl.make("c2", W=6, n=150, m=130)
    log("[case] lane independence")
    g = run_gpu(w, 1e-2)
    g2 = run_gpu(w, 1e-2)
    for k in ("f", "g", "depth", "residual"):
        assert np.array_equal(g[k], g2[k]), k
    perm = [4, 1, 5, 0, 3, 2]
    wp = wl.make("c2", lanes=perm, n=150, m=130)
    gp = run_gpu(wp, 1e-2)
    for q, t in enumerate(perm):
        assert np.array_equal(gp["f"][q], g["f"][t]) and gp["depth"][q] == g["depth"][t]
    solo = run_gpu(wl.make("c2", lanes=[3], n=150, m=130), 1e-2)
    assert np.array_equal(solo["f"][0], g["f"][3]) and np.array_equal(solo["g"][0], g["g"][3])
    assert solo["depth"][0] == g["depth"][3]


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU, F_MATERIALIZE],
                         ids=["default", "fast32", "valu", "materialised"])
@pytest.mark.parametrize("cfg", ["c2", "c3"])
def test_launch_layouts_are_bitwise_identical(cfg, flags):
    """The host picks the update kernel's work layout (row tiles and column
    groups per wave) from each launch's width and column count; a lane's bits
    must not depend on it. Fixed work on full lanes in one sub-batch: the whole
    window and a middle subset (two groups per wave for c2's 1024 columns, four
    for c3's 512) against four lanes (one group per wave)."""
    w = wl.make(cfg)
    log(f"[case] layouts {cfg} flags={flags}: W={w.W} fixed work 12 cycles")
    g = run_gpu(w, 1e-9, max_iter=12, flags=flags, streams=1)
    middle = list(range(20)) if cfg == "c2" else list(range(3, 123, 3))
    for lanes in (middle, [5, 17, 33, 60]):
        log(f"[case] layouts {cfg} flags={flags}: lanes {lanes[:4]}... ({len(lanes)})")
        gs = run_gpu(wl.make(cfg, lanes=lanes), 1e-9, max_iter=12, flags=flags, streams=1)
        for q, t in enumerate(lanes):
            assert np.array_equal(gs["f"][q], g["f"][t]), (t, "f")
            assert np.array_equal(gs["g"][q], g["g"][t]), (t, "g")
            assert gs["residual"][q] == g["residual"][t], t


def test_mixed_shape_layouts_are_bitwise_identical():
    """Mixed lane shapes (offsets-table placement): the whole window runs the
    four-groups-per-wave layout (at most 512 columns, over 512 work items per
    launch), four lanes the narrowest one; a lane's bits must not change, and
    fixed work matches the oracle on sampled lanes."""
    w = wl.make("c5", W=64, n=512, m=480, hetero=(40, 512))
    log("[case] mixed-shape layouts: W=64 fixed work 12 cycles")
    g = run_gpu(w, 1e-9, max_iter=12, streams=1)
    lanes = [2, 19, 40, 63]
    log(f"[case] mixed-shape layouts: lanes {lanes}")
    gs = run_gpu(wl.make("c5", lanes=lanes, n=512, m=480, hetero=(40, 512)), 1e-9, max_iter=12,
                 streams=1)
    for q, t in enumerate(lanes):
        assert np.array_equal(gs["f"][q], g["f"][t]), (t, "f")
        assert np.array_equal(gs["g"][q], g["g"][t]), (t, "g")
        assert gs["residual"][q] == g["residual"][t], t
    for t in lanes[:2]:
        nt, mt = int(w.n[t]), int(w.m[t])
        fw = oracle.solve_lane(w.X[t, :nt], w.Y[t, :mt], w.a[t, :nt], w.b[t, :mt], w.eps[t], 1e-9,
                               fixed_iters=12)
        scale = max(np.abs(fw["f"]).max(), np.abs(fw["g"]).max(), float(w.eps[t]))
        err = max(np.abs(g["f"][t, :nt] - fw["f"]).max(),
                  np.abs(g["g"][t, :mt] - fw["g"]).max()) / scale
        assert err <= 1e-4, (t, err)
        assert abs(g["residual"][t] - fw["residual"]) <= 1e-5


@pytest.mark.parametrize("cfg", ["c2", "c5"])
def test_sub_batches_are_bitwise_identical(cfg):
    """Sub-batches (concurrent lane ranges, each with its own control loop and
    stream) change where a lane runs, never what it computes: every output of
    the split solve equals the one-batch solve bit for bit, and so do the
    work counts. Uniform shapes (c2 lanes) and mixed shapes (c5 lanes)."""
    if cfg == "c2":
        w = wl.make("c2", W=24, n=256, m=256)
    else:
        w = wl.make("c5", W=24, n=600, m=600, hetero=(40, 600))
        # with a proposal: each sub-batch must read its own lanes' rows of it
        rng = np.random.default_rng(5)
        w.g0 = (0.01 * rng.standard_normal((w.W, w.Y.shape[1]))).astype(np.float32)
    log(f"[case] sub-batches {cfg}: W={w.W} tol 1e-3, streams 1")
    base = run_gpu(w, 1e-3, max_iter=3000, streams=1)
    for s in (2, 3, 4):
        log(f"[case] sub-batches {cfg}: streams {s}")
        g = run_gpu(w, 1e-3, max_iter=3000, streams=s)
        for k in ("f", "g", "depth", "residual", "row_residual", "col_residual", "status", "order"):
            assert np.array_equal(g[k], base[k], equal_nan=True), (s, k)
        for k in ("slots_update", "pair_evals", "halfsteps_executed", "l_max", "check_pair_evals"):
            assert getattr(g["stats"], k) == getattr(base["stats"], k), (s, k)


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU, F_MATERIALIZE],
                         ids=["default", "fast32", "valu", "materialised"])
def test_proposal_parity(flags):
    """A proposal g0 (Sec. 2: a carried or warm-started target potential)
    replaces the cold start and the GPU follows the oracle's trajectory from
    the same float32 g0. Ragged c2-shaped lanes; g0 is the oracle's own state
    after 12 cycles shifted by a per-lane gauge constant (the shift must come
    back out exactly in the potentials, Sec. 4.2), except lane 0, which gets a
    random g0. g0 is NaN past each lane's prefix (never read)."""
    w = wl.make("c2", W=6, n=200, m=176)
    mid = oracle.solve(w.X, w.Y, w.a, w.b, w.eps, 1e-2, n=w.n, m=w.m, fixed_iters=12,
                       processes=procs())
    rng = np.random.default_rng(9)
    g0 = mid["g"] + rng.uniform(-1.0, 1.0, size=(w.W, 1))
    g0[0] = 0.05 * rng.standard_normal(w.Y.shape[1])
    for t in range(w.W):
        g0[t, int(w.m[t]):] = np.nan
    w.g0 = g0.astype(np.float32)
    g, o, rep = _case("c2-reduced-proposal", w, 1e-2, flags=flags)
    cold = run_oracle(wl.make("c2", W=6, n=200, m=176), 1e-2)
    # carried lanes start 12 cycles in: they finish no later than from cold
    assert np.all(o["depth"][1:] <= cold["depth"][1:])


def _certified(w, g, tol, lanes, require_tol=True):
    """Recompute, in float64 on the host, both marginal residuals of exactly the
    float32 potentials the GPU returned (cost from the float32 coordinates): the
    guarded release reports that residual, and a converged lane meets tol
    (`require_tol`: the returned state is the one that passed)."""
    worst = 0.0
    for t in lanes:
        nt, mt = int(w.n[t]), int(w.m[t])
        a, b = w.a[t, :nt].astype(np.float64), w.b[t, :mt].astype(np.float64)
        ra, cb = a != 0, b != 0
        C = oracle.sq_euclidean_cost(w.X[t, :nt][ra], w.Y[t, :mt][cb])
        rr, rc = oracle.marginal_residuals(C, g["f"][t, :nt][ra], g["g"][t, :mt][cb], a[ra], b[cb],
                                           float(w.eps[t]))
        r = max(rr, rc)
        err = abs(g["residual"][t] - r)
        worst = max(worst, err / max(r, 1e-12))
        assert err <= 1e-7 * r + 1e-12, (t, g["residual"][t], r)
        if require_tol and g["status"][t] == oracle.CONVERGED:
            assert r <= float(np.float32(tol)) + 1e-12, (t, r)
    return worst


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU, F_MATERIALIZE],
                         ids=["default", "fast32", "valu", "materialised"])
def test_guarded_release_certifies_returned_potentials(flags):
    """DS_F_GUARD: screen-ready lanes are verified by a float64 evaluation of
    both marginals of the float32 potentials the caller receives; the release
    decision and the reported residual are that evaluation. Parity with the
    oracle as usual, and the returned potentials' own residual, recomputed on
    the host in float64, equals the reported one to float32 rounding and meets
    tol for every converged lane (eq:release-contract)."""
    w = wl.make("c2", W=6, n=200, m=176)
    g, o, rep = _case("c2-reduced-guard", w, 1e-2, flags=flags | F_GUARD)
    worst = _certified(w, g, 1e-2, range(w.W))
    log(f"[case] c2-reduced-guard: worst relative residual difference {worst:.2e}")
    assert g["stats"].check_pair_evals > 0


def test_guarded_release_mixed_shapes_and_final_audit():
    """Mixed lane shapes with zero-mass points, several sub-batches, and lanes
    that end at max_iter (the final audit runs the float64 check on every lane
    still running)."""
    w = wl.make("c5", W=12, n=400, m=380, hetero=(30, 400))
    w.a[2, 5] = 0.0
    w.a[2] /= w.a[2].sum()
    w.b[7, 3] = 0.0
    w.b[7] /= w.b[7].sum()
    g, o, rep = _case("c5-reduced-guard", w, 1e-3, flags=F_GUARD,
                      max_iter=60, streams=2)
    assert np.any(g["status"] == oracle.MAX_ITER)
    _certified(w, g, 1e-3, range(w.W))


def test_guarded_release_in_every_mode():
    """Guarded release under logical masking and static packing (eq:slot-identity
    modes): logical returns exactly the active outputs; static keeps every
    lane's first passing depth, status and the completion order, returns each
    lane's state at the common final boundary, and reports the residual the
    final float64 audit measured on exactly those returned potentials."""
    w = wl.make("c1")
    log("[case] guarded release: active, logical, static on c1")
    ga = run_gpu(w, 1e-3, mode="active", flags=F_GUARD)
    gl = run_gpu(w, 1e-3, mode="logical", flags=F_GUARD)
    gs = run_gpu(w, 1e-3, mode="static", flags=F_GUARD)
    for k in ("f", "g", "depth", "residual", "status", "order"):
        assert np.array_equal(ga[k], gl[k], equal_nan=True), k
    for k in ("depth", "status", "order"):
        assert np.array_equal(ga[k], gs[k]), k
    lmax = int(ga["depth"].max())
    assert gs["stats"].slots_update == w.W * lmax
    _certified(w, ga, 1e-3, range(w.W))
    _certified(w, gs, 1e-3, range(w.W), require_tol=False)


def _guard_windows():
    return {
        "stress": (lambda: _stress_lanes(), 1e-3, dict(max_iter=3000)),
        "telemetry": (lambda: wl.make("c3", W=4, n=160, m=224), 1e-2, dict(max_iter=4000)),
        "mixture": (lambda: wl.make("c2", W=6, n=200, m=176), 1e-2, {}),
        "lidar-final-audit": (lambda: wl.make("c5", W=12, n=400, m=380, hetero=(30, 400)), 1e-3,
                              dict(max_iter=60, streams=2)),
    }


@pytest.mark.parametrize("name", ["stress", "telemetry", "mixture", "lidar-final-audit"])
def test_guard_outward_bound_excludes_no_ready_lane(name):
    """Guarded release with the float64 state verifies only the lanes whose
    row residual the outward bound cannot place above tol (Sec. 5.4, C10
    finite-precision stress). The same solve in shadow mode verifies the row
    marginal of every lane at every audit and counts the audits where the
    bound had excluded a lane whose verified row residual met tol: none. The
    gate changes no decision (bitwise equal outputs), saves verifications, and
    the decisions agree with the oracle's up to each lane's derived band."""
    make, tol, kw = _guard_windows()[name]
    w = make()
    log(f"[case] guard bound {name}: guarded, then guarded + shadow")
    g = run_gpu(w, tol, flags=F_GUARD, **kw)
    h = run_gpu(w, tol, flags=F_GUARD | F_SHADOW, **kw)
    st, sh = g["stats"], h["stats"]
    log(f"[case] guard bound {name}: verified rows {st.screen_positive} of {sh.screen_positive} "
        f"audited, check pairs {st.check_pair_evals:.3e} vs {sh.check_pair_evals:.3e}, "
        f"excluded-but-ready {sh.guard_missed}")
    assert sh.guard_missed == 0
    for k in ("f", "g", "residual"):
        assert np.array_equal(g[k], h[k], equal_nan=True), k
    for k in ("depth", "status", "order"):
        assert np.array_equal(g[k], h[k]), k
    assert st.screen_positive < sh.screen_positive
    assert st.check_pair_evals < sh.check_pair_evals
    o = run_oracle(w, tol, **{k: v for k, v in kw.items() if k == "max_iter"})
    band, res_atol = guard_bars(w, g, 0)
    rep = compare(w, g, o, tol, band=band, res_atol=res_atol)
    differ = int((g["depth"] != o["depth"]).sum() + (g["status"] != o["status"]).sum())
    log(f"[case] guard bound {name}: decisions differing from the oracle {differ}/{w.W}, each "
        f"within its lane's band: {rep['near_threshold']}")
    _certified(w, g, tol, range(w.W))


@pytest.mark.parametrize("shape", ["uniform", "mixed"])
def test_guard_verification_grid_is_bitwise_identical(shape):
    """The float64 verification cuts every lane's columns into eight fixed
    chunks and adds each row's chunk sums in chunk order; its launches stride
    at most 2048 blocks over the (row block, chunk) units of the lanes they
    verify. The final audit of a max_iter window verifies both marginals of
    every lane: over 4096 row blocks (each block takes about sixteen units in
    turn), over 2048, over 1024, and four lanes (one unit per block). A lane's
    outputs must not depend on which."""
    if shape == "uniform":
        make = lambda lanes: wl.make("c2", lanes=lanes, n=1024, m=1024)
        W = 520                                   # 8 row blocks per lane
        middle = list(range(0, W, 4))             # 130 lanes
    else:
        make = lambda lanes: wl.make("c5", lanes=lanes, n=1024, m=1024, hetero=(600, 1024))
        W = 720                                   # 5 to 8 row blocks per lane
        middle = list(range(0, W, 3))             # 240 lanes
    half = list(range(1, W, 2))
    few = [3, 77, 200, W - 1]
    log(f"[case] guard verification grid {shape}: W={W}, 3 cycles, tol 1e-9")
    g = run_gpu(make(list(range(W))), 1e-9, max_iter=3, flags=F_GUARD, streams=1)
    assert np.all(g["status"] == oracle.MAX_ITER)
    for lanes in (half, middle, few):
        log(f"[case] guard verification grid {shape}: {len(lanes)} lanes")
        gs = run_gpu(make(lanes), 1e-9, max_iter=3, flags=F_GUARD, streams=1)
        for q, t in enumerate(lanes):
            for k in ("f", "g", "residual", "row_residual", "col_residual", "status", "depth"):
                assert np.array_equal(gs[k][q], g[k][t], equal_nan=True), (t, k)


@pytest.mark.parametrize("k", range(24))
def test_randomised_windows(k):
    """Seeded random small windows (W 1..12, sizes 1..320 per lane, d 1..40,
    Gaussian or uniform clouds, Dirichlet(0.3 / 1 / 5) masses, tol 1e-2 or
    1e-3, audit every 1-3 cycles, default / vector-ALU / float64 /
    materialised / guarded paths, 0-2 sub-batches) against the oracle."""
    w, opt = wl.random_window(k)
    flags, streams = opt["flags"], opt["streams"]
    g, o, rep = _case(f"random{k}", w, opt["tol"], flags=flags,
                      audit_every=opt["audit_every"], max_iter=w.max_iter, streams=streams)
    assert np.all(g["status"] == oracle.CONVERGED)
    if flags == F_GUARD:
        _certified(w, g, opt["tol"], range(w.W))


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU], ids=["default", "fast32", "valu"])
@pytest.mark.parametrize("d", [1, 2])
def test_low_dimensional_lanes(d, flags):
    """d = 1 and 2 (a contraction of K = 4 on the matrix cores, the smallest
    augmented vectors): ragged lanes against the oracle."""
    rng = np.random.default_rng(11 + d)
    W, n_max, m_max = 5, 150, 130
    n = np.array([150, 37, 1, 90, 64], dtype=np.int32)
    m = np.array([130, 1, 41, 77, 128], dtype=np.int32)
    X = np.full((W, n_max, d), np.nan, np.float32)
    Y = np.full((W, m_max, d), np.nan, np.float32)
    a = np.full((W, n_max), np.nan, np.float32)
    b = np.full((W, m_max), np.nan, np.float32)
    for t in range(W):
        X[t, :n[t]] = rng.standard_normal((n[t], d))
        Y[t, :m[t]] = rng.standard_normal((m[t], d)) * 1.5 + 0.7
        aa = rng.gamma(1.0, size=n[t]); a[t, :n[t]] = aa / aa.sum()
        bb = rng.gamma(1.0, size=m[t]); b[t, :m[t]] = bb / bb.sum()
    eps = np.array([0.1, 0.3, 0.05, 0.2, 0.08], np.float32)
    w = wl.Workload(f"d{d}", X, Y, a, b, eps, n, m, 1e-3, 5000)
    _case(f"d{d}", w, 1e-3, flags=flags)


def test_padding_isolation():
    log("[case] NaN vs zero padding")
    wn = wl.make("c5", W=6, n=300, m=300, hetero=(30, 300), pad_value=np.nan)
    wz = wl.make("c5", W=6, n=300, m=300, hetero=(30, 300), pad_value=0.0)
    gn = run_gpu(wn, 1e-3, max_iter=500)
    gz = run_gpu(wz, 1e-3, max_iter=500)
    for k in ("f", "g", "depth", "residual", "status"):
        assert np.array_equal(gn[k], gz[k]), k
    assert np.all(np.isfinite(gn["f"]))


@pytest.mark.parametrize("flags", [0, F_FAST32], ids=["default", "fast32"])
@pytest.mark.parametrize("cfg", ["c1", "c2"])
def test_shadow_replay_screen_against_full_row_check(cfg, flags):
    """Shadow replay (Sec. 5.3): every lane is fully checked at every audit, so
    no releasable lane may be missed by the screen, and the row marginal of
    every audited state is recomputed by a dedicated pass over (i, j): the
    fused screen (read off the next f-update, eq:updated-marginal) must agree
    with it far below the 1e-6 band on the default path. The outputs equal
    the plain run's bit for bit (the shadow work only measures)."""
    w, tol = (wl.make("c1"), 1e-3) if cfg == "c1" else (wl.make("c2", W=6, n=200, m=176), 1e-2)
    log(f"[case] shadow replay {cfg} flags={flags}")
    g = run_gpu(w, tol, flags=F_SHADOW | flags)
    st = g["stats"]
    log(f"[case] shadow replay {cfg} flags={flags}: missed_ready {st.missed_ready}, screen "
        f"discrepancy {st.screen_discrepancy:.3e}, depths {g['depth'].tolist()}")
    assert st.missed_ready == 0
    if flags == 0:
        assert st.screen_discrepancy <= 1e-7
    base = run_gpu(w, tol, flags=flags)
    for k in ("f", "g", "depth", "residual", "status"):
        assert np.array_equal(g[k], base[k]), k


def _tiny_lanes():
    rng = np.random.default_rng(3)
    W, n_max, m_max, d = 5, 40, 33, 3
    X = rng.standard_normal((W, n_max, d)).astype(np.float32)
    Y = (rng.standard_normal((W, m_max, d)) + 0.5).astype(np.float32)
    n = np.array([1, 40, 7, 40, 13], dtype=np.int32)
    m = np.array([33, 1, 9, 33, 20], dtype=np.int32)
    a = np.zeros((W, n_max), np.float32)
    b = np.zeros((W, m_max), np.float32)
    for t in range(W):
        aa = rng.gamma(1.0, size=n[t]); a[t, :n[t]] = aa / aa.sum()
        bb = rng.gamma(1.0, size=m[t]); b[t, :m[t]] = bb / bb.sum()
    eps = np.array([0.3, 0.2, 0.5, 0.1, 0.25], np.float32)
    return wl.Workload("tiny", X, Y, a, b, eps, n, m, 1e-4, 5000)


@pytest.mark.parametrize("flags", [0, F_FAST32, F_FORCE_VALU], ids=["default", "fast32", "valu"])
def test_edge_single_points_and_tiny_lanes(flags):
    w = _tiny_lanes()
    _case("tiny", w, 1e-4, flags=flags)


def _stress_lanes(W=100, seed=23):
    """100 small lanes of different shapes and regularisations (d = 3,
    sizes 40..160, Gaussian clouds at scale s, Dirichlet(1) masses, eps per
    lane s^2 logU(0.02, 0.2)): at tol 1e-3 most of them move by only a few
    1e-6 per cycle near the threshold, where a decision is most fragile."""
    rng = np.random.default_rng(seed)
    n_max = m_max = 160
    d = 3
    X = np.full((W, n_max, d), np.nan, np.float32)
    Y = np.full((W, m_max, d), np.nan, np.float32)
    a = np.full((W, n_max), np.nan, np.float32)
    b = np.full((W, m_max), np.nan, np.float32)
    n = rng.integers(40, n_max + 1, size=W).astype(np.int32)
    m = rng.integers(40, m_max + 1, size=W).astype(np.int32)
    eps = np.zeros(W, np.float32)
    for t in range(W):
        sc = float(np.exp(rng.uniform(np.log(0.5), np.log(2.0))))
        X[t, :n[t]] = sc * rng.standard_normal((n[t], d))
        Y[t, :m[t]] = sc * (rng.standard_normal((m[t], d)) + rng.uniform(0, 1, size=d))
        a[t, :n[t]] = rng.dirichlet(np.ones(n[t]))
        b[t, :m[t]] = rng.dirichlet(np.ones(m[t]))
        eps[t] = sc * sc * float(np.exp(rng.uniform(np.log(0.02), np.log(0.2))))
    return wl.Workload("stress", X, Y, a, b, eps, n, m, 1e-3, 3000)


def test_near_threshold_decisions_against_the_oracle():
    """C10-style stress (Sec. 5.4): release decisions of 100 lanes against the
    float64 oracle's. The default float64 state must decide every lane as the
    oracle does (a lane within 1e-6 of tol exempt); the opt-in float32 state's
    disagreements are counted and printed, as are the near-threshold lanes
    (crossing within 5e-6 of tol)."""
    w = _stress_lanes()
    o = run_oracle(w, 1e-3, max_iter=w.max_iter)
    near = 0
    for t in range(w.W):
        h = {k: max(r1, r2) for k, r1, r2 in o["history"][t]}
        ell = int(o["depth"][t])
        pair = [h[k] for k in (ell - 1, ell) if k in h]
        near += int(min(abs(r - 1e-3) for r in pair) <= 5e-6)
    res = {}
    for name, flags in (("default", 0), ("fast32", F_FAST32)):
        log(f"[case] stress {name}")
        g = run_gpu(w, 1e-3, flags=flags, max_iter=w.max_iter)
        res[name] = int((g["depth"] != o["depth"]).sum() + (g["status"] != o["status"]).sum())
        if name == "default":
            rep = compare(w, g, o, 1e-3, band=EXEMPT_BAND)
            assert rep["beyond_1e6"] == 0
    log(f"[case] stress: {near}/100 lanes cross within 5e-6 of tol; decisions differing from "
        f"the oracle: default {res['default']}/100, fast32 {res['fast32']}/100")
    assert res["default"] == 0 or all(m <= EXEMPT_BAND for _, _, _, m in rep["near_threshold"])


def test_edge_max_iter_and_single_lane():
    w = _tiny_lanes()
    log("[case] max_iter=1 and 3")
    for mi in (1, 3):
        # lanes with a single point on one side are exact after one cycle;
        # the others cannot reach 1e-6 in 3 cycles
        g = run_gpu(w, 1e-6, max_iter=mi)
        o = run_oracle(w, 1e-6, max_iter=mi)
        assert np.all(g["depth"] == o["depth"])
        assert np.array_equal(g["status"], o["status"])
        assert list(g["status"]) == [0, 0, 1, 1, 1]
        compare(w, g, o, 1e-6, max_iter=mi)
    one = wl.make("c1", lanes=[5])
    log("[case] W=1")
    _case("w1", one, 1e-3)


def _max_width_lanes(eps_lo, eps_hi, max_iter, W=4096, seed=11):
    """The widest call the library accepts (4096 lanes): small ragged lanes
    (1 to 48 points a side, some with a single point), d = 3, eps per lane
    log-uniform in [eps_lo, eps_hi]."""
    rng = np.random.default_rng(seed)
    n_max = m_max = 48
    d = 3
    X = rng.standard_normal((W, n_max, d)).astype(np.float32)
    Y = (rng.standard_normal((W, m_max, d)) + 0.5).astype(np.float32)
    n = rng.integers(1, n_max + 1, size=W).astype(np.int32)
    m = rng.integers(1, m_max + 1, size=W).astype(np.int32)
    n[-1], m[-1] = n_max, m_max
    a = np.zeros((W, n_max), np.float32)
    b = np.zeros((W, m_max), np.float32)
    for t in range(W):
        aa = rng.gamma(1.0, size=n[t]); a[t, :n[t]] = aa / aa.sum()
        bb = rng.gamma(1.0, size=m[t]); b[t, :m[t]] = bb / bb.sum()
    eps = np.exp(rng.uniform(np.log(eps_lo), np.log(eps_hi), size=W)).astype(np.float32)
    return wl.Workload("max-width", X, Y, a, b, eps, n, m, 1e-3, max_iter)


def test_edge_max_width():
    # every lane against the oracle at the width limit, with the automatic
    # sub-batch split; eps in [0.25, 1] lets every lane complete within the cap
    w = _max_width_lanes(0.25, 1.0, 1000)
    g, o, rep = _case("max-width", w, 1e-3, max_iter=1000)
    assert g["stats"].sub_batches >= 2
    assert np.all(g["status"] == oracle.CONVERGED)


def test_edge_max_width_capped_lanes_float64_state():
    # Smaller eps leaves a few hundred of the 4096 lanes at the 400-cycle cap,
    # some of them half-way through the escape from a residual plateau (n = 14,
    # m = 3, eps = 0.065: 0.085 for 300 cycles, then 0.060 at the cap). There
    # the residual moves by about 5e-4 per cycle, and the float32 state's
    # rounding, a fraction of a cycle of that motion, moved it by 4.4e-5 from
    # the oracle's at equal depth (potentials within 1e-4). The float64 state
    # follows the oracle's trajectory: every lane, capped or not, meets the
    # parity bar.
    w = _max_width_lanes(0.05, 0.5, 400)
    g, o, rep = _case("max-width float64 state", w, 1e-3, flags=F_PRECISE, max_iter=400)
    assert g["stats"].sub_batches >= 2
    assert int((g["status"] == oracle.MAX_ITER).sum()) > 100


def test_edge_nonfinite_and_zero_mass():
    w = _tiny_lanes()
    w.X[2, 3, 1] = np.nan           # lane 2 non-finite
    w.a[3, 5] = 0.0                 # lane 3 zero mass (point removed)
    w.a[3, :40] /= w.a[3, :40].astype(np.float64).sum()
    log("[case] nonfinite + zero mass")
    g = run_gpu(w, 1e-4, audit_every=2)
    o = run_oracle(w, 1e-4, audit_every=2)
    assert g["status"][2] == oracle.NONFINITE and g["depth"][2] == o["depth"][2] == 2
    assert np.isnan(g["residual"][2])
    assert g["f"][3, 5] == 0.0
    compare(w, g, o, 1e-4, audit_every=2, lanes=[0, 1, 3, 4], check_order=False)


def test_invalid_lane_data_is_a_call_error():
    import paper_2607_24741_amd as ds
    w = _tiny_lanes()
    w.eps[1] = -1.0
    log("[case] invalid eps")
    with pytest.raises(ds.DSError) as ei:
        run_gpu(w, 1e-4)
    assert ei.value.code == 1 and "lane 1" in str(ei.value)
    w = _tiny_lanes()
    w.n[4] = 41
    with pytest.raises(ds.DSError) as ei:
        run_gpu(w, 1e-4)
    assert ei.value.code == 1 and "lane 4" in str(ei.value)
    # in the second of two sub-batches: named by the caller's lane index, and
    # the library stays usable afterwards
    log("[case] invalid eps in a second sub-batch")
    w = _tiny_lanes()
    w.eps[3] = float("nan")
    with pytest.raises(ds.DSError) as ei:
        run_gpu(w, 1e-4, streams=2)
    assert ei.value.code == 1 and "lane 3" in str(ei.value)
    g = run_gpu(_tiny_lanes(), 1e-4, streams=2)
    assert g["stats"].sub_batches == 2 and np.all(g["status"] == oracle.CONVERGED)


def test_caller_outputs_and_workspace_reuse():
    # caller-provided outputs without the optional ones (the library gets NULL
    # for them) and one workspace reused across calls give the default call's
    # bits
    import torch
    import paper_2607_24741_amd as ds
    from tests.gpu_support import to_device
    w = wl.make("c1")
    log("[case] caller outputs + workspace reuse (c1)")
    dv = to_device(w)
    args = (dv["X"], dv["Y"], dv["a"], dv["b"], dv["eps"], 1e-3)
    ref = ds.solve(*args, n=dv["n"], m=dv["m"])
    need = ds.workspace_bytes(w.W, w.X.shape[1], w.Y.shape[1], w.d, tol=1e-3)
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda:0")
    for _ in range(2):
        out = dict(f=torch.full((w.W, w.X.shape[1]), 7.0, device="cuda:0"),
                   g=torch.full((w.W, w.Y.shape[1]), 7.0, device="cuda:0"),
                   depth=torch.zeros(w.W, dtype=torch.int32, device="cuda:0"),
                   residual=torch.zeros(w.W, device="cuda:0"),
                   status=torch.full((w.W,), 9, dtype=torch.int32, device="cuda:0"))
        got = ds.solve(*args, n=dv["n"], m=dv["m"], workspace=ws, out=out)
        torch.cuda.synchronize()
        assert got[5] is None
        for a_, b_ in zip(got[:5], ref[:5]):
            assert torch.equal(a_, b_)


def test_concurrent_calls_from_host_threads():
    # distinct workspaces used at once from two host threads, each on a stream
    # of its own (one call split into two sub-batches): the library's per-device
    # resource pool hands each call its own resources, and every result equals
    # the sequential call's bits
    import threading
    import torch
    import paper_2607_24741_amd as ds
    from tests.gpu_support import to_device
    log("[case] concurrent calls from two host threads (c1 with two sub-batches, tiny lanes)")
    jobs = [(to_device(wl.make("c1")), 1e-3, 2), (to_device(_tiny_lanes()), 1e-4, 0)]

    def call(dv, tol, streams):
        return ds.solve(dv["X"], dv["Y"], dv["a"], dv["b"], dv["eps"], tol, n=dv["n"], m=dv["m"],
                        streams=streams)

    ref = [call(*j) for j in jobs]
    torch.cuda.synchronize()
    got = [[None] * 3 for _ in jobs]
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for r in range(3):
                    got[i][r] = call(*jobs[i])
            s.synchronize()
        except Exception as e:  # pragma: no cover - reported below
            errors.append(e)

    th = [threading.Thread(target=worker, args=(i,)) for i in range(len(jobs))]
    for t in th:
        t.start()
    for t in th:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in th)
    assert not errors, errors
    torch.cuda.synchronize()
    for i in range(len(jobs)):
        for r in range(3):
            for a_, b_ in zip(got[i][r], ref[i]):
                assert torch.equal(a_, b_)
