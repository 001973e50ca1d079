"""Seeded generator checks (CPU): determinism, lane independence, shapes,
marginals, heterogeneous sizes and padding."""

import numpy as np
import pytest

from paper_2607_24741_amd import workloads as wl


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c5"])
def test_same_seed_same_bytes_and_lane_independence(name):
    kw = dict(n=96, m=80) if name != "c1" else {}
    a = wl.make(name, W=3, **kw)
    b = wl.make(name, W=3, **kw)
    for f in ("X", "Y", "a", "b", "eps", "n", "m"):
        assert np.array_equal(getattr(a, f), getattr(b, f), equal_nan=True)
    solo = wl.make(name, lanes=[2], **kw)
    assert np.array_equal(solo.X[0], a.X[2], equal_nan=True)
    assert np.array_equal(solo.b[0], a.b[2], equal_nan=True)
    assert solo.eps[0] == a.eps[2]


def test_shapes_and_marginals():
    for name in ["c1", "c2", "c3"]:
        cfg = wl.CONFIGS[name]
        w = wl.make(name, W=2, n=min(cfg["n"], 128), m=min(cfg["m"], 128))
        assert w.X.dtype == np.float32 and w.X.shape[2] == cfg["d"]
        for t in range(w.W):
            assert abs(w.a[t, :w.n[t]].astype(np.float64).sum() - 1) < 1e-6
            assert abs(w.b[t, :w.m[t]].astype(np.float64).sum() - 1) < 1e-6
            assert np.all(w.a[t, :w.n[t]] > 0) and np.all(w.b[t, :w.m[t]] > 0)
    w = wl.make("c1")
    assert np.all((w.eps >= 0.02 - 1e-7) & (w.eps <= 0.2 + 1e-7))
    assert len(set(w.eps.tolist())) == w.W


def test_features_are_unit_norm_and_clustered():
    w = wl.make("c4", W=1, n=256, m=256)
    nrm = np.linalg.norm(w.X[0].astype(np.float64), axis=1)
    assert np.allclose(nrm, 1.0, atol=1e-6)


def test_heterogeneous_sizes_and_nan_padding():
    w = wl.make("c5", W=16, n=1024, m=1024, hetero=(256, 1024), pad_value=np.nan)
    assert np.all((w.n >= 256) & (w.n <= 1024)) and np.all((w.m >= 256) & (w.m <= 1024))
    assert len(set(w.n.tolist())) > 4
    for t in range(w.W):
        assert np.all(np.isnan(w.X[t, w.n[t]:])) and np.all(np.isfinite(w.X[t, :w.n[t]]))
        assert np.all(np.isnan(w.a[t, w.n[t]:]))
    assert np.all((w.eps >= 0.005 - 1e-7) & (w.eps <= 0.1 + 1e-7))


def test_random_windows_are_seeded_and_well_formed():
    for k in range(24):
        w, opt = wl.random_window(k)
        w2, opt2 = wl.random_window(k)
        assert opt == opt2
        for f in ("X", "Y", "a", "b", "eps", "n", "m"):
            assert np.array_equal(getattr(w, f), getattr(w2, f), equal_nan=True)
        assert 1 <= w.W <= 12 and 1 <= w.d <= 40
        assert opt["flags"] in (0, 4, 16, 32, 64, 128) and opt["audit_every"] in (1, 2, 3)
        if w.d > 16:
            assert opt["flags"] != 16
        if w.d > 32:
            assert opt["flags"] in (0, 64)
        for t in range(w.W):
            nt, mt = int(w.n[t]), int(w.m[t])
            assert 1 <= nt <= w.X.shape[1] and 1 <= mt <= w.Y.shape[1]
            assert abs(w.a[t, :nt].astype(np.float64).sum() - 1) < 1e-5
            assert abs(w.b[t, :mt].astype(np.float64).sum() - 1) < 1e-5
            assert np.all(np.isfinite(w.X[t, :nt])) and np.all(np.isnan(w.X[t, nt:]))
            assert np.all(np.isnan(w.b[t, mt:])) and w.eps[t] > 0
