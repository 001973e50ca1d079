"""Seeded synthetic workloads shaped like the paper's evaluation campaigns.

This module only draws random numbers: it holds none of the method's
arithmetic (no cost, no log-sum-exp, no residual), so both the GPU library's
tests and the float64 oracle can consume its output without sharing code.

Every lane is drawn from its own stream, ``SeedSequence([seed, cfg], spawn_key=(t,))``,
so a lane's data depends only on (config, lane index) -- never on W or on
which other lanes are generated. Sampling and normalisation are float64; the
result is cast to float32 once, and both the GPU path and the oracle consume
those same float32 bytes.

The paper's datasets (MetroPT-3 telemetry, Packer19 scRNA, ImageNet-32 PCA500
features, A2D2 LiDAR) are not available; the recipes below are stand-ins with
the shapes, sizes and value structure of those workloads; where the paper's
description of a workload is open, the choice is stated in the recipe's docstring.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED = 260724741

#: residual tolerances of the Packer19-style sweep (tab:packer-pareto, Sec. 5.2)
TOL_SWEEP = (1e-2, 3e-3, 1e-3, 3e-4, 1e-4)


@dataclass
class Workload:
    name: str
    X: np.ndarray      # [W, n_max, d] float32
    Y: np.ndarray      # [W, m_max, d] float32
    a: np.ndarray      # [W, n_max]   float32
    b: np.ndarray      # [W, m_max]   float32
    eps: np.ndarray    # [W]          float32
    n: np.ndarray      # [W]          int32
    m: np.ndarray      # [W]          int32
    tol: float
    max_iter: int
    meta: dict = field(default_factory=dict)

    @property
    def W(self):
        return self.a.shape[0]

    @property
    def d(self):
        return self.X.shape[2]


def _rng(seed, cfg_id, t):
    return np.random.default_rng(np.random.SeedSequence([seed, cfg_id], spawn_key=(t,)))


def _dirichlet(rng, alpha, k):
    w = rng.gamma(alpha, 1.0, size=k)
    return w / w.sum()


def _normalise_rows(v):
    return v / np.linalg.norm(v, axis=-1, keepdims=True)


# ---------------------------------------------------------------- lane recipes
def _lane_toy(rng, n, m, d):
    """Gaussian clouds, target shifted by a per-lane offset ~ U(0,1)^d."""
    x = rng.standard_normal((n, d))
    off = rng.uniform(0.0, 1.0, size=d)
    y = rng.standard_normal((m, d)) + off
    eps = float(np.exp(rng.uniform(np.log(0.02), np.log(0.2))))
    return x, y, np.full(n, 1.0 / n), np.full(m, 1.0 / m), eps


def _mixture(rng, k, d, count):
    mu = rng.normal(0.0, 2.0, size=(4, d))          # means ~ N(0, 4 I)
    comp = rng.integers(0, 4, size=count)           # equal weights
    return mu[comp] + 0.5 * rng.standard_normal((count, d))


def _lane_mixture(rng, n, m, d):
    """Separate 4-component Gaussian mixtures for source and target;
    Dirichlet(1) marginals renormalised in float64."""
    x = _mixture(rng, 4, d, n)
    y = _mixture(rng, 4, d, m)
    a = _dirichlet(rng, 1.0, n)
    b = _dirichlet(rng, 1.0, m)
    return x, y, a, b, 0.05


def _lane_telemetry(rng, n, m, d, gap=512, burn=200):
    """d AR(1) channels with a per-lane phi ~ U(0.5, 0.99) and unit stationary
    variance; the source window is n consecutive steps, the target window is
    m steps after a gap, shifted by a drift of length U(0.5, 2) along a random
    unit direction."""
    phi = rng.uniform(0.5, 0.99)
    T = burn + n + gap + m
    z = rng.standard_normal((T, d)) * np.sqrt(1.0 - phi * phi)
    s = np.empty((T, d))
    s[0] = rng.standard_normal(d)
    for k in range(1, T):
        s[k] = phi * s[k - 1] + z[k]
    x = s[burn:burn + n]
    y = s[burn + n + gap:burn + n + gap + m].copy()
    u = _normalise_rows(rng.standard_normal(d))
    y += rng.uniform(0.5, 2.0) * u
    return x, y, np.full(n, 1.0 / n), np.full(m, 1.0 / m), 0.01


def _lane_features(rng, n, m, d, classes=10, mean_cos=0.7):
    """Unit-norm features clustered around 10 unit class means with
    E cos(x, mean) ~ 0.7; source and target drawn independently."""
    means = _normalise_rows(rng.standard_normal((classes, d)))
    sigma = np.sqrt((mean_cos ** -2 - 1.0) / d)
    def draw(cnt):
        lab = rng.integers(0, classes, size=cnt)
        return _normalise_rows(means[lab] + sigma * rng.standard_normal((cnt, d)))
    return draw(n), draw(m), np.full(n, 1.0 / n), np.full(m, 1.0 / m), 0.05


def _lane_lidar(rng, n, m, d):
    """Uniform cube [-1,1]^3 against a noisy unit sphere (std 0.02);
    Dirichlet(0.5) marginals; eps ~ logU(0.005, 0.1)."""
    x = rng.uniform(-1.0, 1.0, size=(n, d))
    y = _normalise_rows(rng.standard_normal((m, d))) + 0.02 * rng.standard_normal((m, d))
    a = _dirichlet(rng, 0.5, n)
    b = _dirichlet(rng, 0.5, m)
    eps = float(np.exp(rng.uniform(np.log(0.005), np.log(0.1))))
    return x, y, a, b, eps


# ------------------------------------------------------------------- configs
#: name -> (cfg id, lane recipe, W, n, m, d, tol, max_iter, heterogeneous sizes)
CONFIGS = {
    "c1": dict(cid=1, recipe=_lane_toy, W=8, n=64, m=64, d=2, tol=1e-3, max_iter=5000),
    "c2": dict(cid=2, recipe=_lane_mixture, W=64, n=1024, m=1024, d=8, tol=1e-3, max_iter=5000),
    "c3": dict(cid=3, recipe=_lane_telemetry, W=256, n=512, m=512, d=16, tol=1e-3, max_iter=5000),
    "c4": dict(cid=4, recipe=_lane_features, W=32, n=4096, m=4096, d=512, tol=1e-3, max_iter=5000),
    "c5": dict(cid=5, recipe=_lane_lidar, W=1024, n=8192, m=8192, d=3, tol=1e-3, max_iter=5000,
               hetero=(256, 8192)),
}

DESCRIPTIONS = {
    "c1": "toy: W=8, n=m=64, d=2, Gaussian clouds with per-lane offset, uniform marginals, "
          "eps~logU(0.02,0.2)",
    "c2": "Packer19-shaped: W=64, n=m=1024, d=8, 4-component mixtures, Dirichlet(1) marginals, "
          "eps=0.05",
    "c3": "MetroPT-shaped telemetry: W=256, n=m=512, d=16, AR(1) windows with drift, uniform "
          "marginals, eps=0.01",
    "c4": "ImageNet-32-feature-shaped: W=32, n=m=4096, d=512, unit features around 10 class "
          "means, uniform marginals, eps=0.05",
    "c5": "A2D2-LiDAR-shaped heterogeneous: W=1024, n,m~U{256..8192} padded to 8192, d=3, cube vs "
          "noisy sphere, Dirichlet(0.5) marginals, eps~logU(0.005,0.1)",
}


def make(name, *, W=None, n=None, m=None, lanes=None, pad_value=0.0, seed=SEED,
         hetero=None) -> Workload:
    """Build a workload. ``W``/``lanes`` select lanes (lane t always gets the
    same data); ``n``/``m`` override the per-lane point counts (reduced-size
    parity cases follow the same recipe); ``hetero=(lo, hi)`` draws each lane's
    n_t, m_t ~ U{lo..hi} (c5 does this by default) and pads to ``n``/``m``;
    ``pad_value`` fills the padded tail (0 for benchmarks, NaN in tests so a
    leak is visible)."""
    cfg = CONFIGS[name]
    lanes = list(range(cfg["W"] if W is None else W)) if lanes is None else list(lanes)
    n_max = cfg["n"] if n is None else n
    m_max = cfg["m"] if m is None else m
    d = cfg["d"]
    hetero = cfg.get("hetero") if hetero is None else hetero
    if hetero is not None and hetero is not False:
        lo, hi = hetero
        hi_n, hi_m = min(hi, n_max), min(hi, m_max)
    Wl = len(lanes)
    X = np.full((Wl, n_max, d), pad_value, dtype=np.float32)
    Y = np.full((Wl, m_max, d), pad_value, dtype=np.float32)
    A = np.full((Wl, n_max), pad_value, dtype=np.float32)
    B = np.full((Wl, m_max), pad_value, dtype=np.float32)
    E = np.zeros(Wl, dtype=np.float32)
    N = np.zeros(Wl, dtype=np.int32)
    M = np.zeros(Wl, dtype=np.int32)
    for q, t in enumerate(lanes):
        rng = _rng(seed, cfg["cid"], t)
        if hetero is not None and hetero is not False:
            nt = int(rng.integers(min(lo, hi_n), hi_n + 1))
            mt = int(rng.integers(min(lo, hi_m), hi_m + 1))
        else:
            nt, mt = n_max, m_max
        x, y, a, b, eps = cfg["recipe"](rng, nt, mt, d)
        X[q, :nt] = x
        Y[q, :mt] = y
        A[q, :nt] = a
        B[q, :mt] = b
        E[q] = eps
        N[q], M[q] = nt, mt
    return Workload(name=name, X=X, Y=Y, a=A, b=B, eps=E, n=N, m=M, tol=cfg["tol"],
                    max_iter=cfg["max_iter"],
                    meta=dict(lanes=lanes, seed=seed, description=DESCRIPTIONS[name]))


# ------------------------------------------------------- randomised windows
def random_window(k, *, seed=SEED):
    """Randomised small window number ``k`` for parity sweeps: W in 1..12,
    padded sizes n_max, m_max in 1..320 with per-lane n_t, m_t in 1..n_max
    (m_max), d in 1..40, point clouds that are Gaussian or uniform at a random
    scale s (offsets ~ N(0, s^2 I)), Dirichlet(alpha) masses with alpha in
    {0.3, 1, 5}, and per-lane eps = 2 d s^2 logU(0.02, 0.2) (mean costs of 10
    to 100 eps). Also returns the run options drawn for the case: tol,
    audit_every, flags and sub-batch count. NaN-padded."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 900, k]))
    W = int(rng.integers(1, 13))
    n_max = int(rng.integers(1, 321))
    m_max = int(rng.integers(1, 321))
    d = int(rng.integers(1, 41))
    X = np.full((W, n_max, d), np.nan, dtype=np.float32)
    Y = np.full((W, m_max, d), np.nan, dtype=np.float32)
    A = np.full((W, n_max), np.nan, dtype=np.float32)
    B = np.full((W, m_max), np.nan, dtype=np.float32)
    E = np.zeros(W, dtype=np.float32)
    N = np.zeros(W, dtype=np.int32)
    M = np.zeros(W, dtype=np.int32)
    for t in range(W):
        nt, mt = int(rng.integers(1, n_max + 1)), int(rng.integers(1, m_max + 1))
        s = float(np.exp(rng.uniform(np.log(0.2), np.log(3.0))))
        def cloud(cnt):   # unit-variance shape at scale s, offset ~ N(0, s^2 I)
            if rng.random() < 0.5:
                return s * (rng.standard_normal((cnt, d)) + rng.standard_normal(d))
            return s * (rng.uniform(-1.7, 1.7, size=(cnt, d)) + rng.standard_normal(d))
        alpha = float(rng.choice([0.3, 1.0, 5.0]))
        X[t, :nt] = cloud(nt)
        Y[t, :mt] = cloud(mt)
        A[t, :nt] = _dirichlet(rng, alpha, nt)
        B[t, :mt] = _dirichlet(rng, alpha, mt)
        E[t] = 2.0 * d * s * s * float(np.exp(rng.uniform(np.log(0.02), np.log(0.2))))
        N[t], M[t] = nt, mt
    tol = float(rng.choice([1e-2, 1e-3]))
    audit_every = int(rng.integers(1, 4))
    # default, float32 matrix cores, float32 vector ALU, float64 (explicit),
    # materialised, guarded
    flags = int(rng.choice([0, 128, 4, 16, 32, 64]))
    if d > 32:
        flags = 0 if flags != 64 else 64               # d > 32 is always materialised
    if d > 16 and flags == 16:
        flags = 0                                      # the float64 state supports d <= 16
    streams = int(rng.choice([0, 1, 2])) if W >= 2 else 0
    w = Workload(name=f"random{k}", X=X, Y=Y, a=A, b=B, eps=E, n=N, m=M, tol=tol, max_iter=2000,
                 meta=dict(seed=seed, description="randomised small window"))
    return w, dict(tol=tol, audit_every=audit_every, flags=flags, streams=streams)
