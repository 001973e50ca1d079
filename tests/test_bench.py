"""Host logic of bench.py (no GPU): the one-GPU refusal, the roofline
records of each path, the source-hash gate on the committed HBM traffic, and
the algorithmic bytes of the float64 update."""

import hashlib
import os
import subprocess
import sys
from types import SimpleNamespace

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr


def _window(d, n, m, W=2):
    return SimpleNamespace(d=d, W=W, n=np.full(W, n, np.int32), m=np.full(W, m, np.int32),
                           X=np.zeros((W, n, 1), np.float32), Y=np.zeros((W, m, 1), np.float32),
                           max_iter=5000)


def _args(**kw):
    base = dict(matrix_free=False, materialize=False, fast32=False, force_valu=False)
    base.update(kw)
    return SimpleNamespace(**base)


def _stats(tpairs, ms, launches, kept):
    return [SimpleNamespace(timed_pair_evals=tpairs, ms_update=ms, update_launches=launches,
                            pair_evals=kept)]


@pytest.mark.parametrize("d", [3, 8, 16])
def test_small_d_roofline_is_the_vector_unit_model(d):
    # 1e12 terms timed over 100 ms: (d + 4) lane operations each, as multiply-adds
    w = _window(d, 1024, 1024)
    rec = bench.roofline(w, _args(), _stats(1e12, 100.0, 50, 2e12), 0.5, "absent.md")
    assert rec["bound"] == "alu" and rec["unit"] == "TFLOP/s" and rec["peak"] == 78.6
    assert rec["achieved"] == pytest.approx(2 * (d + 4) * 1e12 / 0.1 / 1e12)
    assert rec["frac"] == pytest.approx(rec["achieved"] / 78.6)
    assert rec["avg_launch_us"] == pytest.approx(2000.0)
    assert rec["device_frac_lb"] == pytest.approx(2 * (d + 4) * 2e12 / 0.5 / 1e12 / 78.6)
    assert rec["traffic"] is None and "k_update_f64" in rec["kernel"]
    # the exponential's share of the model: 1 / R_e against (d + 4) / R_v
    assert rec["exp_bound_frac"] == pytest.approx((d + 4) ** -1 * (78.6e12 / 2) /
                                                  (256 * 4 * 8 * 2.4e9))
    fast = bench.roofline(w, _args(fast32=True), _stats(1e12, 100.0, 50, 2e12), 0.5, "absent.md")
    assert "k_update_mfma" in fast["kernel"]


def test_large_d_roofline_follows_the_kernel_the_library_picks():
    st = _stats(1e11, 100.0, 10, 1e11)
    mat = bench.roofline(_window(512, 4096, 4096), _args(), st, 1.0, "absent.md")
    assert mat["bound"] == "hbm" and mat["unit"] == "GB/s"
    assert mat["achieved"] == pytest.approx(4 * 1e11 / 0.1 / 1e9)
    free = bench.roofline(_window(512, 4096, 4096), _args(matrix_free=True), st, 1.0, "absent.md")
    assert free["bound"] == "mfma" and free["peak"] == 157.3
    assert free["achieved"] == pytest.approx(2 * 512 * 1e11 / 0.1 / 1e12)
    # beyond the points the materialised kernels stage, the matrix-free kernel runs
    big = bench.roofline(_window(64, 17000, 300), _args(), st, 1.0, "absent.md")
    assert big["bound"] == "mfma"
    forced = bench.roofline(_window(64, 300, 300), _args(materialize=True), st, 1.0, "absent.md")
    assert forced["bound"] == "hbm"


def test_traffic_is_reported_only_for_the_profiled_code(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2607_24741_amd" / "csrc"
    csrc.mkdir(parents=True)
    (tmp_path / "profiles").mkdir()
    code = {n: f"// {n}\nint f_{i}() {{ return {i}; }}  // trailing\n\n"
            for i, n in enumerate(bench.LIBRARY_SOURCES)}
    for name, text in code.items():
        (csrc / name).write_text(text)
    # the hash covers the code lines only: comments and blank lines are out
    h = hashlib.sha256()
    for i, n in enumerate(bench.LIBRARY_SOURCES):
        h.update(f"int f_{i}() {{ return {i}; }}".encode() + b"\n")
        h.update(b"\0")
    assert bench.source_code_hash(code[n] for n in bench.LIBRARY_SOURCES) == h.hexdigest()
    (tmp_path / "profiles" / "t.md").write_text(
        f"# summary\n\nkernel_code_sha256: {h.hexdigest()}\ntraffic_bytes_per_launch: 12345\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("t.md") == 12345.0
    assert bench.measured_traffic("missing.md") is None
    # a comment edit keeps the profile valid, a code edit does not
    (csrc / "ds_host.cpp").write_text("// another comment\n" + code["ds_host.cpp"])
    assert bench.measured_traffic("t.md") == 12345.0
    (csrc / "ds_host.cpp").write_text("int f_1() { return 7; }\n")
    assert bench.measured_traffic("t.md") is None


def test_committed_traffic_profile_matches_the_library_code():
    # the committed summary of the headline kernel's HBM traffic belongs to
    # the code in the tree (a code change needs the counters taken again)
    assert bench.measured_traffic("k_update_f64_c5_traffic.md") is not None


def test_algorithmic_bytes_of_the_float64_update():
    import torch
    w = _window(3, 100, 60)
    depth = torch.tensor([10, 4], dtype=torch.int32)
    last = (None, None, depth)
    st = SimpleNamespace(l_max=10)
    rec = bench.algorithmic_bytes(w, last, True, st)
    dp = 4                                    # d = 3 rounded up to even
    per_cycle = (100 + 60) * (16 * dp + 40)   # both half-steps of one lane-cycle
    assert rec["hbm_bytes_per_launch_algorithmic"] == pytest.approx(per_cycle * 14 / 20)
    assert bench.algorithmic_bytes(w, last, False, st) == {}
