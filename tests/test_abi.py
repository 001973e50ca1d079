"""C-ABI checks that need no GPU: the built library loads, exports every
function include/ds.h declares, and rejects bad arguments on the host before
any device work (no compute call is made here)."""

import ctypes
import os
import re

import pytest

import paper_2607_24741_amd as ds

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ds.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_\s\*]*?\b(ds_[a-z_]+)\s*\(",
                                 text, flags=re.M)))


def test_library_exports_every_declared_function():
    lib = ds.load_library()
    names = _declared_functions()
    assert set(names) == {"ds_api_version", "ds_workspace_bytes", "ds_solve", "ds_error_string",
                          "ds_last_error_message", "ds_solve_noalloc"}
    for nm in names:
        assert hasattr(lib, nm), nm
    assert lib.ds_api_version() == 4
    for code in range(6):
        assert lib.ds_error_string(code).decode()


def _problem(**kw):
    p = dict(W=4, n_max=100, m_max=90, d=3)
    p.update(kw)
    return ds._Problem(**p)


def _bytes(pr, op):
    lib = ds.load_library()
    out = ctypes.c_size_t(0)
    code = lib.ds_workspace_bytes(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(out))
    return code, out.value


def test_workspace_query_and_validation():
    op = ds._options(1e-3, None, 100, 1, "active", 0)
    code, n = _bytes(_problem(), op)
    assert code == 0 and n > 0 and n % 256 == 0
    code2, n2 = _bytes(_problem(W=8), op)
    assert code2 == 0 and n2 > n
    for bad in (dict(W=0), dict(n_max=0), dict(m_max=-1), dict(d=0), dict(d=513)):
        assert _bytes(_problem(**bad), op)[0] == 1, bad
    assert _bytes(_problem(W=5000), op)[0] == 4
    assert _bytes(_problem(W=4096), op)[0] == 0 and _bytes(_problem(W=4097), op)[0] == 4
    for tol, mi, ae, mode in ((0.0, 10, 1, 0), (1e-3, 0, 1, 0), (1e-3, 10, 0, 0), (1e-3, 10, 1, 7)):
        o = ds._Options(tol=tol, screen_tol=0.0, max_iter=mi, audit_every=ae, mode=mode, flags=0)
        assert _bytes(_problem(), o)[0] == 1
    o = ds._Options(tol=1e-3, screen_tol=0.0, max_iter=10, audit_every=1, mode=0, flags=4 | 8)
    assert _bytes(_problem(), o)[0] == 1
    assert ds.load_library().ds_last_error_message().decode()


def test_precise_state_default_validation_and_size():
    """The float64 state is the default for d <= 16 (DS_F_PRECISE states it
    explicitly, with the same workspace); DS_F_FAST32 selects the float32
    state, whose per-point state is half the size. DS_F_PRECISE excludes the
    float32 selectors and d > 16; above 16 the default is the float32 state."""
    op = ds._options(1e-3, None, 100, 1, "active", 0)
    opp = ds._options(1e-3, None, 100, 1, "active", ds.F_PRECISE)
    opf = ds._options(1e-3, None, 100, 1, "active", ds.F_FAST32)
    code, n_def = _bytes(_problem(W=4, d=8), op)
    code2, n64 = _bytes(_problem(W=4, d=8), opp)
    code3, n32 = _bytes(_problem(W=4, d=8), opf)
    assert code == code2 == code3 == 0
    assert n_def == n64 and n64 > 1.5 * n32
    for fl in (ds.F_FORCE_MFMA, ds.F_FORCE_VALU, ds.F_FAST32):
        bad = ds._options(1e-3, None, 100, 1, "active", ds.F_PRECISE | fl)
        assert _bytes(_problem(d=8), bad)[0] == 1
    assert _bytes(_problem(d=17), opp)[0] == 4
    code, n17 = _bytes(_problem(W=4, d=17), op)
    code2, n17f = _bytes(_problem(W=4, d=17), opf)
    assert code == code2 == 0 and n17 == n17f


def test_materialised_cost_validation_and_size():
    """d > 32 selects the materialised cost: the workspace holds W n_pad m_pad
    floats of cost; the float64 state and forced kernels are refused for it.
    More than 16384 points on a side (or DS_F_MATRIX_FREE) selects the
    matrix-free large-d half-step instead."""
    op = ds._options(1e-3, None, 100, 1, "active", 0)
    code, n512 = _bytes(_problem(W=2, n_max=256, m_max=200, d=512), op)
    assert code == 0 and n512 >= 2 * 256 * 256 * 4
    opm = ds._options(1e-3, None, 100, 1, "active", ds.F_MATERIALIZE)
    code, nm = _bytes(_problem(W=2, n_max=256, m_max=200, d=3), opm)
    assert code == 0 and nm >= 2 * 256 * 256 * 4
    for fl in (ds.F_PRECISE, ds.F_FAST32, ds.F_FORCE_VALU, ds.F_FORCE_MFMA):
        o = ds._options(1e-3, None, 100, 1, "active", fl)
        assert _bytes(_problem(d=64), o)[0] == 4
    # a side beyond 16384 points cannot be materialised: the matrix-free large-d
    # half-step takes it (no cost matrix in the workspace); forcing the
    # materialised cost there is refused, and the two flags are exclusive
    code, nfree = _bytes(_problem(W=2, n_max=17000, m_max=200, d=64), op)
    assert code == 0 and nfree < 2 * 17000 * 200 * 4
    assert _bytes(_problem(n_max=17000, d=64), opm)[0] == 4
    # up to 16384 a side is materialised (its column operand staged in 64 KB of LDS)
    code, n16k = _bytes(_problem(W=2, n_max=16384, m_max=200, d=64), op)
    assert code == 0 and n16k >= 2 * 16384 * 256 * 4
    opf = ds._options(1e-3, None, 100, 1, "active", ds.F_MATRIX_FREE)
    code, nf = _bytes(_problem(W=2, n_max=256, m_max=200, d=512), opf)
    # point records (2 banks x 2 sides x W x 256 padded points x 512 floats), no cost
    assert code == 0 and nf >= 2 * 2 * 2 * 256 * 512 * 4 and nf != n512
    both = ds._options(1e-3, None, 100, 1, "active", ds.F_MATRIX_FREE | ds.F_MATERIALIZE)
    assert _bytes(_problem(d=64), both)[0] == 1


def test_solve_rejects_bad_arguments_before_device_work():
    lib = ds.load_library()
    op = ds._options(1e-3, None, 100, 1, "active", 0)
    res = ds._Result()
    st = ds._Stats()
    # NULL problem / NULL inputs / NULL outputs / missing workspace: all host-side
    assert lib.ds_solve(None, ctypes.byref(op), ctypes.byref(res), None, 0, None, None) == 1
    pr = _problem()
    assert lib.ds_solve(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res), None, 0, None,
                        ctypes.byref(st)) == 1
    fake = ctypes.c_void_p(0x1000)
    pr = _problem(X=fake, Y=fake, a=fake, b=fake, eps=fake)
    assert lib.ds_solve(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res), None, 0, None,
                        None) == 1
    res = ds._Result(f=fake, g=fake, depth=fake, residual=fake, status=fake)
    assert lib.ds_solve(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res), None, 0, None,
                        None) == 2
    assert lib.ds_solve(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res),
                        ctypes.c_void_p(0x1001), 1 << 30, None, None) == 2
    assert lib.ds_solve(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res),
                        ctypes.c_void_p(0x1000), 16, None, None) == 2
    assert "workspace" in lib.ds_last_error_message().decode()


def test_sub_batch_validation_and_size():
    """streams is 0 (automatic) .. 4; more than one sub-batch needs the active
    mode; the workspace of a split window holds one part per sub-batch, each
    sized like a window of its own lanes."""
    lib = ds.load_library()
    for s in (-1, 5):
        assert _bytes(_problem(W=64), ds._options(1e-3, None, 100, 1, "active", 0, s))[0] == 1
    for mode in ("static", "logical"):
        assert _bytes(_problem(W=64), ds._options(1e-3, None, 100, 1, mode, 0, 2))[0] == 1
        assert _bytes(_problem(W=64), ds._options(1e-3, None, 100, 1, mode, 0, 1))[0] == 0
    _bytes(_problem(W=64), ds._options(1e-3, None, 100, 1, "static", 0, 2))
    assert "active mode" in lib.ds_last_error_message().decode()
    one = _bytes(_problem(W=64), ds._options(1e-3, None, 100, 1, "active", 0, 1))[1]
    parts = [_bytes(_problem(W=w), ds._options(1e-3, None, 100, 1, "active", 0, 1))[1]
             for w in (21, 21, 22)]
    three = _bytes(_problem(W=64), ds._options(1e-3, None, 100, 1, "active", 0, 3))[1]
    assert three == sum(parts) and three >= one
    # automatic: one below 32 lanes, two from 32 lanes on (active mode)
    def auto_is(pr, k):
        a = _bytes(pr, ds._options(1e-3, None, 100, 1, "active", 0, 0))[1]
        return a == _bytes(pr, ds._options(1e-3, None, 100, 1, "active", 0, k))[1]
    assert auto_is(_problem(W=16), 1)
    assert auto_is(_problem(W=40), 2)
    assert auto_is(_problem(W=64, n_max=1024, m_max=1024, d=8), 2)
    assert auto_is(_problem(W=256, n_max=512, m_max=512, d=16), 2)
    assert auto_is(_problem(W=1024, n_max=256, m_max=256, d=3), 2)


def test_guarded_release_validation_and_size():
    """DS_F_GUARD keeps two float64 partials per row block and lane, one row
    certificate per lane, and for the float64 verification its per-row sums of
    the eight column chunks (8 B per row and chunk), an arrival word and two
    list entries per row block (4 B each) and the two list lengths (one
    256-byte slice of the workspace); with the float64 state also the
    export-rounding sums of both sides per row block and lane (the outward
    bound), which a float32 state does not have. At most 16384 points per
    side."""
    op = ds._options(1e-3, None, 100, 1, "active", 0, 1)
    opg = ds._options(1e-3, None, 100, 1, "active", ds.F_GUARD, 1)
    code, n0 = _bytes(_problem(W=4, n_max=256, m_max=256, d=8), op)
    code2, n1 = _bytes(_problem(W=4, n_max=256, m_max=256, d=8), opg)
    assert code == 0 and code2 == 0 and n1 > n0
    W, rb = 512, 8192 // 128          # float64 state at d = 8: 128-row blocks
    big = _problem(W=W, n_max=8192, m_max=8192, d=8)
    c3, g64 = _bytes(big, opg)
    c4, p64 = _bytes(big, op)
    assert c3 == 0 and c4 == 0
    # agg64 (2 x 16 B) and the rounding sums (2 x 16 B) per row block, 16 B per
    # lane, per row block the chunk sums (8 chunks x 128 rows x 8 B), its word
    # and two list entries, and the list lengths
    assert g64 - p64 == W * rb * 64 + W * 16 + W * rb * (8 * 128 * 8 + 12) + 256
    f32 = ds._options(1e-3, None, 100, 1, "active", ds.F_GUARD | ds.F_FAST32, 1)
    f0 = ds._options(1e-3, None, 100, 1, "active", ds.F_FAST32, 1)
    rb32 = 8192 // 32                 # float32 matrix-core kernel: 32-row blocks
    assert (_bytes(big, f32)[1] - _bytes(big, f0)[1]
            == W * rb32 * 32 + W * 16 + W * rb32 * (8 * 32 * 8 + 12) + 256)
    assert _bytes(_problem(W=2, n_max=17000, m_max=100, d=3), opg)[0] == 4
    assert _bytes(_problem(W=2, n_max=17000, m_max=100, d=3), op)[0] == 0


def test_caller_outputs_are_validated():
    # the library writes through raw pointers: wrong dtype, shape or a missing
    # required output must be refused before the call
    import torch
    dev = torch.device("cpu")
    W, n_max, m_max = 3, 5, 4
    ok = dict(f=torch.empty((W, n_max)), g=torch.empty((W, m_max)),
              depth=torch.empty(W, dtype=torch.int32), residual=torch.empty(W),
              status=torch.empty(W, dtype=torch.int32))
    got = ds._check_out(ok, W, n_max, m_max, dev)
    assert got["order"] is None and got["row_residual"] is None and got["f"] is ok["f"]
    bad = [dict(ok, f=torch.empty((W, m_max))), dict(ok, depth=torch.empty(W)),
           dict(ok, g=torch.empty((m_max, W)).t()), dict(ok, extra=torch.empty(W)),
           {k: v for k, v in ok.items() if k != "status"}]
    for o in bad:
        with pytest.raises(ValueError):
            ds._check_out(o, W, n_max, m_max, dev)


def test_noalloc_entry_rejects_options_before_device_work():
    """ds_solve_noalloc runs one sub-batch and does not time launches: other
    options are refused on the host (no GPU needed to get here)."""
    lib = ds.load_library()
    fake = ctypes.c_void_p(0x1000)
    pr = _problem(X=fake, Y=fake, a=fake, b=fake, eps=fake)
    res = ds._Result(f=fake, g=fake, depth=fake, residual=fake, status=fake)
    for streams, flags in ((2, 0), (4, 0), (0, ds.F_TIMING)):
        op = ds._options(1e-3, None, 100, 1, "active", flags, streams)
        assert lib.ds_solve_noalloc(ctypes.byref(pr), ctypes.byref(op), ctypes.byref(res), None,
                                    None) == 1
        assert "ds_solve_noalloc" in lib.ds_last_error_message().decode()
    bad = ds._options(0.0, None, 100, 1, "active", 0)
    assert lib.ds_solve_noalloc(ctypes.byref(pr), ctypes.byref(bad), ctypes.byref(res), None,
                                None) == 1
