"""The C ABI without a GPU: libdeer.so loads, exports every function include/deer.h declares,
and its host-side logic (workspace sizes, argument validation, status strings) answers
before any device work is queued."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "deer.h")

_b = pytest.importorskip("paper_2605_12683_amd._binding")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    names = re.findall(r"^\s*(?:const\s+)?(?:int|size_t|char|void|float)\s*\*?\s*(\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_b.LIB_PATH):
        pytest.skip("libdeer.so is not built (run __graft_entry__.build())")
    return _b.load()


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("deer_solve", "deer_adjoint", "plrnn_jacobian", "deer_scan", "deer_solve_quasi", "deer_adjoint_quasi",
              "deer_workspace_bytes", "deer_status_string", "deer_last_error"):
        assert n in names, n


def test_every_declared_function_is_exported(lib):
    raw = ctypes.CDLL(_b.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(raw, n)]
    assert not missing, missing
    # the binding declares a signature for every one of them
    assert set(_b.EXPORTED) <= set(_declared())


def _vanilla_model(M=16, kind=_b.DEER_PLRNN):
    buf = (ctypes.c_float * (M * M))()
    p = ctypes.cast(buf, ctypes.c_void_p)
    return _b.deer_model(kind, M, 8 if kind == _b.DEER_SHPLRNN else 0, p, p, p if kind == _b.DEER_SHPLRNN else None,
                         None, None), buf


def test_workspace_queries(lib):
    m, _keep = _vanilla_model(16)
    for op in (_b.DEER_OP_SOLVE, _b.DEER_OP_ADJOINT):
        assert lib.deer_workspace_bytes(ctypes.byref(m), 16, 16384, op) > 0
        assert lib.deer_quasi_workspace_bytes(ctypes.byref(m), 16, 16384, op) > 0
    assert lib.deer_workspace_bytes(ctypes.byref(m), 0, 16, _b.DEER_OP_SOLVE) == 0
    assert lib.deer_workspace_bytes(ctypes.byref(m), 4, 16, 7) == 0
    bad = _b.deer_model(_b.DEER_PLRNN, 65, 0, m.A, m.W, None, None, None)
    assert lib.deer_workspace_bytes(ctypes.byref(bad), 4, 16, _b.DEER_OP_SOLVE) == 0
    sh, _keep2 = _vanilla_model(4, _b.DEER_SHPLRNN)
    assert lib.deer_quasi_workspace_bytes(ctypes.byref(sh), 4, 16, _b.DEER_OP_SOLVE) > 0
    dg = _b.deer_model(_b.DEER_DIAG_SSM, 4, 3, m.A, m.W, None, None, None)
    assert lib.deer_quasi_workspace_bytes(ctypes.byref(dg), 4, 16, _b.DEER_OP_SOLVE) == 0   # PLRNN kinds only


def test_argument_errors_before_device_work(lib):
    m, _keep = _vanilla_model(4)
    o = _b.deer_solve_opts(1e-5, 10, 0, 0, 0.0)
    f = _b.deer_forcing(1.5, 2)                       # alpha outside [0, 1]
    for entry in ("deer_solve", "deer_solve_quasi"):
        st = getattr(lib, entry)(ctypes.byref(m), ctypes.byref(f), ctypes.byref(o), 2, 8, None, None, None, None,
                                 None, None, None, 0, None)
        assert st == _b.DEER_ERR_INVALID_ARG, entry
        assert b"alpha" in lib.deer_last_error()
    f = _b.deer_forcing(0.1, 2)
    gs = _b.deer_grads()
    st = lib.deer_adjoint_quasi(ctypes.byref(m), ctypes.byref(f), 2, 8, None, None, None, None, None,
                                ctypes.byref(gs), None, 0, None)
    assert st == _b.DEER_ERR_INVALID_ARG                # x and z are required
    dg = _b.deer_model(_b.DEER_DIAG_SSM, 4, 3, m.A, m.W, None, None, None)
    st = lib.deer_solve_quasi(ctypes.byref(dg), ctypes.byref(f), ctypes.byref(o), 2, 8, None, None, None, None,
                              None, None, None, 0, None)
    assert st == _b.DEER_ERR_INVALID_ARG and b"PLRNN" in lib.deer_last_error()


def test_status_strings(lib):
    for code in range(6):
        assert lib.deer_status_string(code)


def test_warmup_arguments(lib):
    m, _keep = _vanilla_model(4)
    o = _b.deer_solve_opts(1e-5, 10, 0, 0, 0.0)
    base = lib.deer_workspace_bytes(ctypes.byref(m), 2, 64, _b.DEER_OP_SOLVE)
    f0 = _b.deer_forcing(0.1, 2, 0)
    assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(f0), 2, 64, _b.DEER_OP_SOLVE, 0) == base
    fw = _b.deer_forcing(0.1, 2, 16)
    for op in (_b.DEER_OP_SOLVE, _b.DEER_OP_ADJOINT):
        for q in (0, 1):
            assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(fw), 2, 64, op, q) > 0
    bad = _b.deer_forcing(0.1, 2, 64)                  # T_w must be < T
    assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(bad), 2, 64, _b.DEER_OP_SOLVE, 0) == 0
    st = lib.deer_solve(ctypes.byref(m), ctypes.byref(bad), ctypes.byref(o), 2, 64, None, None, None, None,
                        None, None, None, 0, None)
    assert st == _b.DEER_ERR_INVALID_ARG and b"T_w" in lib.deer_last_error()
    # the warm-up is part of the one Newton iteration (GTF-DEER and quasi-DEER, both PLRNN kinds),
    # which needs no more workspace than the plain solve
    m20, _keep20 = _vanilla_model(20)
    ms, _keeps = _vanilla_model(16, _b.DEER_SHPLRNN)
    for mm in (m, m20, ms):
        for op in (_b.DEER_OP_SOLVE, _b.DEER_OP_ADJOINT):
            assert lib.deer_workspace_bytes_ex(ctypes.byref(mm), ctypes.byref(fw), 2, 64, op, 0) == \
                lib.deer_workspace_bytes(ctypes.byref(mm), 2, 64, op)
            assert lib.deer_workspace_bytes_ex(ctypes.byref(mm), ctypes.byref(fw), 2, 64, op, 1) == \
                lib.deer_quasi_workspace_bytes(ctypes.byref(mm), 2, 64, op)
    dg = _b.deer_model(_b.DEER_DIAG_SSM, 4, 3, m.A, m.W, None, None, None)
    assert lib.deer_workspace_bytes_ex(ctypes.byref(dg), ctypes.byref(fw), 2, 64, _b.DEER_OP_SOLVE, 0) == 0


def test_scan_workspace_query_every_orientation(lib):
    for rev in (0, 1):
        for tr in (0, 1):
            assert lib.deer_scan_workspace_bytes(_b.DEER_SCAN_DENSE, rev, tr, 2, 1000, 32) > 0
            assert lib.deer_scan_workspace_bytes(_b.DEER_SCAN_DIAG_C64, rev, tr, 2, 1000, 64) > 0
    assert lib.deer_scan_workspace_bytes(_b.DEER_SCAN_DENSE, 0, 0, 2, 1000, 128) > 0
    assert lib.deer_scan_workspace_bytes(_b.DEER_SCAN_DENSE, 0, 0, 2, 1000, 129) == 0
    assert lib.deer_scan_workspace_bytes(_b.DEER_SCAN_DENSE, 0, 0, 0, 1000, 16) == 0
    dummy = (ctypes.c_float * 4)()
    p = ctypes.cast(dummy, ctypes.c_void_p)
    st = lib.deer_scan(_b.DEER_SCAN_DENSE, 0, 1, 2, 10, 129, p, p, p, None, 0, None)
    assert st == _b.DEER_ERR_INVALID_ARG
    st = lib.deer_scan(_b.DEER_SCAN_DENSE, 0, 1, 2, 10, 4, p, p, p, None, 0, None)   # y aliases b
    assert st == _b.DEER_ERR_INVALID_ARG and b"alias" in lib.deer_last_error()


def test_solve_with_tolerance_needs_the_threads_host_block(lib):
    """A solve with a tolerance on a thread that has not reserved its pinned host block is
    refused before any device work (the solve itself allocates nothing)."""
    import threading
    m, _keep = _vanilla_model(4)
    dummy = (ctypes.c_float * 64)()
    p = ctypes.cast(dummy, ctypes.c_void_p)
    out = {}

    def run():
        f = _b.deer_forcing(0.1, 2, 0)
        o = _b.deer_solve_opts(1e-5, 10, 0, 0, 0.0)
        out["st"] = lib.deer_solve(ctypes.byref(m), ctypes.byref(f), ctypes.byref(o), 2, 8, p, None, p, None,
                                   None, None, p, 64, None)
        out["msg"] = lib.deer_last_error()
        out["q"] = lib.deer_solve_quasi(ctypes.byref(m), ctypes.byref(f), ctypes.byref(o), 2, 8, p, None, p, None,
                                        None, None, p, 64, None)
        out["bad"] = lib.deer_host_reserve(0)
        out["rel"] = lib.deer_host_release()
    t = threading.Thread(target=run)
    t.start()
    t.join()
    assert out["st"] == _b.DEER_ERR_INVALID_ARG and b"deer_host_reserve" in out["msg"]
    assert out["q"] == _b.DEER_ERR_INVALID_ARG
    assert out["bad"] == _b.DEER_ERR_INVALID_ARG
    assert out["rel"] == _b.DEER_OK                 # nothing to free


def test_observation_matrix_arguments(lib):
    """A general observation matrix B: workspace queries for the solve, the adjoint and the
    Jacobian entry point; n_forced (B's row count) in [1, 64], may exceed M; the entry points
    that take the identity read-out only refuse it before any device work."""
    m, _keep = _vanilla_model(8)
    obs = (ctypes.c_float * 64)()
    po = ctypes.cast(obs, ctypes.c_void_p)
    f = _b.deer_forcing(0.1, 3, 0, po)
    for op in (_b.DEER_OP_SOLVE, _b.DEER_OP_ADJOINT, _b.DEER_OP_JACOBIAN):
        assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(f), 2, 64, op, 0) > 0
    assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(f), 2, 64, _b.DEER_OP_SOLVE, 1) == 0  # quasi
    tall = _b.deer_forcing(0.1, 12, 0, po)                 # N = 12 > M = 8
    assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(tall), 2, 64, _b.DEER_OP_SOLVE, 0) > 0
    for bad_n in (0, 65):
        bad = _b.deer_forcing(0.1, bad_n, 0, po)
        assert lib.deer_workspace_bytes_ex(ctypes.byref(m), ctypes.byref(bad), 2, 64, _b.DEER_OP_SOLVE, 0) == 0
    dummy = (ctypes.c_float * 64)()
    p = ctypes.cast(dummy, ctypes.c_void_p)
    o = _b.deer_solve_opts(1e-5, 10, 2, 0, 0.0)
    st = lib.deer_solve_quasi(ctypes.byref(m), ctypes.byref(f), ctypes.byref(o), 2, 8, p, None, p, None, None, None,
                              p, 64, None)
    assert st == _b.DEER_ERR_INVALID_ARG and b"observation" in lib.deer_last_error()
    st = lib.plrnn_jacobian(ctypes.byref(m), ctypes.byref(f), 2, 8, p, None, p, p, None, None, None, None)
    assert st == _b.DEER_ERR_INVALID_ARG and b"observation" in lib.deer_last_error()
    gs = _b.deer_grads()
    st = lib.deer_sequential(ctypes.byref(m), ctypes.byref(f), 2, 8, p, None, p, None, None, ctypes.byref(gs), p, 64,
                             None)
    assert st == _b.DEER_ERR_INVALID_ARG
    dg = _b.deer_model(_b.DEER_DIAG_SSM, 4, 3, m.A, m.W, None, None, None)
    assert lib.deer_workspace_bytes_ex(ctypes.byref(dg), ctypes.byref(f), 2, 64, _b.DEER_OP_SOLVE, 0) == 0
