"""ctypes binding of libdeer (the C ABI in include/deer.h).

Argument marshalling only: every step of the GTF-DEER path runs in the HIP kernels of
libdeer.so.  PyTorch provides device memory and the stream.  There is no fallback: if the
library is missing, loading fails with an error.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdeer.so")

DEER_OK, DEER_ERR_INVALID_ARG, DEER_ERR_NOT_CONVERGED, DEER_ERR_NONFINITE, DEER_ERR_HIP, DEER_ERR_WORKSPACE = range(6)
DEER_PLRNN, DEER_SHPLRNN, DEER_DIAG_SSM = 0, 1, 2
DEER_INIT_TEACHER, DEER_INIT_ZERO, DEER_INIT_USER = 0, 1, 2
DEER_OP_SOLVE, DEER_OP_ADJOINT, DEER_OP_JACOBIAN = 0, 1, 2
DEER_SCAN_DENSE, DEER_SCAN_DIAG_C64 = 0, 1
DEER_G_NATIVE, DEER_G_REAL = 0, 1

EXPORTED = ["deer_workspace_bytes", "deer_solve", "deer_adjoint", "deer_adjoint_ex", "plrnn_jacobian", "deer_scan",
            "deer_scan_workspace_bytes", "deer_readout_workspace_bytes", "deer_readout_loss", "deer_status_string",
            "deer_last_error", "deer_timing_enable", "deer_timing_report", "deer_solve_quasi", "deer_adjoint_quasi",
            "deer_quasi_workspace_bytes", "deer_sequential", "deer_sequential_workspace_bytes",
            "deer_workspace_bytes_ex", "deer_train_step", "deer_train_workspace_bytes", "deer_train_params",
            "deer_host_reserve", "deer_host_release", "deer_scan_noalloc", "deer_noalloc_scratch_bytes",
            "plrnn_jacobian_ex"]

_fp = ctypes.c_void_p


class deer_model(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("M", ctypes.c_int), ("L", ctypes.c_int),
                ("A", _fp), ("W", _fp), ("W2", _fp), ("h", _fp), ("h2", _fp)]


class deer_train_opts(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
                ("step", ctypes.c_int), ("mar_lambda", ctypes.c_float), ("mar_units", ctypes.c_int),
                ("mar_p", ctypes.c_int), ("mar_gamma_w", ctypes.c_float), ("mar_gamma_v", ctypes.c_float),
                ("quasi", ctypes.c_int)]


class deer_forcing(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("n_forced", ctypes.c_int), ("T_w", ctypes.c_int), ("obs", _fp)]


class deer_solve_opts(ctypes.Structure):
    _fields_ = [("tol", ctypes.c_float), ("max_iter", ctypes.c_int), ("fixed_iters", ctypes.c_int),
                ("init", ctypes.c_int), ("step_bound", ctypes.c_float)]


class deer_grads(ctypes.Structure):
    _fields_ = [("A", _fp), ("W", _fp), ("W2", _fp), ("h", _fp), ("h2", _fp), ("obs", _fp)]


class deer_readout(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int), ("n_out", ctypes.c_int), ("Wa", _fp), ("ca", _fp), ("Wb", _fp), ("cb", _fp)]


class deer_readout_grads(ctypes.Structure):
    _fields_ = [("Wa", _fp), ("ca", _fp), ("Wb", _fp), ("cb", _fp)]


_lib = None


def load(path: str = LIB_PATH):
    """Load libdeer.so and declare its signatures (raises if the library is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2605_12683_amd.build` "
                           "(there is no non-HIP fallback)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    sz, i32, vp = ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p
    lib.deer_workspace_bytes.argtypes = [P(deer_model), i32, i32, i32]
    lib.deer_workspace_bytes.restype = sz
    lib.deer_scan_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32]
    lib.deer_scan_workspace_bytes.restype = sz
    lib.deer_solve.argtypes = [P(deer_model), P(deer_forcing), P(deer_solve_opts), i32, i32, vp, vp, vp, vp,
                               P(ctypes.c_int32), P(ctypes.c_float), vp, sz, vp]
    lib.deer_solve.restype = i32
    lib.deer_adjoint.argtypes = [P(deer_model), P(deer_forcing), i32, i32, vp, vp, vp, vp, vp, P(deer_grads), vp, sz,
                                 vp]
    lib.deer_adjoint.restype = i32
    lib.deer_solve_quasi.argtypes = lib.deer_solve.argtypes
    lib.deer_solve_quasi.restype = i32
    lib.deer_adjoint_quasi.argtypes = lib.deer_adjoint.argtypes
    lib.deer_adjoint_quasi.restype = i32
    lib.deer_train_step.argtypes = [P(deer_model), P(deer_forcing), P(deer_solve_opts), P(deer_train_opts), i32, i32,
                                    vp, vp, vp, vp, vp, P(deer_grads), vp, P(ctypes.c_int32), vp, sz, vp]
    lib.deer_train_step.restype = i32
    lib.deer_train_workspace_bytes.argtypes = [P(deer_model), P(deer_forcing), i32, i32, i32]
    lib.deer_train_workspace_bytes.restype = sz
    lib.deer_train_params.argtypes = [P(deer_model)]
    lib.deer_train_params.restype = sz
    lib.deer_workspace_bytes_ex.argtypes = [P(deer_model), P(deer_forcing), i32, i32, i32, i32]
    lib.deer_workspace_bytes_ex.restype = sz
    lib.deer_quasi_workspace_bytes.argtypes = [P(deer_model), i32, i32, i32]
    lib.deer_quasi_workspace_bytes.restype = sz
    lib.deer_adjoint_ex.argtypes = [P(deer_model), P(deer_forcing), i32, i32, vp, vp, vp, vp, i32, vp, P(deer_grads),
                                    vp, sz, vp]
    lib.deer_adjoint_ex.restype = i32
    lib.deer_sequential.argtypes = [P(deer_model), P(deer_forcing), i32, i32, vp, vp, vp, vp, vp, P(deer_grads), vp,
                                    sz, vp]
    lib.deer_sequential.restype = i32
    lib.deer_sequential_workspace_bytes.argtypes = [P(deer_model), i32, i32]
    lib.deer_sequential_workspace_bytes.restype = sz
    lib.deer_readout_workspace_bytes.argtypes = [P(deer_readout), i32, i32, i32]
    lib.deer_readout_workspace_bytes.restype = sz
    lib.deer_readout_loss.argtypes = [P(deer_readout), i32, i32, i32, vp, vp, vp, vp, vp, P(deer_readout_grads), vp,
                                      sz, vp]
    lib.deer_readout_loss.restype = i32
    lib.plrnn_jacobian.argtypes = [P(deer_model), P(deer_forcing), i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.plrnn_jacobian.restype = i32
    lib.plrnn_jacobian_ex.argtypes = [P(deer_model), P(deer_forcing), i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.plrnn_jacobian_ex.restype = i32
    lib.deer_scan.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, sz, vp]
    lib.deer_scan.restype = i32
    lib.deer_scan_noalloc.argtypes = [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp]
    lib.deer_scan_noalloc.restype = i32
    lib.deer_noalloc_scratch_bytes.argtypes = []
    lib.deer_noalloc_scratch_bytes.restype = sz
    lib.deer_host_reserve.argtypes = [i32]
    lib.deer_host_reserve.restype = i32
    lib.deer_host_release.argtypes = []
    lib.deer_host_release.restype = i32
    lib.deer_status_string.argtypes = [i32]
    lib.deer_status_string.restype = ctypes.c_char_p
    lib.deer_last_error.argtypes = []
    lib.deer_last_error.restype = ctypes.c_char_p
    lib.deer_timing_enable.argtypes = [i32]
    lib.deer_timing_enable.restype = i32
    lib.deer_timing_report.argtypes = [i32, ctypes.c_char_p, i32, P(ctypes.c_double), P(ctypes.c_long)]
    lib.deer_timing_report.restype = i32
    _lib = lib
    return lib


def timing_enable(on: bool):
    load().deer_timing_enable(1 if on else 0)


def timing_report() -> dict:
    """{kernel name: (total ms, launches)} of the launches recorded since timing_enable(True)."""
    lib = load()
    n = lib.deer_timing_report(-1, None, 0, None, None)
    if n < 0:
        raise RuntimeError("deer_timing_report failed")
    out = {}
    for i in range(n):
        buf = ctypes.create_string_buffer(128)
        ms = ctypes.c_double()
        cnt = ctypes.c_long()
        lib.deer_timing_report(i, buf, 128, ctypes.byref(ms), ctypes.byref(cnt))
        out[buf.value.decode()] = (ms.value, cnt.value)
    return out


class DeerError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        msg = lib.deer_last_error().decode() or lib.deer_status_string(status).decode()
        super().__init__(f"{where}: {lib.deer_status_string(status).decode()} ({msg})")
        self.status = status


def _check(status: int, where: str, allow=(DEER_OK,)):
    if status not in allow:
        raise DeerError(status, where)
    return status
