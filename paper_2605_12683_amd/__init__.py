"""GTF-DEER hot path on AMD Instinct MI355X: Python binding of libdeer.

The functions below carry the names of the C entry points (include/deer.h) and take
torch tensors that already live on the GPU; they only marshal arguments, allocate the
outputs and the workspace with torch, and call the library on torch's current stream.

Model dictionaries use the paper's names:
  vanilla PLRNN  {"kind": "plrnn",   "A": [M], "W": [M,M], "h": [M]}
  shallow PLRNN  {"kind": "shplrnn", "A": [M], "W1": [M,L], "W2": [L,M], "h1": [M], "h2": [L]}
  diagonal SSM   {"kind": "diag_ssm", "lam": complex64 [M], "Bc": complex64 [M,K]}
  its read-out   {"Wa": [H,M], "ca": [H], "Wb": [No,H], "cb": [No]}
"""
from __future__ import annotations

import ctypes
import threading

import torch

from . import _binding as _b
from ._binding import DeerError, load  # noqa: F401

__all__ = ["deer_solve", "deer_adjoint", "deer_readout_loss", "plrnn_jacobian", "deer_scan", "deer_workspace_bytes",
           "deer_scan_workspace_bytes", "deer_readout_workspace_bytes", "deer_status_string", "DeerError", "load",
           "deer_sequential", "deer_sequential_workspace_bytes", "deer_solve_quasi", "deer_adjoint_quasi", "deer_train_step",
           "deer_host_reserve"]

_KINDS = {"plrnn": _b.DEER_PLRNN, "shplrnn": _b.DEER_SHPLRNN, "diag_ssm": _b.DEER_DIAG_SSM}
_INITS = {"teacher": _b.DEER_INIT_TEACHER, "zero": _b.DEER_INIT_ZERO, "user": _b.DEER_INIT_USER}


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t, dtype=torch.float32):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        t = torch.as_tensor(t)
    if t.is_complex():
        t = torch.view_as_real(t.to(torch.complex64).contiguous())
    t = t.to(device="cuda", dtype=dtype).contiguous()
    return t


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


_host = threading.local()


def deer_host_reserve(B: int) -> None:
    """Reserve the calling thread's pinned host block for solves of up to B sequences
    (deer_host_reserve in the C ABI; the solves themselves allocate nothing)."""
    if getattr(_host, "cap", 0) >= B:
        return
    _b._check(load().deer_host_reserve(int(B)), "deer_host_reserve")
    _host.cap = int(B)


class _Model:
    """Device copies of the parameters plus the C struct that points at them."""

    def __init__(self, model: dict):
        kind = model["kind"]
        self.kind = kind
        if kind == "plrnn":
            self.t = {k: _dev(model[k]) for k in ("A", "W")}
            self.t["h"] = _dev(model.get("h"))
            M = self.t["A"].shape[0]
            self.c = _b.deer_model(_b.DEER_PLRNN, M, 0, _ptr(self.t["A"]), _ptr(self.t["W"]), None,
                                   _ptr(self.t["h"]), None)
        elif kind == "shplrnn":
            self.t = {k: _dev(model[k]) for k in ("A", "W1", "W2")}
            self.t["h1"] = _dev(model.get("h1"))
            self.t["h2"] = _dev(model.get("h2"))
            M, L = self.t["W1"].shape
            self.c = _b.deer_model(_b.DEER_SHPLRNN, M, L, _ptr(self.t["A"]), _ptr(self.t["W1"]), _ptr(self.t["W2"]),
                                   _ptr(self.t["h1"]), _ptr(self.t["h2"]))
        elif kind == "diag_ssm":
            self.t = {"lam": _dev(model["lam"]), "Bc": _dev(model["Bc"])}
            M, K = self.t["Bc"].shape[:2]
            self.c = _b.deer_model(_b.DEER_DIAG_SSM, M, K, _ptr(self.t["lam"]), _ptr(self.t["Bc"]), None, None, None)
        else:
            raise ValueError(kind)
        self.M = self.c.M
        self.L = self.c.L


def _model(model):
    return model if isinstance(model, _Model) else _Model(model)


class _Readout:
    """Device copies of the read-out MLP parameters plus the C struct."""

    def __init__(self, params: dict):
        self.t = {k: _dev(params[k]) for k in ("Wa", "Wb")}
        self.t["ca"] = _dev(params.get("ca"))
        self.t["cb"] = _dev(params.get("cb"))
        self.H, self.M = self.t["Wa"].shape
        self.No = self.t["Wb"].shape[0]
        self.c = _b.deer_readout(self.H, self.No, _ptr(self.t["Wa"]), _ptr(self.t["ca"]), _ptr(self.t["Wb"]),
                                 _ptr(self.t["cb"]))


def _readout(r):
    return r if isinstance(r, _Readout) else _Readout(r)


def deer_readout_workspace_bytes(readout, B: int, T: int, M: int) -> int:
    r = _readout(readout)
    return int(load().deer_readout_workspace_bytes(ctypes.byref(r.c), B, T, M))


def deer_readout_loss(readout, h, x, *, want_grads: bool = True, want_masks: bool = False, want_loss: bool = True,
                      g=None, ws=None) -> dict:
    """Read-out MLP forward + backward at the complex states h [B,T,M][2]: returns
    dict(g = dL/dRe h [B,T,M], loss [1], masks, grads {Wa, ca, Wb, cb})."""
    lib = load()
    r = _readout(readout)
    h = _dev(h)
    x = _dev(x)
    B, T, M = h.shape[:3]
    out_g = torch.empty(B, T, M, device="cuda") if g is None else g
    loss = torch.empty(1, device="cuda") if want_loss else None
    masks = torch.empty(B, T, (r.H + 31) // 32, dtype=torch.int32, device="cuda") if want_masks else None
    grads = {}
    gs = None
    if want_grads:
        grads = {"Wa": torch.empty(r.H, M, device="cuda"), "ca": torch.empty(r.H, device="cuda"),
                 "Wb": torch.empty(r.No, r.H, device="cuda"), "cb": torch.empty(r.No, device="cuda")}
        gs = _b.deer_readout_grads(_ptr(grads["Wa"]), _ptr(grads["ca"]), _ptr(grads["Wb"]), _ptr(grads["cb"]))
    if ws is None:
        ws = _workspace(lib.deer_readout_workspace_bytes(ctypes.byref(r.c), B, T, M))
    st = lib.deer_readout_loss(ctypes.byref(r.c), B, T, M, _ptr(h), _ptr(x), _ptr(out_g), _ptr(loss), _ptr(masks),
                               ctypes.byref(gs) if gs is not None else None, _ptr(ws), ws.numel(), _stream())
    _b._check(st, "deer_readout_loss")
    return {"g": out_g, "loss": loss, "masks": masks, "grads": grads}


def deer_status_string(status: int) -> str:
    return load().deer_status_string(status).decode()


def deer_workspace_bytes(model, B: int, T: int, op: int) -> int:
    m = _model(model)
    return int(load().deer_workspace_bytes(ctypes.byref(m.c), B, T, op))


def deer_scan_workspace_bytes(layout: int, B: int, T: int, M: int, reverse: bool = False, transpose=None) -> int:
    tr = reverse if transpose is None else transpose
    return int(load().deer_scan_workspace_bytes(layout, int(bool(reverse)), int(bool(tr)), B, T, M))


def _workspace(nbytes: int):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


def deer_solve(model, x, alpha: float, n_forced: int, *, z0=None, tol: float = 1e-5, max_iter: int = 500,
               fixed_iters: int = 0, init: str = "teacher", z=None, want_masks: bool = False, ws=None,
               check: bool = True, step_bound: float = 0.0, T_w: int = 0, obs=None) -> dict:
    """GTF-DEER forward solve.  Returns dict(z, masks, iters, norms, status).  step_bound:
    threshold of the update safeguard (0: library default, < 0: only non-finite updates are
    rejected).  T_w: latent warm-up steps.  obs: observation matrix B [N, M] (N = n_forced) of
    the read-out x^ = B z, or None for the identity read-out of the first n_forced latents."""
    return _solve("deer_solve", 0, model, x, alpha, n_forced, z0=z0, tol=tol, max_iter=max_iter,
                  fixed_iters=fixed_iters, init=init, z=z, want_masks=want_masks, ws=ws, check=check,
                  step_bound=step_bound, T_w=T_w, obs=obs)


def deer_solve_quasi(model, x, alpha: float, n_forced: int, *, z0=None, tol: float = 1e-5, max_iter: int = 500,
                     fixed_iters: int = 0, init: str = "teacher", z=None, want_masks: bool = False, ws=None,
                     check: bool = True, step_bound: float = 0.0, T_w: int = 0) -> dict:
    """Quasi-DEER forward solve (diagonal Jacobians; PLRNN kinds): arguments and result as
    deer_solve."""
    return _solve("deer_solve_quasi", 1, model, x, alpha, n_forced, z0=z0, tol=tol, max_iter=max_iter,
                  fixed_iters=fixed_iters, init=init, z=z, want_masks=want_masks, ws=ws, check=check,
                  step_bound=step_bound, T_w=T_w)


def _solve(entry, quasi, model, x, alpha, n_forced, *, z0, tol, max_iter, fixed_iters, init, z, want_masks, ws,
           check, step_bound, T_w, obs=None):
    lib = load()
    m = _model(model)
    x = _dev(x)
    B, T1, _ = x.shape
    T = T1 - 1
    if m.kind == "diag_ssm":
        out = torch.empty(B, T, m.M, 2, device="cuda") if z is None else z
    else:
        out = torch.empty(B, T, m.M, device="cuda") if z is None else z
    if init == "user" and z is None:
        raise ValueError("init='user' needs z")
    masks = None
    if want_masks:
        H = m.M if m.kind == "plrnn" else m.L
        masks = torch.empty(B, T, (H + 31) // 32, dtype=torch.int32, device="cuda")
    obsd = _dev(obs)
    f = _b.deer_forcing(float(alpha), int(n_forced), int(T_w), _ptr(obsd))
    if ws is None:
        ws = _workspace(lib.deer_workspace_bytes_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, _b.DEER_OP_SOLVE, quasi))
    iters = (ctypes.c_int32 * B)()
    norms = (ctypes.c_float * B)()
    o = _b.deer_solve_opts(float(tol), int(max_iter), int(fixed_iters), _INITS[init], float(step_bound))
    if m.kind != "diag_ssm" and int(fixed_iters) <= 0:
        deer_host_reserve(B)
    z0d = _dev(z0)
    st = getattr(lib, entry)(ctypes.byref(m.c), ctypes.byref(f), ctypes.byref(o), B, T, _ptr(x), _ptr(z0d),
                             _ptr(out), _ptr(masks), iters, norms, _ptr(ws), ws.numel(), _stream())
    if check:
        _check_solve = (_b.DEER_OK, _b.DEER_ERR_NOT_CONVERGED, _b.DEER_ERR_NONFINITE)
        _b._check(st, entry, allow=_check_solve)
    return {"z": out, "masks": masks, "iters": list(iters), "norms": list(norms), "status": st}


def deer_adjoint(model, x, z, alpha: float, n_forced: int, *, z0=None, g=None, want_lam: bool = True,
                 want_grads: bool = True, ws=None, T_w: int = 0, obs=None) -> dict:
    """Adjoint scan lam = dL/dz and parameter gradients at trajectory z.  Diagonal SSM: g is
    complex [B,T,M] (or [B,T,M,2] float) = dL/dRe h + i dL/dIm h, or a real float tensor
    [B,T,M] = dL/dRe h (the read-out's cotangent).  obs: observation matrix B [N, M] as in
    deer_solve; the gradients then include "obs" = dL/dB."""
    lib = load()
    m = _model(model)
    x = _dev(x)
    B, T1, _ = x.shape
    T = T1 - 1
    z = _dev(z)
    g_layout = _b.DEER_G_NATIVE
    if m.kind == "diag_ssm" and g is not None:
        gt = g if isinstance(g, torch.Tensor) else torch.as_tensor(g)
        if not gt.is_complex() and gt.dim() == 3:
            g_layout = _b.DEER_G_REAL
    g = _dev(g)
    shape = (B, T, m.M, 2) if m.kind == "diag_ssm" else (B, T, m.M)
    lam = torch.empty(shape, device="cuda") if want_lam else None
    grads = {}
    gs = _b.deer_grads()
    if want_grads:
        if m.kind == "plrnn":
            grads = {"A": torch.empty(m.M, device="cuda"), "W": torch.empty(m.M, m.M, device="cuda"),
                     "h": torch.empty(m.M, device="cuda")}
            gs = _b.deer_grads(_ptr(grads["A"]), _ptr(grads["W"]), None, _ptr(grads["h"]), None)
        elif m.kind == "shplrnn":
            grads = {"A": torch.empty(m.M, device="cuda"), "W1": torch.empty(m.M, m.L, device="cuda"),
                     "W2": torch.empty(m.L, m.M, device="cuda"), "h1": torch.empty(m.M, device="cuda"),
                     "h2": torch.empty(m.L, device="cuda")}
            gs = _b.deer_grads(_ptr(grads["A"]), _ptr(grads["W1"]), _ptr(grads["W2"]), _ptr(grads["h1"]),
                               _ptr(grads["h2"]))
        else:
            grads = {"lam": torch.empty(m.M, 2, device="cuda"), "Bc": torch.empty(m.M, m.L, 2, device="cuda")}
            gs = _b.deer_grads(_ptr(grads["lam"]), _ptr(grads["Bc"]), None, None, None)
    obsd = _dev(obs)
    if want_grads and obsd is not None:
        grads["obs"] = torch.empty(obsd.shape, device="cuda")
        gs.obs = _ptr(grads["obs"])
    f = _b.deer_forcing(float(alpha), int(n_forced), int(T_w), _ptr(obsd))
    if ws is None:
        ws = _workspace(lib.deer_workspace_bytes_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, _b.DEER_OP_ADJOINT, 0))
    z0d = _dev(z0)
    st = lib.deer_adjoint_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, _ptr(x), _ptr(z0d), _ptr(z), _ptr(g),
                             g_layout, _ptr(lam), ctypes.byref(gs), _ptr(ws), ws.numel(), _stream())
    _b._check(st, "deer_adjoint")
    return {"lam": lam, "grads": grads}


def deer_adjoint_quasi(model, x, z, alpha: float, n_forced: int, *, z0=None, g=None, want_lam: bool = True,
                       want_grads: bool = True, ws=None, T_w: int = 0) -> dict:
    """Quasi-DEER adjoint (diagonal Jacobians; PLRNN kinds) and parameter gradients at
    trajectory z: arguments and result as deer_adjoint."""
    lib = load()
    m = _model(model)
    if m.kind not in ("plrnn", "shplrnn"):
        raise ValueError("quasi-DEER is built for the PLRNN kinds")
    x = _dev(x)
    B, T1, _ = x.shape
    T = T1 - 1
    z = _dev(z)
    g = _dev(g)
    lam = torch.empty((B, T, m.M), device="cuda") if want_lam else None
    grads, gs = _plrnn_grads(m) if want_grads else ({}, _b.deer_grads())
    f = _b.deer_forcing(float(alpha), int(n_forced), int(T_w))
    if ws is None:
        ws = _workspace(lib.deer_workspace_bytes_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, _b.DEER_OP_ADJOINT, 1))
    z0d = _dev(z0)
    st = lib.deer_adjoint_quasi(ctypes.byref(m.c), ctypes.byref(f), B, T, _ptr(x), _ptr(z0d), _ptr(z), _ptr(g),
                                _ptr(lam), ctypes.byref(gs), _ptr(ws), ws.numel(), _stream())
    _b._check(st, "deer_adjoint_quasi")
    return {"lam": lam, "grads": grads}


def deer_train_step(model, x, alpha: float, n_forced: int, *, step: int, state=None, lr: float = 1e-3,
                    beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8, mar_lambda: float = 0.0,
                    mar_units: int = 0, mar_p: int = 2, mar_gamma_w: float = 0.0, mar_gamma_v: float = 0.0,
                    quasi: bool = False, T_w: int = 0, tol: float = 1e-5, max_iter: int = 500, z0=None,
                    want_grads: bool = False, ws=None) -> dict:
    """One GTF-DEER training step (solve, MSE + MAR loss, gradient, Adam) through the C ABI.
    `model` must be a _Model (its device parameter tensors are updated in place); `state`
    holds the Adam moments {"m", "v"} (created as zeros when None).  Returns dict(loss, z,
    iters, grads, state, status)."""
    lib = load()
    if not isinstance(model, _Model):
        raise TypeError("deer_train_step updates the parameters in place: pass a _Model")
    m = model
    x = _dev(x)
    B, T1, _ = x.shape
    T = T1 - 1
    P = int(lib.deer_train_params(ctypes.byref(m.c)))
    if state is None:
        state = {"m": torch.zeros(P, device="cuda"), "v": torch.zeros(P, device="cuda")}
    f = _b.deer_forcing(float(alpha), int(n_forced), int(T_w))
    o = _b.deer_solve_opts(float(tol), int(max_iter), 0, _INITS["teacher"], 0.0)
    tr = _b.deer_train_opts(float(lr), float(beta1), float(beta2), float(eps), int(step), float(mar_lambda),
                            int(mar_units), int(mar_p), float(mar_gamma_w), float(mar_gamma_v), int(bool(quasi)))
    if ws is None:
        ws = _workspace(lib.deer_train_workspace_bytes(ctypes.byref(m.c), ctypes.byref(f), B, T, int(bool(quasi))))
    z = torch.empty(B, T, m.M, device="cuda")
    loss = torch.empty(1, device="cuda")
    iters = (ctypes.c_int32 * B)()
    grads, gs = _plrnn_grads(m) if want_grads else ({}, None)
    z0d = _dev(z0)
    deer_host_reserve(B)
    st = lib.deer_train_step(ctypes.byref(m.c), ctypes.byref(f), ctypes.byref(o), ctypes.byref(tr), B, T, _ptr(x),
                             _ptr(z0d), _ptr(z), _ptr(state["m"]), _ptr(state["v"]),
                             ctypes.byref(gs) if gs is not None else None, _ptr(loss), iters, _ptr(ws), ws.numel(),
                             _stream())
    _b._check(st, "deer_train_step")
    return {"loss": loss, "z": z, "iters": list(iters), "grads": grads, "state": state, "status": st}


def _plrnn_grads(m):
    """Gradient outputs of a PLRNN-kind model and the C struct pointing at them."""
    if m.kind == "plrnn":
        grads = {"A": torch.empty(m.M, device="cuda"), "W": torch.empty(m.M, m.M, device="cuda"),
                 "h": torch.empty(m.M, device="cuda")}
        return grads, _b.deer_grads(_ptr(grads["A"]), _ptr(grads["W"]), None, _ptr(grads["h"]), None)
    grads = {"A": torch.empty(m.M, device="cuda"), "W1": torch.empty(m.M, m.L, device="cuda"),
             "W2": torch.empty(m.L, m.M, device="cuda"), "h1": torch.empty(m.M, device="cuda"),
             "h2": torch.empty(m.L, device="cuda")}
    return grads, _b.deer_grads(_ptr(grads["A"]), _ptr(grads["W1"]), _ptr(grads["W2"]), _ptr(grads["h1"]),
                                _ptr(grads["h2"]))


def deer_sequential(model, x, alpha: float, n_forced: int, *, z0=None, g=None, want_lam: bool = True,
                    want_grads: bool = True, ws=None, z=None) -> dict:
    """Sequential GTF baseline: the rollout z and, if asked, back-propagation through time (lam
    and the parameter gradients), step by step in time.  Returns dict(z, lam, grads)."""
    lib = load()
    m = _model(model)
    x = _dev(x)
    B, T1, _ = x.shape
    T = T1 - 1
    out = torch.empty(B, T, m.M, device="cuda") if z is None else z
    lam = torch.empty(B, T, m.M, device="cuda") if want_lam else None
    grads, gs = _plrnn_grads(m) if want_grads else ({}, None)
    if ws is None:
        ws = _workspace(lib.deer_sequential_workspace_bytes(ctypes.byref(m.c), B, T))
    f = _b.deer_forcing(float(alpha), int(n_forced))
    z0d, gd = _dev(z0), _dev(g)
    st = lib.deer_sequential(ctypes.byref(m.c), ctypes.byref(f), B, T, _ptr(x), _ptr(z0d), _ptr(out), _ptr(gd),
                             _ptr(lam), ctypes.byref(gs) if gs is not None else None, _ptr(ws), ws.numel(), _stream())
    _b._check(st, "deer_sequential")
    return {"z": out, "lam": lam, "grads": grads}


def deer_sequential_workspace_bytes(model, B: int, T: int) -> int:
    return int(load().deer_sequential_workspace_bytes(ctypes.byref(_model(model).c), B, T))


def plrnn_jacobian(model, x, z, alpha: float, n_forced: int, *, z0=None, want=("F", "r", "masks"),
                   dense_J: bool = False, obs=None, T_w: int = 0) -> dict:
    """F, r, masks (and optionally the dense forced Jacobians) at trajectory z.  obs / T_w: an
    observation matrix B [N, M] and a warm-up (plrnn_jacobian_ex in the C ABI)."""
    lib = load()
    m = _model(model)
    x = _dev(x)
    z = _dev(z)
    B, T, M = z.shape
    H = m.M if m.kind == "plrnn" else m.L
    out = {}
    F = torch.empty(B, T, M, device="cuda") if "F" in want else None
    r = torch.empty(B, T, M, device="cuda") if "r" in want else None
    J = torch.empty(B, T, M, M, device="cuda") if dense_J else None
    masks = torch.empty(B, T, (H + 31) // 32, dtype=torch.int32, device="cuda") if "masks" in want else None
    obsd = _dev(obs)
    f = _b.deer_forcing(float(alpha), int(n_forced), int(T_w), _ptr(obsd))
    z0d = _dev(z0)
    if obsd is None and T_w == 0:
        st = lib.plrnn_jacobian(ctypes.byref(m.c), ctypes.byref(f), B, T, _ptr(x), _ptr(z0d), _ptr(z), _ptr(F),
                                _ptr(r), _ptr(J), _ptr(masks), _stream())
    else:
        ws = _workspace(lib.deer_workspace_bytes_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, _b.DEER_OP_JACOBIAN, 0))
        st = lib.plrnn_jacobian_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, _ptr(x), _ptr(z0d), _ptr(z), _ptr(F),
                                   _ptr(r), _ptr(J), _ptr(masks), _ptr(ws), ws.numel(), _stream())
    _b._check(st, "plrnn_jacobian")
    out.update({"F": F, "r": r, "J": J, "masks": masks})
    return out


def deer_scan(layout: int, J, b, reverse: bool = False, ws=None, transpose=None):
    """Bare affine scan (DEER_SCAN_DENSE: J [B,T,M,M]; DEER_SCAN_DIAG_C64: lambda [M] complex).
    transpose defaults to `reverse` (the adjoint's orientation)."""
    lib = load()
    J = _dev(J)
    b = _dev(b)
    B, T, M = b.shape[:3]
    tr = reverse if transpose is None else transpose
    y = torch.empty_like(b)
    if ws is None:
        ws = _workspace(lib.deer_scan_workspace_bytes(layout, int(bool(reverse)), int(bool(tr)), B, T, M))
    st = lib.deer_scan(layout, 1 if reverse else 0, 1 if tr else 0, B, T, M, _ptr(J), _ptr(b), _ptr(y), _ptr(ws),
                       ws.numel(), _stream())
    _b._check(st, "deer_scan")
    return y

def deer_scan_noalloc(layout: int, J, b, y, reverse: bool = False, transpose=None):
    """deer_scan without a workspace argument: the scratch is the library's static device array
    (deer_noalloc_scratch_bytes() bytes per GPU).  y is the caller's output buffer."""
    lib = load()
    J, b = _dev(J), _dev(b)
    B, T, M = b.shape[:3]
    tr = reverse if transpose is None else transpose
    st = lib.deer_scan_noalloc(layout, 1 if reverse else 0, 1 if tr else 0, B, T, M, _ptr(J), _ptr(b), _ptr(y),
                               _stream())
    _b._check(st, "deer_scan_noalloc")
    return y


def deer_noalloc_scratch_bytes() -> int:
    return int(load().deer_noalloc_scratch_bytes())

