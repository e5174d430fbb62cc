"""Seeded synthetic inputs for the GTF-DEER hot path.

This module only *generates inputs*: model parameters drawn from the stated
distributions and standardised ODE trajectories that stand in for the paper's
datasets (Lorenz-63 and Lorenz-96, datasets appendix).  It holds none of the
method's arithmetic and is imported both by the CPU oracle's tests and by the
GPU path's tests and benchmark, so that both sides read the very same fp32
arrays.

The five named workloads (``CONFIGS``) follow the benchmark configurations of
this project: vanilla PLRNN M=3/16/64, shallow PLRNN M=32 L=256 and a diagonal
complex SSM with N=64 states.  Every array is returned as float32 (C order).

Input recipe (shared by all trajectories):
  * initial condition ~ N(0, 1) per state variable (Lorenz-63: z offset +25),
  * classical fixed-step RK4 in float64, 1000-step transient discarded,
  * T+1 samples kept, each variable z-scored over the kept samples,
  * optional slow triangle-wave drift (amplitude 1, given period, random phase),
  * i.i.d. N(0, noise_std^2) observation noise, then cast to float32.
Seeds: parameters use ``default_rng(1000*i)``, sequence b of workload i uses
``default_rng(1000*i + 1 + b)``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_ODE_SRC = os.path.join(_HERE, "_ode.c")
_ODE_SO = os.path.join(_HERE, "_ode.so")
_ode_lib = None
_ode_lock = threading.Lock()

TRANSIENT = 1000


def build_ode_helper(force: bool = False) -> str:
    """Compile the RK4 helper with gcc (data generation only)."""
    if force or not os.path.exists(_ODE_SO) or os.path.getmtime(_ODE_SO) < os.path.getmtime(_ODE_SRC):
        tmp = _ODE_SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-o", tmp, _ODE_SRC])
        os.replace(tmp, _ODE_SO)
    return _ODE_SO


def _lib():
    global _ode_lib
    with _ode_lock:
        if _ode_lib is None:
            try:
                path = build_ode_helper()
            except (OSError, subprocess.CalledProcessError):
                path = _ODE_SO if os.path.exists(_ODE_SO) else None
            if path is None:
                return None
            lib = ctypes.CDLL(path)
            dp = ctypes.POINTER(ctypes.c_double)
            lib.lorenz63_rk4.argtypes = [dp, ctypes.c_double, ctypes.c_long, ctypes.c_long,
                                         ctypes.c_double, ctypes.c_double, ctypes.c_double, dp]
            lib.lorenz96_rk4.argtypes = [dp, ctypes.c_long, ctypes.c_double, ctypes.c_long, ctypes.c_long,
                                         ctypes.c_double, dp, dp]
            _ode_lib = lib
        return _ode_lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _numpy_rk4(rhs, state, dt, n_transient, n_keep):
    out = np.empty((n_keep, state.size))
    s = state.copy()
    for step in range(n_transient + n_keep):
        if step >= n_transient:
            out[step - n_transient] = s
        k1 = rhs(s)
        k2 = rhs(s + 0.5 * dt * k1)
        k3 = rhs(s + 0.5 * dt * k2)
        k4 = rhs(s + dt * k3)
        s = s + dt / 6.0 * (k1 + 2.0 * k2 + 2.0 * k3 + k4)
    return out


def lorenz63(n_keep: int, rng: np.random.Generator, dt: float = 0.01,
             sigma: float = 10.0, rho: float = 28.0, beta: float = 8.0 / 3.0) -> np.ndarray:
    """Raw (unstandardised) Lorenz-63 trajectory, float64 [n_keep, 3]."""
    state = rng.standard_normal(3) + np.array([0.0, 0.0, 25.0])
    lib = _lib()
    if lib is None:
        def rhs(s):
            return np.array([sigma * (s[1] - s[0]), s[0] * (rho - s[2]) - s[1], s[0] * s[1] - beta * s[2]])
        return _numpy_rk4(rhs, state, dt, TRANSIENT, n_keep)
    state = np.ascontiguousarray(state, dtype=np.float64)
    out = np.empty((n_keep, 3))
    lib.lorenz63_rk4(_ptr(state), dt, TRANSIENT, n_keep, sigma, rho, beta, _ptr(out))
    return out


def lorenz96(n_keep: int, n: int, rng: np.random.Generator, dt: float = 0.01, forcing: float = 8.0) -> np.ndarray:
    """Raw Lorenz-96 trajectory (cyclic indices), float64 [n_keep, n]; n >= 4."""
    if n < 4:
        raise ValueError("Lorenz-96 needs at least 4 variables")
    state = np.ascontiguousarray(rng.standard_normal(n), dtype=np.float64)
    lib = _lib()
    if lib is None:
        def rhs(s):
            return (np.roll(s, -1) - np.roll(s, 2)) * np.roll(s, 1) - s + forcing
        return _numpy_rk4(rhs, state, dt, TRANSIENT, n_keep)
    out = np.empty((n_keep, n))
    work = np.empty(5 * n)
    lib.lorenz96_rk4(_ptr(state), n, dt, TRANSIENT, n_keep, forcing, _ptr(work), _ptr(out))
    return out


def triangle_wave(n: int, period: float, phase: float) -> np.ndarray:
    """Triangle wave with amplitude 1 (range [-1, 1]) sampled at n steps."""
    s = (np.arange(n) + phase) / period
    return 4.0 * np.abs(s - np.floor(s + 0.5)) - 1.0


def observed_sequence(system: str, n_obs: int, T: int, rng: np.random.Generator, *,
                      noise_std: float = 0.01, drift_period: float | None = None) -> np.ndarray:
    """One standardised, noisy trajectory of T+1 samples, float64 [T+1, n_obs]."""
    if system == "lorenz63":
        raw = lorenz63(T + 1, rng)
    elif system == "lorenz96":
        raw = lorenz96(T + 1, n_obs, rng)
    else:
        raise ValueError(system)
    sd = raw.std(axis=0)
    sd[sd == 0] = 1.0
    x = (raw - raw.mean(axis=0)) / sd
    if drift_period is not None:
        phase = rng.uniform(0.0, drift_period)
        x = x + triangle_wave(T + 1, drift_period, phase)[:, None]
    x = x + noise_std * rng.standard_normal(x.shape)
    return x[:, :n_obs]


def observed_batch(system: str, n_obs: int, B: int, T: int, seed_base: int, **kw) -> np.ndarray:
    """[B, T+1, n_obs] float32; sequence b drawn from default_rng(seed_base + b)."""
    out = np.empty((B, T + 1, n_obs), dtype=np.float32)

    def one(b):
        out[b] = observed_sequence(system, n_obs, T, np.random.default_rng(seed_base + b), **kw)

    if B * T < (1 << 16):
        for b in range(B):
            one(b)
    else:  # sequences are independent; the integrator and numpy release the GIL
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(max_workers=min(B, os.cpu_count() or 1, 16)) as ex:
            list(ex.map(one, range(B)))
    return out


# --------------------------------------------------------------------------------------
# model parameters
# --------------------------------------------------------------------------------------

def plrnn_params(M: int, rng: np.random.Generator, a_range=(0.5, 0.9), w_std=0.1, h_std=0.1) -> dict:
    """Vanilla PLRNN z' = diag(A) z + W relu(z) + h (full W, diagonal kept)."""
    A = rng.uniform(a_range[0], a_range[1], M)
    W = rng.normal(0.0, w_std, (M, M))
    h = rng.normal(0.0, h_std, M)
    return {"A": A.astype(np.float32), "W": W.astype(np.float32), "h": h.astype(np.float32)}


def shplrnn_params(M: int, L: int, rng: np.random.Generator, a_range=(0.5, 0.95), h_std=0.1) -> dict:
    """Shallow PLRNN z' = diag(A) z + W1 relu(W2 z + h2) + h1, W1, W2 ~ N(0, 1/L)."""
    A = rng.uniform(a_range[0], a_range[1], M)
    W1 = rng.normal(0.0, 1.0 / np.sqrt(L), (M, L))
    W2 = rng.normal(0.0, 1.0 / np.sqrt(L), (L, M))
    h1 = rng.normal(0.0, h_std, M)
    h2 = rng.normal(0.0, h_std, L)
    f = np.float32
    return {"A": A.astype(f), "W1": W1.astype(f), "W2": W2.astype(f), "h1": h1.astype(f), "h2": h2.astype(f)}


def diag_ssm_params(n_state: int, n_in: int, n_hidden: int, n_out: int, rng: np.random.Generator,
                    mag_range=(0.9, 0.999), phase_max=np.pi / 10) -> dict:
    """Diagonal complex SSM h' = lam * h + Bc u with MLP read-out Wb relu(Wa Re h + ca) + cb."""
    mag = rng.uniform(mag_range[0], mag_range[1], n_state)
    ph = rng.uniform(0.0, phase_max, n_state)
    lam = mag * np.exp(1j * ph)
    Bc = rng.normal(0.0, np.sqrt(1.0 / 6.0), (n_state, n_in)) + 1j * rng.normal(0.0, np.sqrt(1.0 / 6.0), (n_state, n_in))
    Wa = rng.normal(0.0, 1.0 / np.sqrt(n_state), (n_hidden, n_state))
    Wb = rng.normal(0.0, 1.0 / np.sqrt(n_hidden), (n_out, n_hidden))
    f = np.float32
    return {"lam": lam.astype(np.complex64), "Bc": Bc.astype(np.complex64),
            "Wa": Wa.astype(f), "ca": np.zeros(n_hidden, f), "Wb": Wb.astype(f), "cb": np.zeros(n_out, f)}


# --------------------------------------------------------------------------------------
# named workloads
# --------------------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    kind: str                 # "plrnn" | "shplrnn" | "diag_ssm"
    B: int
    T: int
    M: int                    # latent / state dimension
    n_obs: int                # observed (forced) latents N
    alpha: float
    params: dict
    x: np.ndarray             # [B, T+1, n_obs] float32
    L: int = 0                # hidden width (shallow PLRNN) / MLP hidden (diag SSM)
    tol: float = 1e-5
    max_iter: int = 500
    fixed_iters: int = 0
    meta: dict = field(default_factory=dict)


CONFIG_SPECS = {
    1: dict(name="plrnn_M3_T1024_B1", kind="plrnn", M=3, n_obs=3, B=1, T=1024, alpha=0.1, fixed_iters=5,
            system="lorenz63", params=dict(a_range=(0.5, 0.9), w_std=0.1, h_std=0.1)),
    2: dict(name="plrnn_M16_T16384_B16", kind="plrnn", M=16, n_obs=3, B=16, T=16384, alpha=0.2,
            system="lorenz63", params=dict(a_range=(0.5, 0.9), w_std=0.1, h_std=0.1)),
    3: dict(name="shplrnn_M32_L256_T65536_B8", kind="shplrnn", M=32, L=256, n_obs=32, B=8, T=65536, alpha=0.1,
            system="lorenz96", params=dict(a_range=(0.5, 0.95), h_std=0.1)),
    4: dict(name="diagssm_N64_T1048576_B4", kind="diag_ssm", M=64, L=128, n_obs=3, B=4, T=1 << 20, alpha=0.0,
            system="lorenz63", params={}),
    5: dict(name="plrnn_M64_T131072_B32", kind="plrnn", M=64, n_obs=64, B=32, T=131072, alpha=0.05,
            system="lorenz96", drift_period=5000.0, params=dict(a_range=(0.5, 0.9), w_std=0.05, h_std=0.1)),
}


def make_config(i: int, B: int | None = None, T: int | None = None) -> Workload:
    """Workload i (1..5) at its full size, or with B/T reduced (same distributions and seeds)."""
    spec = dict(CONFIG_SPECS[i])
    B = spec["B"] if B is None else B
    T = spec["T"] if T is None else T
    prng = np.random.default_rng(1000 * i)
    kind = spec["kind"]
    if kind == "plrnn":
        params = plrnn_params(spec["M"], prng, **spec["params"])
    elif kind == "shplrnn":
        params = shplrnn_params(spec["M"], spec["L"], prng, **spec["params"])
    else:
        params = diag_ssm_params(spec["M"], spec["n_obs"], spec["L"], spec["n_obs"], prng)
    x = observed_batch(spec["system"], spec["n_obs"], B, T, 1000 * i + 1,
                       drift_period=spec.get("drift_period"))
    return Workload(name=spec["name"], kind=kind, B=B, T=T, M=spec["M"], n_obs=spec["n_obs"],
                    alpha=spec["alpha"], params=params, x=x, L=spec.get("L", 0),
                    fixed_iters=spec.get("fixed_iters", 0),
                    meta={"config": i, "system": spec["system"], "drift_period": spec.get("drift_period")})


def random_plrnn_case(M: int, n_obs: int, B: int, T: int, alpha: float, seed: int, w_std: float = 0.1,
                      system: str = "lorenz63", w_norm: float | None = None, a_range=(0.5, 0.9)) -> Workload:
    """Small vanilla-PLRNN case for tests (any M >= 1, any n_obs <= M).  With w_norm, W is
    rescaled to that spectral norm (max A + w_norm < 1 makes the map a contraction)."""
    rng = np.random.default_rng(seed)
    params = plrnn_params(M, rng, a_range=a_range, w_std=w_std)
    if w_norm is not None:
        Wm = params["W"].astype(np.float64)
        s = np.linalg.norm(Wm, 2)
        params["W"] = (Wm * (w_norm / s if s > 0 else 1.0)).astype(np.float32)
    if system == "lorenz63" and n_obs <= 3:
        x = observed_batch("lorenz63", n_obs, B, T, seed + 1)
    else:
        x = observed_batch("lorenz96", max(n_obs, 4), B, T, seed + 1)[:, :, :n_obs].copy()
    return Workload(name=f"plrnn_M{M}_N{n_obs}_T{T}_B{B}", kind="plrnn", B=B, T=T, M=M, n_obs=n_obs,
                    alpha=alpha, params=params, x=np.ascontiguousarray(x))


def random_shplrnn_case(M: int, L: int, n_obs: int, B: int, T: int, alpha: float, seed: int,
                        w_norm: float | None = None, a_range=(0.5, 0.95)) -> Workload:
    """Small shallow-PLRNN case for tests.  With w_norm, W1 is rescaled so that
    ||W1||_2 ||W2||_2 = w_norm (max A + w_norm < 1 makes the map a contraction)."""
    rng = np.random.default_rng(seed)
    params = shplrnn_params(M, L, rng, a_range=a_range)
    if w_norm is not None:
        W1 = params["W1"].astype(np.float64)
        s = np.linalg.norm(W1, 2) * np.linalg.norm(params["W2"].astype(np.float64), 2)
        params["W1"] = (W1 * (w_norm / s)).astype(np.float32)
    x = observed_batch("lorenz96", max(n_obs, 4), B, T, seed + 1)[:, :, :n_obs].copy()
    return Workload(name=f"shplrnn_M{M}_L{L}_N{n_obs}_T{T}_B{B}", kind="shplrnn", B=B, T=T, M=M, n_obs=n_obs,
                    alpha=alpha, params=params, x=np.ascontiguousarray(x), L=L)
