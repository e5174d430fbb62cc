"""Float64 CPU oracle for the GTF-DEER hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's CPU
baseline leg use it.  It shares no code with the HIP library; the two meet only
through the seeded input generators (``workloads``), which hold none of the
method's arithmetic.

Everything here is plain and sequential on purpose: float64 (complex128 for the
diagonal SSM), Python loops over time, NumPy matrix products as the only
library primitive.  Inputs are the float32 arrays the GPU reads, promoted to
float64 (the forcing strength alpha too is rounded through float32 first).

Conventions (0-based arrays, paper indices in the comments):
  x    [B, T+1, N]   observations x_0..x_T
  z    [B, T, M]     states z_1..z_T (z[:, k] is z_{k+1})
  z0   [B, M]        fixed initial state z_0
  zt   [B, T, M]     forced states zt[:, k] = z~_k, the input of step k+1
  mask [B, T, H]     ReLU activation pattern of step k+1 (H = M or L)
The observation matrix is the identity read-out of the first N latents,
B = [I_N 0] (model-setup appendix, initialisation paragraph), so the teacher
states are zbar_t = [x_t; 0] and the projector P_alpha = I - alpha B^+ B is
diag(1 - a) with a_i = alpha for i < N and 0 otherwise -- except in the section
"general observation matrix" at the end, whose functions (suffix _obs) take any
N x M matrix B, form B^+ with numpy.linalg.pinv and the dense P_alpha, and give
the gradient with respect to B.

Readings of the paper taken here (each also listed in the design notes):
  * step 1 is unforced: z~_0 := z_0 (GTF-DEER residual definition); with the
    default z_0 = zbar_0 both readings coincide;
  * phi'(0) = 0, i.e. the activation mask is (u > 0) strictly;
  * the convergence test is absolute, per sequence, on max |Delta z| over all
    (t, m); the update is applied before the test and a converged sequence is
    frozen; ``iters`` counts updates including the verifying one;
  * loss = mean over the batch of the per-sequence MSE, so the seed is
    dL/dz_t = 2/(B N T) [z_t[:N] - x_t; 0];
  * the adjoint is exported as lam = dL/dz (= -v in the paper's sign).
Parity unpinned: nothing.  Every function is pinned by tests/test_oracle_pins.py
(closed forms, dense solves, brute force, finite differences and independent
automatic differentiation); absolute Newton iteration counts of the named
workloads have no paper value and are only reported.
"""
from __future__ import annotations

import numpy as np

f64 = np.float64


# --------------------------------------------------------------------------------------
# forcing: GTF mix and error-forcing projector (eqs. GTF, error_forcing)
# --------------------------------------------------------------------------------------

def alpha_as_gpu(alpha: float) -> float:
    """The forcing strength as the GPU sees it (float32), promoted to float64."""
    return float(np.float32(alpha))


def forcing_weights(M: int, n_forced: int, alpha: float) -> np.ndarray:
    """a with P_alpha = I - alpha B^+ B = diag(1 - a) for B = [I_N 0] (eq. error_forcing)."""
    a = np.zeros(M, f64)
    a[:n_forced] = alpha_as_gpu(alpha)
    return a


def forcing_schedule(M: int, n_forced: int, alpha: float, T: int, T_w: int = 0) -> np.ndarray:
    """a_k of the forced input z~_k for k = 0..T-1, shape [T, M]: alpha on the observed latents,
    and 1 there during the latent warm-up, k = 1..T_w (Alg. GTF-DEER: P_1 and the full forcing
    for t <= T_w; latent state warm-up paragraph).  Row 0 is unused (z~_0 = z_0)."""
    a = np.tile(forcing_weights(M, n_forced, alpha), (max(T, 1), 1))
    a[1:T_w + 1, :n_forced] = 1.0
    return a


def teacher_states(x: np.ndarray, M: int) -> np.ndarray:
    """zbar_t = B^+ x_t = [x_t; 0] for t = 0..T (Alg. GTF-DEER, forcing targets)."""
    x = np.asarray(x, f64)
    Bn, T1, N = x.shape
    zbar = np.zeros((Bn, T1, M), f64)
    zbar[:, :, :N] = x
    return zbar


def initial_state(x: np.ndarray, M: int, z0=None) -> np.ndarray:
    """z_0 = zbar_0 unless given (Alg. GTF-DEER initialisation)."""
    if z0 is None:
        return teacher_states(x[:, :1], M)[:, 0]
    return np.asarray(z0, f64).copy()


def forced_states(z: np.ndarray, zbar: np.ndarray, a: np.ndarray, z0: np.ndarray) -> np.ndarray:
    """z~_{t-1} = (1 - a) z_{t-1} + a zbar_{t-1} for t >= 2 and z~_0 = z_0 (eqs. GTF,
    error_forcing; GTF-DEER residual for step 1).  a is [M] or per step [T, M]."""
    zt = np.zeros_like(z)
    zt[:, 0] = z0
    ak = a if a.ndim == 1 else a[1:]
    zt[:, 1:] = (1.0 - ak) * z[:, :-1] + ak * zbar[:, 1:-1]
    return zt


# --------------------------------------------------------------------------------------
# models: vanilla PLRNN and shallow PLRNN (eq. shplrnn_nonlinear)
# --------------------------------------------------------------------------------------

def _p(model, k):
    return np.asarray(model[k], f64)


def _model64(model: dict) -> dict:
    """The parameters promoted to float64 once (the per-step helpers then reuse them)."""
    return {k: (v if k == "kind" or v is None else np.asarray(v, f64)) for k, v in model.items()}


def preactivation(model: dict, zt: np.ndarray) -> np.ndarray:
    """Argument of the ReLU: z~ itself (vanilla, V = I, b = 0) or W2 z~ + h2 (shallow)."""
    if model["kind"] == "plrnn":
        return zt
    return zt @ _p(model, "W2").T + _p(model, "h2")


def model_map(model: dict, zt: np.ndarray) -> np.ndarray:
    """F(z~) = diag(A) z~ + W relu(V z~ + b) + h (eq. shplrnn_nonlinear; no external inputs)."""
    u = preactivation(model, zt)
    relu = np.maximum(u, 0.0)
    if model["kind"] == "plrnn":
        return _p(model, "A") * zt + relu @ _p(model, "W").T + _p(model, "h")
    return _p(model, "A") * zt + relu @ _p(model, "W1").T + _p(model, "h1")


def activation_mask(model: dict, zt: np.ndarray) -> np.ndarray:
    """phi'(u) for phi = ReLU, decided in float64: (u > 0)."""
    return preactivation(model, zt) > 0.0


def activation_mask_fp32(model: dict, z: np.ndarray, x: np.ndarray, alpha: float, n_forced: int,
                         z0=None, T_w: int = 0) -> np.ndarray:
    """The same ReLU decision taken in float32, in the order the GPU kernels take it.

    Where floating point decides an integer both sides decide in the same
    precision.  z~ = fl(fl(p*z) + fl(a*zbar)) with p = fl(1 - a) (no fused
    multiply-add); at step 1, z~ = z_0.  Shallow model: u = h2 + sum_j W2_ij z~_j,
    accumulated left to right from h2 with a separate rounding after every
    multiply and every add.
    """
    f = np.float32
    z = np.asarray(z, f)
    Bn, T, M = z.shape
    a32 = np.zeros((T, M), f)
    a32[:, :n_forced] = f(alpha)
    a32[1:T_w + 1, :n_forced] = f(1.0)
    p32 = (f(1.0) - a32).astype(f)
    zbar = np.zeros((Bn, T + 1, M), f)
    zbar[:, :, :x.shape[2]] = np.asarray(x, f)
    zt = np.zeros((Bn, T, M), f)
    zt[:, 0] = zbar[:, 0] if z0 is None else np.asarray(z0, f)
    zt[:, 1:] = (p32[1:] * z[:, :-1]).astype(f) + (a32[1:] * zbar[:, 1:-1]).astype(f)
    if model["kind"] == "plrnn":
        return zt > 0
    W2 = np.asarray(model["W2"], f)
    acc = np.broadcast_to(np.asarray(model["h2"], f), (Bn, T, W2.shape[0])).copy()
    for j in range(M):
        acc = acc + (zt[:, :, j:j + 1] * W2[:, j]).astype(f)
    return acc > 0


def jvp(model: dict, mask: np.ndarray, v: np.ndarray) -> np.ndarray:
    """J_F v with J_F = diag(A) + W diag(phi') V (model-setup appendix, Jacobian of F)."""
    if model["kind"] == "plrnn":
        return _p(model, "A") * v + (mask * v) @ _p(model, "W").T
    return _p(model, "A") * v + (mask * (v @ _p(model, "W2").T)) @ _p(model, "W1").T


def vjp(model: dict, mask: np.ndarray, w: np.ndarray) -> np.ndarray:
    """J_F^T w for the same Jacobian."""
    if model["kind"] == "plrnn":
        return _p(model, "A") * w + mask * (w @ _p(model, "W"))
    return _p(model, "A") * w + (mask * (w @ _p(model, "W1"))) @ _p(model, "W2")


def jacobian_dense(model: dict, mask: np.ndarray) -> np.ndarray:
    """Dense J_F for masks [..., H]: diag(A) + W diag(m) V."""
    A = _p(model, "A")
    if model["kind"] == "plrnn":
        J = _p(model, "W") * mask[..., None, :]
    else:
        J = (_p(model, "W1") * mask[..., None, :]) @ _p(model, "W2")
    return J + np.diag(A)


def jacobian_diagonal(model: dict, mask: np.ndarray) -> np.ndarray:
    """diag(J_F) for masks [..., H], the quasi-DEER approximation of the Jacobian (DEER
    section, the diagonal replacing J_F in eq. DEER_update): A_i + W_ii m_i (vanilla) or
    A_i + sum_l W1_il m_l W2_li (shallow)."""
    A = _p(model, "A")
    if model["kind"] == "plrnn":
        return A + np.diagonal(_p(model, "W")) * mask
    C = _p(model, "W1") * _p(model, "W2").T          # C_il = W1_il W2_li
    return A + mask @ C.T


def forced_jacobians(model: dict, mask: np.ndarray, a: np.ndarray) -> np.ndarray:
    """J~_t = J_F(z~_{t-1}) P_alpha (eq. error_forcing_decomp), dense [B, T, M, M]."""
    return jacobian_dense(model, mask) * (1.0 - a)[None, :]


# --------------------------------------------------------------------------------------
# O1: sequential GTF rollout (Alg. initial value / trajectory matching with GTF)
# --------------------------------------------------------------------------------------

def rollout(model: dict, x: np.ndarray, alpha: float, n_forced: int, z0=None, T_w: int = 0) -> np.ndarray:
    """z_t = F(z~_{t-1}) for t = 1..T, one step at a time.  This is the unique
    zero-residual trajectory that DEER converges to.  T_w: latent warm-up (full forcing of
    the observed latents for z~_1..z~_{T_w})."""
    model = _model64(model)
    x = np.asarray(x, f64)
    Bn, T1, _ = x.shape
    T = T1 - 1
    M = np.asarray(model["A"]).shape[0]
    a = forcing_schedule(M, n_forced, alpha, T, T_w)
    zbar = teacher_states(x, M)
    zprev = initial_state(x, M, z0)
    z = np.zeros((Bn, T, M), f64)
    for t in range(1, T + 1):
        ztil = zprev if t == 1 else (1.0 - a[t - 1]) * zprev + a[t - 1] * zbar[:, t - 1]
        zprev = model_map(model, ztil)
        z[:, t - 1] = zprev
    return z


# --------------------------------------------------------------------------------------
# sequential affine recurrences (the operation the associative scan evaluates)
# --------------------------------------------------------------------------------------

def affine_recurrence(apply_J, b: np.ndarray) -> np.ndarray:
    """y_t = J_t y_{t-1} + b_t for t = 1..T with y_0 = 0 (eq. DEER_update as a linear
    recursion).  apply_J(k, v) returns J_{k+1} v for every batch row."""
    Bn, T, M = b.shape
    out = np.zeros_like(b)
    prev = np.zeros((Bn, M), b.dtype)
    for k in range(T):
        prev = apply_J(k, prev) + b[:, k]
        out[:, k] = prev
    return out


def reverse_affine_recurrence(apply_JT, g: np.ndarray) -> np.ndarray:
    """l_T = g_T and l_{t-1} = J_t^T l_t + g_{t-1} for t = T..2 (eq. backward_recursion).
    apply_JT(k, w) returns J_{k+1}^T w for every batch row."""
    Bn, T, M = g.shape
    out = np.zeros_like(g)
    nxt = g[:, T - 1].copy()
    out[:, T - 1] = nxt
    for k in range(T - 2, -1, -1):      # l_{k+1} (array index k) uses J_{k+2}
        nxt = apply_JT(k + 1, nxt) + g[:, k]
        out[:, k] = nxt
    return out


# --------------------------------------------------------------------------------------
# O2: explicit GTF-DEER Newton loop (Alg. GTF-DEER; eq. GTF_DEER_update)
# --------------------------------------------------------------------------------------

def residual_and_masks(model: dict, x: np.ndarray, z: np.ndarray, alpha: float, n_forced: int, z0=None,
                       T_w: int = 0):
    """r_t = z_t - F(z~_{t-1}) (eq. GTF_residual) together with F and the masks at z~."""
    model = _model64(model)
    x = np.asarray(x, f64)
    z = np.asarray(z, f64)
    M = z.shape[2]
    a = forcing_schedule(M, n_forced, alpha, z.shape[1], T_w)
    zbar = teacher_states(x, M)
    zt = forced_states(z, zbar, a, initial_state(x, M, z0))
    F = model_map(model, zt)
    return z - F, F, activation_mask(model, zt), zt


def newton(model: dict, x: np.ndarray, alpha: float, n_forced: int, *, z0=None, init: str = "teacher",
           z_init=None, tol: float = 1e-5, max_iter: int = 500, fixed_iters: int = 0, history: bool = False,
           gamma: float = 1.0, quasi: bool = False, T_w: int = 0):
    """GTF-DEER forward solve.  Each update linearises at z^(k): Delta_t =
    J~_t Delta_{t-1} - r_t, Delta_0 = 0, solved here by the sequential recursion,
    then z^(k+1) = z^(k) + Delta.  Returns dict(z, iters, norms, status[, history]).

    gamma scales the linearisation (Delta_t = gamma J~_t Delta_{t-1} - r_t): 1 is Newton's
    step of the algorithm, 0 the fixed-point step z_t <- F(z~_{t-1}); any gamma leaves the
    fixed point (r = 0) unchanged.  Used to pin the safeguarded GPU iteration.

    quasi: quasi-DEER, J~_t replaced by its diagonal diag(J_F(z~_{t-1})) P_alpha (the
    diagonal approximation discussed with eq. DEER_update), Delta_t = d_t * Delta_{t-1} - r_t;
    the fixed point is the same.

    T_w: latent warm-up, z~_k and J~_{k+1} with full forcing (P_1) for k = 1..T_w."""
    model = _model64(model)
    x = np.asarray(x, f64)
    Bn, T1, _ = x.shape
    T = T1 - 1
    M = np.asarray(model["A"]).shape[0]
    a = forcing_schedule(M, n_forced, alpha, T, T_w)
    p = 1.0 - a
    zbar = teacher_states(x, M)
    z0v = initial_state(x, M, z0)
    if init == "teacher":
        z = zbar[:, 1:].copy()
    elif init == "zero":
        z = np.zeros((Bn, T, M), f64)
    elif init == "user":
        z = np.asarray(z_init, f64).copy()
    else:
        raise ValueError(init)
    active = np.ones(Bn, bool)
    iters = np.zeros(Bn, np.int64)
    norms = np.full(Bn, np.nan)
    nonfinite = np.zeros(Bn, bool)
    hist = [z.copy()] if history else None
    k = 0
    while True:
        if fixed_iters > 0:
            if k == fixed_iters:
                break
        elif not active.any() or k == max_iter:
            break
        zt = forced_states(z, zbar, a, z0v)
        r = z - model_map(model, zt)
        mask = activation_mask(model, zt)
        if quasi:
            dg = jacobian_diagonal(model, mask) * p
            delta = affine_recurrence(lambda kk, v: gamma * (dg[:, kk] * v), -r)
        else:
            delta = affine_recurrence(lambda kk, v: gamma * jvp(model, mask[:, kk], p[kk] * v), -r)
        e = np.abs(delta).reshape(Bn, -1).max(axis=1) if T > 0 else np.zeros(Bn)
        e = np.where(np.isnan(delta).reshape(Bn, -1).any(axis=1), np.nan, e)
        upd = active if fixed_iters == 0 else np.ones(Bn, bool)
        z[upd] += delta[upd]
        iters[upd] += 1
        norms[upd] = e[upd]
        bad = upd & ~np.isfinite(e)
        nonfinite |= bad
        if fixed_iters == 0:
            active &= ~((e < tol) | bad)
        if history:
            hist.append(z.copy())
        k += 1
    status = "ok"
    if nonfinite.any():
        status = "nonfinite"
    elif fixed_iters == 0 and active.any():
        status = "not_converged"
    out = {"z": z, "iters": iters, "norms": norms, "status": status}
    if history:
        out["history"] = hist
    return out


# --------------------------------------------------------------------------------------
# O3: loss seed, IFT adjoint and parameter gradients (gradients appendix)
# --------------------------------------------------------------------------------------

def mse_loss(z: np.ndarray, x: np.ndarray, T_w: int = 0) -> float:
    """Batch mean of (1/(N (T - T_w))) sum_{t > T_w} ||x_t - B z_t||^2 (eqs. mse_loss_series,
    mse_loss_warmup: the warm-up states are excluded)."""
    z = np.asarray(z, f64)
    x = np.asarray(x, f64)
    Bn, T, _ = z.shape
    N = x.shape[2]
    return float(((z[:, T_w:, :N] - x[:, 1 + T_w:]) ** 2).sum() / (Bn * N * (T - T_w)))


def mse_seed(z: np.ndarray, x: np.ndarray, T_w: int = 0) -> np.ndarray:
    """dL/dz_t = 2/(B N (T - T_w)) B^T (B z_t - x_t) for t = T_w+1..T, zero in the warm-up."""
    z = np.asarray(z, f64)
    x = np.asarray(x, f64)
    Bn, T, M = z.shape
    N = x.shape[2]
    g = np.zeros((Bn, T, M), f64)
    g[:, T_w:, :N] = 2.0 / (Bn * N * (T - T_w)) * (z[:, T_w:, :N] - x[:, 1 + T_w:])
    return g


def _masks_at(model, x, z, alpha, n_forced, z0, mask_precision, T_w=0):
    r, F, mask64, zt = residual_and_masks(model, x, z, alpha, n_forced, z0, T_w)
    if mask_precision == "float32":
        mask = activation_mask_fp32(model, z, x, alpha, n_forced, z0, T_w)
    elif mask_precision == "float64":
        mask = mask64
    else:
        raise ValueError(mask_precision)
    return mask, zt


def adjoint(model: dict, x: np.ndarray, z: np.ndarray, alpha: float, n_forced: int, *, z0=None,
            g=None, mask_precision: str = "float64", quasi: bool = False, T_w: int = 0) -> np.ndarray:
    """lam = dL/dz by the backward recursion lam_T = g_T, lam_{t-1} = J~_t^T lam_t + g_{t-1}
    (eqs. adjoint_eq, backward_recursion with lam = -v).  J~_t is taken at z~_{t-1} of
    the given trajectory z (normally the converged one).

    quasi: the quasi-DEER backward recursion of the gradients appendix, the Jacobians
    replaced by their diagonals: lam_{t-1} = d_t * lam_t + g_{t-1}, d_t = diag(J~_t).  The
    parameter gradients then follow from this lam by param_grads unchanged."""
    model = _model64(model)
    z = np.asarray(z, f64)
    M = z.shape[2]
    p = 1.0 - forcing_schedule(M, n_forced, alpha, z.shape[1], T_w)
    mask, _ = _masks_at(model, x, z, alpha, n_forced, z0, mask_precision, T_w)
    g = mse_seed(z, x, T_w) if g is None else np.asarray(g, f64)
    if quasi:
        dg = jacobian_diagonal(model, mask) * p
        return reverse_affine_recurrence(lambda k, w: dg[:, k] * w, g)
    # J~^T w = P_alpha J_F^T w
    return reverse_affine_recurrence(lambda k, w: p[k] * vjp(model, mask[:, k], w), g)


def param_grads(model: dict, x: np.ndarray, z: np.ndarray, alpha: float, n_forced: int, lam: np.ndarray, *,
                z0=None, mask_precision: str = "float64", T_w: int = 0) -> dict:
    """dL/dtheta = sum_t lam_t^T dF(z~_{t-1})/dtheta (gradients appendix, IFT summary),
    summed directly over every (b, t) in float64."""
    model = _model64(model)
    z = np.asarray(z, f64)
    lam = np.asarray(lam, f64)
    mask, zt = _masks_at(model, x, z, alpha, n_forced, z0, mask_precision, T_w)
    out = {"A": np.einsum("bti,bti->i", lam, zt, optimize=True)}
    if model["kind"] == "plrnn":
        relu = np.where(mask, zt, 0.0)
        out["W"] = np.einsum("bti,btj->ij", lam, relu, optimize=True)
        out["h"] = lam.sum(axis=(0, 1))
    else:
        u = preactivation(model, zt)
        relu = np.where(mask, u, 0.0)
        delta = (lam @ _p(model, "W1")) * mask
        out["W1"] = np.einsum("bti,btl->il", lam, relu, optimize=True)
        out["W2"] = np.einsum("btl,btj->lj", delta, zt, optimize=True)
        out["h1"] = lam.sum(axis=(0, 1))
        out["h2"] = delta.sum(axis=(0, 1))
    return out


# --------------------------------------------------------------------------------------
# O4: residual, masks and forced Jacobians at a given trajectory
# --------------------------------------------------------------------------------------

def jacobian_at(model: dict, x: np.ndarray, z: np.ndarray, alpha: float, n_forced: int, *, z0=None,
                mask_precision: str = "float64", dense_index=None) -> dict:
    """F, r, masks and (for the (b, t) pairs in dense_index) dense J~_t at trajectory z."""
    r, F, mask64, zt = residual_and_masks(model, x, z, alpha, n_forced, z0)
    mask = mask64 if mask_precision == "float64" else activation_mask_fp32(model, z, x, alpha, n_forced, z0)
    out = {"F": F, "r": r, "mask": mask, "zt": zt}
    if dense_index is not None:
        M = z.shape[2]
        a = forcing_weights(M, n_forced, alpha)
        out["J"] = np.stack([forced_jacobians(model, mask[b, t], a) for (b, t) in dense_index])
    return out


# --------------------------------------------------------------------------------------
# O5: diagonal complex SSM (eq. shplrnn_ssm with diagonal complex A; Alg. LSSM)
# --------------------------------------------------------------------------------------

def diag_scan(lam: np.ndarray, b: np.ndarray) -> np.ndarray:
    """h_t = lam * h_{t-1} + b_t, h_0 = 0, t = 1..T, complex128."""
    lam = np.asarray(lam, np.complex128)
    b = np.asarray(b, np.complex128)
    h = np.zeros_like(b)
    prev = np.zeros(b.shape[:1] + b.shape[2:], np.complex128)
    for k in range(b.shape[1]):
        prev = lam * prev + b[:, k]
        h[:, k] = prev
    return h


def diag_scan_reverse(lam: np.ndarray, g: np.ndarray) -> np.ndarray:
    """a_T = g_T and a_{t-1} = conj(lam) * a_t + g_{t-1}: the transpose of diag_scan
    with the complex plane read as R^2 (the 2x2 block [[p,-q],[q,p]] transposes to
    multiplication by conj(lam))."""
    lam = np.asarray(lam, np.complex128)
    g = np.asarray(g, np.complex128)
    out = np.zeros_like(g)
    nxt = np.zeros(g.shape[:1] + g.shape[2:], np.complex128)
    for k in range(g.shape[1] - 1, -1, -1):
        nxt = np.conj(lam) * nxt + g[:, k]
        out[:, k] = nxt
    return out


def diag_ssm_inputs(params: dict, x: np.ndarray) -> np.ndarray:
    """b_t = Bc u_t with u_t = x_{t-1} (teacher input of the LSSM), t = 1..T."""
    u = np.asarray(x, f64)[:, :-1]
    return u @ np.asarray(params["Bc"], np.complex128).T


def diag_ssm_readout(params: dict, h: np.ndarray) -> np.ndarray:
    """y_t = Wb relu(Wa Re(h_t) + ca) + cb (one-hidden-layer MLP read-out)."""
    s = np.real(h) @ np.asarray(params["Wa"], f64).T + np.asarray(params["ca"], f64)
    return np.maximum(s, 0.0) @ np.asarray(params["Wb"], f64).T + np.asarray(params["cb"], f64)


def diag_ssm_readout_preactivation(params: dict, h: np.ndarray) -> np.ndarray:
    """s_t = Wa Re(h_t) + ca, the hidden pre-activation of the read-out."""
    return np.real(h) @ np.asarray(params["Wa"], f64).T + np.asarray(params["ca"], f64)


def diag_ssm_loss_and_seed(params: dict, h: np.ndarray, x: np.ndarray, mask=None):
    """MSE of the read-out against x_{1:T} and g = dL/dRe(h) (chain rule through the MLP).

    mask: optional boolean [B, T, H] of ReLU decisions to use instead of s > 0 (the
    decisions another implementation took; relu(s) = s * mask and relu' = mask)."""
    x = np.asarray(x, f64)
    Bn, T, _ = h.shape
    No = x.shape[2]
    Wa = np.asarray(params["Wa"], f64)
    Wb = np.asarray(params["Wb"], f64)
    s = diag_ssm_readout_preactivation(params, h)
    m = (s > 0.0) if mask is None else np.asarray(mask, bool)
    a1 = s * m
    y = a1 @ Wb.T + np.asarray(params["cb"], f64)
    err = y - x[:, 1:]
    loss = float((err ** 2).sum() / (Bn * No * T))
    dy = 2.0 / (Bn * No * T) * err
    ds = (dy @ Wb) * m
    g = ds @ Wa
    grads = {"Wb": np.einsum("bto,btk->ok", dy, a1, optimize=True), "cb": dy.sum(axis=(0, 1)),
             "Wa": np.einsum("btk,btn->kn", ds, np.real(h), optimize=True), "ca": ds.sum(axis=(0, 1))}
    return loss, g, grads


def diag_ssm_param_grads(a_adj: np.ndarray, h: np.ndarray, x: np.ndarray) -> dict:
    """dlam = sum_t a_t conj(h_{t-1}) and dBc = sum_t a_t u_t^T (u_t = x_{t-1}), the
    complex gradients d/dRe + i d/dIm."""
    hprev = np.concatenate([np.zeros_like(h[:, :1]), h[:, :-1]], axis=1)
    u = np.asarray(x, f64)[:, :-1]
    return {"lam": (a_adj * np.conj(hprev)).sum(axis=(0, 1)),
            "Bc": np.einsum("btn,btk->nk", a_adj, u, optimize=True)}


def diag_ssm_step(params: dict, x: np.ndarray) -> dict:
    """Forward scan, read-out loss, reverse scan and all gradients of the diagonal SSM."""
    b = diag_ssm_inputs(params, x)
    h = diag_scan(params["lam"], b)
    loss, g, mlp_grads = diag_ssm_loss_and_seed(params, h, x)
    a_adj = diag_scan_reverse(params["lam"], g.astype(np.complex128))
    grads = diag_ssm_param_grads(a_adj, h, x)
    grads.update(mlp_grads)
    return {"b": b, "h": h, "loss": loss, "g": g, "a": a_adj, "grads": grads}


# --------------------------------------------------------------------------------------
# training step around the gradient: MAR penalty and the parameter update
# --------------------------------------------------------------------------------------

def mar_loss_and_grads(model: dict, M_r: int, lam_mar: float, p: int, gamma_w: float, gamma_v: float):
    """Manifold attractor regularisation on the last M_r latents (eq. mar_loss_latent_initscale):
    lam_mar / M_r * sum_i [ |1 - A_i|^p + (1/L) sum_j (gamma_w |W_ij|^p + gamma_v |V_ji|^p) + |h_i|^p ].
    Vanilla PLRNN: V = I is not a parameter (no V term) and L = M; shallow: W = W1, V = W2,
    h = h1.  Returns (loss, grads) with the derivative of |u|^p taken as p |u|^(p-1) sign(u)
    (0 at u = 0 for p = 1)."""
    model = _model64(model)
    A = _p(model, "A")
    M = A.shape[0]
    sl = slice(M - M_r, M)
    c = lam_mar / M_r

    def pen(u):
        return np.abs(u) ** p

    def dpen(u):
        return p * np.abs(u) ** (p - 1) * np.sign(u) if p > 1 else np.sign(u)

    vanilla = model["kind"] == "plrnn"
    W = _p(model, "W") if vanilla else _p(model, "W1")
    h = _p(model, "h") if vanilla else _p(model, "h1")
    L = W.shape[1]
    loss = c * (pen(1.0 - A[sl]).sum() + pen(h[sl]).sum() + gamma_w / L * pen(W[sl]).sum())
    gA = np.zeros_like(A)
    gA[sl] = -c * dpen(1.0 - A[sl])
    gW = np.zeros_like(W)
    gW[sl] = c * gamma_w / L * dpen(W[sl])
    gh = np.zeros_like(h)
    gh[sl] = c * dpen(h[sl])
    if vanilla:
        return float(loss), {"A": gA, "W": gW, "h": gh}
    V = _p(model, "W2")
    loss += c * gamma_v / L * pen(V[:, sl]).sum()
    gV = np.zeros_like(V)
    gV[:, sl] = c * gamma_v / L * dpen(V[:, sl])
    return float(loss), {"A": gA, "W1": gW, "W2": gV, "h1": gh, "h2": np.zeros(L)}


def adam_update(params: dict, grads: dict, state: dict, step: int, lr: float, beta1: float = 0.9,
                beta2: float = 0.999, eps: float = 1e-8):
    """One Adam step (Kingma and Ba): m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2,
    theta -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps), t = step >= 1.  The paper
    names no optimiser; this is the reading taken.  Returns (new params, new state)."""
    out, st = {}, {}
    for k, g in grads.items():
        g = np.asarray(g, f64)
        m = beta1 * state.get(("m", k), np.zeros_like(g)) + (1 - beta1) * g
        v = beta2 * state.get(("v", k), np.zeros_like(g)) + (1 - beta2) * g * g
        mh = m / (1 - beta1 ** step)
        vh = v / (1 - beta2 ** step)
        out[k] = np.asarray(params[k], f64) - lr * mh / (np.sqrt(vh) + eps)
        st[("m", k)], st[("v", k)] = m, v
    return out, st


# --------------------------------------------------------------------------------------
# general observation matrix B (N x M): dense projector and its gradient
# (eqs. error_forcing, error_forcing_decomp; Alg. GTF-DEER: pinv(B), P_alpha, P_1, the
# forcing targets B^+ x and the gradient g_B)
# --------------------------------------------------------------------------------------

def obs_projectors(obs: np.ndarray, alpha: float):
    """B^+ = pinv(B), P_alpha = I - alpha B^+ B and P_1 = I - B^+ B (Alg. GTF-DEER, first line
    of the outer loop; eq. error_forcing).  Returns (B^+ [M, N], P_alpha, P_1)."""
    Bm = np.asarray(obs, f64)
    Bp = np.linalg.pinv(Bm)
    M = Bm.shape[1]
    a = alpha_as_gpu(alpha)
    return Bp, np.eye(M) - a * (Bp @ Bm), np.eye(M) - Bp @ Bm


def obs_alpha_schedule(alpha: float, T: int, T_w: int = 0) -> np.ndarray:
    """alpha_k of the forced input z~_k, k = 0..T-1: 1 in the warm-up k = 1..T_w, alpha after
    (Alg. GTF-DEER, warm-up and forced-input lines).  Entry 0 is unused (z~_0 = z_0)."""
    a = np.full(max(T, 1), alpha_as_gpu(alpha))
    a[1:T_w + 1] = 1.0
    return a


def obs_initial_state(x: np.ndarray, obs: np.ndarray, z0=None) -> np.ndarray:
    """z_0 = zbar_0 = B^+ x_0 unless given (Alg. GTF-DEER initialisation)."""
    if z0 is not None:
        return np.asarray(z0, f64).copy()
    Bp = np.linalg.pinv(np.asarray(obs, f64))
    return np.asarray(x, f64)[:, 0] @ Bp.T


def obs_forced_states(z: np.ndarray, x: np.ndarray, obs: np.ndarray, alpha: float, z0=None, T_w: int = 0):
    """z~_k = (I - alpha_k B^+ B) z_k + alpha_k B^+ x_k for k >= 1 and z~_0 = z_0 (eq.
    error_forcing with the warm-up schedule).  z holds z_1..z_T; returns [B, T, M]."""
    z = np.asarray(z, f64)
    x = np.asarray(x, f64)
    Bm = np.asarray(obs, f64)
    Bp = np.linalg.pinv(Bm)
    Bn, T, M = z.shape
    ak = obs_alpha_schedule(alpha, T, T_w)
    zt = np.zeros_like(z)
    zt[:, 0] = obs_initial_state(x, obs, z0)
    for k in range(1, T):
        zk = z[:, k - 1]
        zt[:, k] = zk - ak[k] * (zk @ (Bp @ Bm).T) + ak[k] * (x[:, k] @ Bp.T)
    return zt


def rollout_obs(model: dict, x: np.ndarray, obs: np.ndarray, alpha: float, z0=None, T_w: int = 0) -> np.ndarray:
    """Sequential GTF rollout z_t = F(z~_{t-1}) with the forcing of a general observation
    matrix (Alg. GTF-DEER's forward model; eq. error_forcing), one step at a time."""
    model = _model64(model)
    x = np.asarray(x, f64)
    Bm = np.asarray(obs, f64)
    Bp = np.linalg.pinv(Bm)
    Bn, T1, _ = x.shape
    T = T1 - 1
    M = Bm.shape[1]
    ak = obs_alpha_schedule(alpha, T, T_w)
    zprev = obs_initial_state(x, obs, z0)
    z = np.zeros((Bn, T, M), f64)
    for t in range(1, T + 1):
        k = t - 1
        if k == 0:
            ztil = zprev
        else:
            ztil = zprev - ak[k] * (zprev @ (Bp @ Bm).T) + ak[k] * (x[:, k] @ Bp.T)
        zprev = model_map(model, ztil)
        z[:, t - 1] = zprev
    return z


def newton_obs(model: dict, x: np.ndarray, obs: np.ndarray, alpha: float, *, z0=None, init: str = "teacher",
               tol: float = 1e-5, max_iter: int = 500, fixed_iters: int = 0, T_w: int = 0, history: bool = False):
    """GTF-DEER Newton loop (Alg. GTF-DEER) with a general observation matrix: initial guess
    z^(0)_t = B^+ x_t, residual r_t = z_t - F(z~_{t-1}), forced Jacobians J~_t =
    J_F(z~_{t-1}) P_{alpha_{t-1}} (eq. error_forcing_decomp; P_1 in the warm-up), the
    update Delta_t = J~_t Delta_{t-1} - r_t by the sequential recursion, z += Delta, until
    max |Delta| < tol per sequence (the same test as newton)."""
    model = _model64(model)
    x = np.asarray(x, f64)
    Bm = np.asarray(obs, f64)
    Bp = np.linalg.pinv(Bm)
    Bn, T1, _ = x.shape
    T = T1 - 1
    M = Bm.shape[1]
    ak = obs_alpha_schedule(alpha, T, T_w)
    Pk = np.stack([np.eye(M) - ak[k] * (Bp @ Bm) for k in range(T)])
    if init == "teacher":
        z = x[:, 1:] @ Bp.T
    elif init == "zero":
        z = np.zeros((Bn, T, M), f64)
    else:
        raise ValueError(init)
    active = np.ones(Bn, bool)
    iters = np.zeros(Bn, np.int64)
    norms = np.full(Bn, np.nan)
    hist = [z.copy()] if history else None
    k = 0
    while True:
        if fixed_iters > 0:
            if k == fixed_iters:
                break
        elif not active.any() or k == max_iter:
            break
        zt = obs_forced_states(z, x, obs, alpha, z0, T_w)
        r = z - model_map(model, zt)
        mask = activation_mask(model, zt)
        delta = affine_recurrence(lambda kk, v: jvp(model, mask[:, kk], v @ Pk[kk].T), -r)
        e = np.abs(delta).reshape(Bn, -1).max(axis=1)
        upd = active if fixed_iters == 0 else np.ones(Bn, bool)
        z[upd] += delta[upd]
        iters[upd] += 1
        norms[upd] = e[upd]
        if fixed_iters == 0:
            active &= ~(e < tol)
        if history:
            hist.append(z.copy())
        k += 1
    out = {"z": z, "iters": iters, "norms": norms,
           "status": "ok" if (fixed_iters > 0 or not active.any()) else "not_converged"}
    if history:
        out["history"] = hist
    return out


def mse_loss_obs(z: np.ndarray, x: np.ndarray, obs: np.ndarray, T_w: int = 0) -> float:
    """Batch mean of (1/(N (T - T_w))) sum_{t > T_w} ||x_t - B z_t||^2 (eq. mse_loss_warmup with
    the read-out x^_t = B z_t of eq. shplrnn_nonlinear)."""
    z = np.asarray(z, f64)
    x = np.asarray(x, f64)
    Bm = np.asarray(obs, f64)
    Bn, T, _ = z.shape
    N = Bm.shape[0]
    e = z[:, T_w:] @ Bm.T - x[:, 1 + T_w:]
    return float((e ** 2).sum() / (Bn * N * (T - T_w)))


def mse_seed_obs(z: np.ndarray, x: np.ndarray, obs: np.ndarray, T_w: int = 0) -> np.ndarray:
    """dL/dz_t = 2/(B N (T - T_w)) B^T (B z_t - x_t) for t > T_w, zero in the warm-up."""
    z = np.asarray(z, f64)
    x = np.asarray(x, f64)
    Bm = np.asarray(obs, f64)
    Bn, T, M = z.shape
    N = Bm.shape[0]
    g = np.zeros((Bn, T, M), f64)
    g[:, T_w:] = 2.0 / (Bn * N * (T - T_w)) * ((z[:, T_w:] @ Bm.T - x[:, 1 + T_w:]) @ Bm)
    return g


def adjoint_obs(model: dict, x: np.ndarray, z: np.ndarray, obs: np.ndarray, alpha: float, *, z0=None, g=None,
                T_w: int = 0, mask=None) -> np.ndarray:
    """lam = dL/dz by the backward recursion lam_T = g_T, lam_{t-1} = J~_t^T lam_t + g_{t-1}
    with J~_t^T = P_{alpha_{t-1}}^T J_F(z~_{t-1})^T (eqs. adjoint_eq, backward_recursion).
    mask: ReLU decisions to use instead of the float64 ones (the GPU's, for parity)."""
    model = _model64(model)
    z = np.asarray(z, f64)
    Bm = np.asarray(obs, f64)
    Bp = np.linalg.pinv(Bm)
    M = z.shape[2]
    ak = obs_alpha_schedule(alpha, z.shape[1], T_w)
    Pk = np.stack([np.eye(M) - ak[k] * (Bp @ Bm) for k in range(z.shape[1])])
    zt = obs_forced_states(z, x, obs, alpha, z0, T_w)
    mk = activation_mask(model, zt) if mask is None else np.asarray(mask, bool)
    g = mse_seed_obs(z, x, obs, T_w) if g is None else np.asarray(g, f64)
    return reverse_affine_recurrence(lambda k, w: vjp(model, mk[:, k], w) @ Pk[k], g)


def param_grads_obs(model: dict, x: np.ndarray, z: np.ndarray, obs: np.ndarray, alpha: float, lam: np.ndarray, *,
                    z0=None, T_w: int = 0, mask=None) -> dict:
    """dL/dtheta = sum_t lam_t^T dF(z~_{t-1})/dtheta (gradients appendix) at the forced inputs
    of a general observation matrix; the same sums as param_grads."""
    model = _model64(model)
    lam = np.asarray(lam, f64)
    zt = obs_forced_states(z, x, obs, alpha, z0, T_w)
    mk = activation_mask(model, zt) if mask is None else np.asarray(mask, bool)
    out = {"A": np.einsum("bti,bti->i", lam, zt, optimize=True)}
    if model["kind"] == "plrnn":
        out["W"] = np.einsum("bti,btj->ij", lam, np.where(mk, zt, 0.0), optimize=True)
        out["h"] = lam.sum(axis=(0, 1))
    else:
        u = preactivation(model, zt)
        delta = (lam @ _p(model, "W1")) * mk
        out["W1"] = np.einsum("bti,btl->il", lam, np.where(mk, u, 0.0), optimize=True)
        out["W2"] = np.einsum("btl,btj->lj", delta, zt, optimize=True)
        out["h1"] = lam.sum(axis=(0, 1))
        out["h2"] = delta.sum(axis=(0, 1))
    return out


def _dpinv_vjp(Bm: np.ndarray, Bp: np.ndarray, mu: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Gradient with respect to B of mu^T (dB^+) v for one pair of vectors (mu in R^M, v in
    R^N), from the differential of the Moore-Penrose inverse at constant rank (Golub and
    Pereyra 1973): dB^+ = -B^+ dB B^+ + B^+ B^+T dB^T (I - B B^+) + (I - B^+ B) dB^T B^+T B^+.
    Returns the N x M matrix G with mu^T (dB^+) v = sum(G * dB)."""
    M = Bm.shape[1]
    N = Bm.shape[0]
    g = -np.outer(Bp.T @ mu, Bp @ v)
    g += np.outer((np.eye(N) - Bm @ Bp) @ v, Bp @ (Bp.T @ mu))
    g += np.outer(Bp.T @ (Bp @ v), (np.eye(M) - Bp @ Bm) @ mu)
    return g


def obs_grad(model: dict, x: np.ndarray, z: np.ndarray, obs: np.ndarray, alpha: float, lam: np.ndarray, *,
             z0=None, T_w: int = 0, mask=None, with_mse: bool = True) -> np.ndarray:
    """dL/dB (Alg. GTF-DEER, g_B of the IFT gradient): the MSE's direct term
    2/(B N (T - T_w)) sum_{t > T_w} (B z_t - x_t) z_t^T, plus sum_t lam_t^T J_F(z~_{t-1})
    dz~_{t-1}/dB, where z~_k = z_k + alpha_k B^+ (x_k - B z_k) for k >= 1 and, when z_0 is
    not given, z~_0 = z_0 = B^+ x_0: with mu = J_F(z~_k)^T lam_{k+1},
    mu^T dz~_k = alpha_k [mu^T (dB^+) e_k - mu^T B^+ dB z_k],  e_k = x_k - B z_k.
    Each (b, k) is summed directly in float64."""
    model = _model64(model)
    x = np.asarray(x, f64)
    z = np.asarray(z, f64)
    lam = np.asarray(lam, f64)
    Bm = np.asarray(obs, f64)
    Bp = np.linalg.pinv(Bm)
    Bn, T, M = z.shape
    N = Bm.shape[0]
    ak = obs_alpha_schedule(alpha, T, T_w)
    zt = obs_forced_states(z, x, obs, alpha, z0, T_w)
    mk = activation_mask(model, zt) if mask is None else np.asarray(mask, bool)
    G = np.zeros((N, M), f64)
    for b in range(Bn):
        for k in range(T):
            mu = vjp(model, mk[b, k], lam[b, k])
            if k == 0:
                if z0 is None:
                    G += _dpinv_vjp(Bm, Bp, mu, x[b, 0])
                continue
            zk = z[b, k - 1]
            e = x[b, k] - Bm @ zk
            G += ak[k] * (_dpinv_vjp(Bm, Bp, mu, e) - np.outer(Bp.T @ mu, zk))
    if with_mse:
        e = z[:, T_w:] @ Bm.T - x[:, 1 + T_w:]
        G += 2.0 / (Bn * N * (T - T_w)) * np.einsum("btn,btj->nj", e, z[:, T_w:])
    return G
