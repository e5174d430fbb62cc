"""Pins of the float64 oracle against facts that do not come from the oracle.

Each test names the passage or mathematical fact it relies on.  The paper
prints no worked numerical example, so the pins are closed forms, textbook
routines (LAPACK dense solves, SVD), brute force over tiny sizes, central
finite differences and independent automatic differentiation (torch, CPU,
float64) of the sequential rollout.
"""
import itertools

import numpy as np
import pytest

import oracle as O
from oracle import brute
from workloads import plrnn_params, shplrnn_params, random_plrnn_case, random_shplrnn_case

torch = pytest.importorskip("torch")


def _vanilla(M, seed, w_std=0.3, a_range=(0.5, 0.9)):
    p = plrnn_params(M, np.random.default_rng(seed), a_range=a_range, w_std=w_std)
    return {"kind": "plrnn", **p}


def _shallow(M, L, seed):
    p = shplrnn_params(M, L, np.random.default_rng(seed))
    return {"kind": "shplrnn", **p}


def _x(B, T, N, seed):
    return np.random.default_rng(seed).standard_normal((B, T + 1, N)).astype(np.float32)


# ------------------------------------------------------------------------------------
# F itself: special cases with a closed form (eq. shplrnn_nonlinear)
# ------------------------------------------------------------------------------------

def test_model_map_permutation_closed_form():
    """With A = 0, h = 0 and W a permutation matrix, F(z)_i = relu(z_pi(i)); a transposed
    W would give relu(z_pi^-1(i)) instead (pi is a 3-cycle, not an involution)."""
    pi = np.array([1, 2, 0, 4, 3])
    W = np.zeros((5, 5), np.float32)
    W[np.arange(5), pi] = 1.0
    m = {"kind": "plrnn", "A": np.zeros(5, np.float32), "W": W, "h": np.zeros(5, np.float32)}
    z = np.array([[1.5, -2.0, 0.25, -0.5, 3.0]])
    F = O.model_map(m, z)
    assert np.array_equal(F[0], np.maximum(z[0, pi], 0.0))
    m2 = dict(m, A=np.array([0.5, 0.5, 0.5, 0.5, 0.5], np.float32), h=np.arange(5, dtype=np.float32))
    assert np.allclose(O.model_map(m2, z)[0], 0.5 * z[0] + np.maximum(z[0, pi], 0.0) + np.arange(5))


def test_shallow_map_permutation_closed_form():
    """Shallow PLRNN with W2 = permutation, W1 = I, h2 = 0: F = A z + relu(z_pi) + h1;
    with W2 = I, W1 = permutation: F = A z + relu(z)_pi + h1 (pi a 3-cycle)."""
    M = 3
    pi = np.array([2, 0, 1])
    P = np.zeros((M, M), np.float32)
    P[np.arange(M), pi] = 1.0
    A = np.array([0.1, 0.2, 0.3], np.float32)
    h1 = np.array([1.0, -1.0, 0.5], np.float32)
    z = np.array([[0.7, -1.2, 2.0]])
    m = {"kind": "shplrnn", "A": A, "W1": np.eye(M, dtype=np.float32), "W2": P, "h1": h1,
         "h2": np.zeros(M, np.float32)}
    assert np.allclose(O.model_map(m, z)[0], A * z[0] + np.maximum(z[0, pi], 0) + h1)
    m = dict(m, W1=P, W2=np.eye(M, dtype=np.float32))
    assert np.allclose(O.model_map(m, z)[0], A * z[0] + np.maximum(z[0], 0)[pi] + h1)
    m = dict(m, h2=np.array([-10.0, 10.0, 0.0], np.float32))   # hidden biases shift the kinks
    assert np.allclose(O.model_map(m, z)[0], A * z[0] + np.maximum(z[0] + m["h2"], 0)[pi] + h1)


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_jacobian_matches_finite_differences(kind):
    """J_F = diag(A) + W diag(phi'(Vz+b)) V (model-setup appendix) against central
    differences of F at points away from the ReLU kinks (F is linear on each cell)."""
    rng = np.random.default_rng(3)
    m = _vanilla(6, 1) if kind == "plrnn" else _shallow(5, 12, 2)
    for _ in range(5):
        z = rng.standard_normal((1, m["A"].shape[0]))
        u = O.preactivation(m, z)
        assume = np.abs(u).min() > 1e-3
        if not assume:
            continue
        J = O.jacobian_dense(m, O.activation_mask(m, z))[0]
        eps = 1e-6
        Jfd = np.empty_like(J)
        for j in range(z.shape[1]):
            e = np.zeros_like(z)
            e[0, j] = eps
            Jfd[:, j] = (O.model_map(m, z + e) - O.model_map(m, z - e))[0] / (2 * eps)
        assert np.allclose(J, Jfd, atol=1e-8)
        v = rng.standard_normal((1, z.shape[1]))
        mask = O.activation_mask(m, z)
        assert np.allclose(O.jvp(m, mask, v)[0], J @ v[0])
        assert np.allclose(O.vjp(m, mask, v)[0], J.T @ v[0])


def test_forcing_projector_is_identity_readout():
    """P_alpha = I - alpha B^+ B with B = [I_N 0]: B^+ = B^T, so P_alpha = diag(1-a)
    (eq. error_forcing); checked against numpy's pseudo-inverse."""
    M, N, alpha = 7, 3, 0.3
    Bm = np.hstack([np.eye(N), np.zeros((N, M - N))])
    P = np.eye(M) - O.alpha_as_gpu(alpha) * np.linalg.pinv(Bm) @ Bm
    assert np.allclose(P, np.diag(1.0 - O.forcing_weights(M, N, alpha)))
    x = _x(2, 4, N, 0)
    zbar = O.teacher_states(x, M)
    assert np.allclose(zbar, np.einsum("mn,btn->btm", np.linalg.pinv(Bm), x))


# ------------------------------------------------------------------------------------
# P1: the affine recurrence, its transpose and the scan decomposition
# ------------------------------------------------------------------------------------

@pytest.mark.parametrize("T", [1, 2, 3, 7, 16])
def test_affine_recurrence_equals_block_bidiagonal_solve(T):
    """y_t = J_t y_{t-1} + b_t is the solution of the block-bidiagonal system of
    eq. blockdiag_jacobian; its transpose solves the adjoint system (eq. adjoint_eq)."""
    rng = np.random.default_rng(T)
    M = 3
    J = rng.standard_normal((T, M, M)) * 0.7
    b = rng.standard_normal((T, M))
    y = O.affine_recurrence(lambda k, v: v @ J[k].T, b[None])[0]
    assert np.allclose(y, brute.block_bidiagonal_solve(J, b), rtol=1e-12, atol=1e-12)
    g = rng.standard_normal((T, M))
    lam = O.reverse_affine_recurrence(lambda k, w: w @ J[k], g[None])[0]
    assert np.allclose(lam, brute.block_bidiagonal_adjoint_solve(J, g), rtol=1e-12, atol=1e-12)
    # transpose identity <g, S b> = <S^T g, b>
    assert np.isclose((g * y).sum(), (lam * b).sum(), rtol=1e-12)


@pytest.mark.parametrize("T", [1, 2, 4, 6, 8])
def test_every_bracketing_gives_the_same_map(T):
    """Associativity of (A2, b2) o (A1, b1) = (A2 A1, A2 b1 + b2) (scheduled-sampling
    appendix): every bracketing equals the sequential fold; its b is y_T."""
    rng = np.random.default_rng(10 + T)
    M = 2
    J = rng.standard_normal((T, M, M))
    b = rng.standard_normal((T, M))
    elems = [(J[k], b[k]) for k in range(T)]
    y = O.affine_recurrence(lambda k, v: v @ J[k].T, b[None])[0]
    Pseq = np.eye(M)
    for k in range(T):
        Pseq = J[k] @ Pseq
    for P, v in brute.all_bracketings(elems):
        assert np.allclose(P, Pseq, rtol=1e-12, atol=1e-12)
        assert np.allclose(v, y[-1], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("T", [1, 5, 16])
def test_chunked_scan_equals_recurrence_for_every_chunk(T):
    rng = np.random.default_rng(20 + T)
    M = 4
    J = rng.standard_normal((T, M, M)) * 0.5
    b = rng.standard_normal((T, M))
    y = O.affine_recurrence(lambda k, v: v @ J[k].T, b[None])[0]
    for C in range(1, T + 1):
        assert np.allclose(brute.chunked_scan(J, b, C), y, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------------------------
# P2/P3/P6: Newton reaches the rollout; prefix exactness; finite termination
# ------------------------------------------------------------------------------------

@pytest.mark.parametrize("kind,M,N,alpha", [("plrnn", 4, 3, 0.2), ("plrnn", 3, 3, 0.1), ("plrnn", 16, 3, 0.2),
                                            ("shplrnn", 5, 5, 0.1), ("shplrnn", 6, 2, 0.3)])
def test_newton_converges_to_rollout(kind, M, N, alpha):
    """The zero of the GTF residual is the sequential GTF rollout (DEER section and
    GTF-DEER residual); Newton in float64 with eps = 1e-13 reaches it to 1e-11."""
    m = _vanilla(M, 5) if kind == "plrnn" else _shallow(M, 3 * M, 6)
    x = _x(3, 60, N, 7)
    ref = O.rollout(m, x, alpha, N)
    res = O.newton(m, x, alpha, N, tol=1e-13, max_iter=200)
    assert res["status"] == "ok"
    assert np.abs(res["z"] - ref).max() <= 1e-11
    zr = O.rollout(m, x, alpha, N, z0=np.ones((3, M)))     # user initial state
    rz = O.newton(m, x, alpha, N, z0=np.ones((3, M)), init="zero", tol=1e-13, max_iter=200)
    assert np.abs(rz["z"] - zr).max() <= 1e-11


def test_rollout_residual_is_zero():
    m = _vanilla(5, 8)
    x = _x(2, 30, 3, 9)
    z = O.rollout(m, x, 0.3, 3)
    r, _, _, _ = O.residual_and_masks(m, x, z, 0.3, 3)
    assert np.abs(r).max() < 1e-13


@pytest.mark.parametrize("init", ["teacher", "zero"])
def test_newton_prefix_exactness(init):
    """With Delta_0 = 0 and z_0 fixed, after k updates z_1..z_k are exact (eq. DEER_update
    read step by step); hence termination within T updates plus the verifying one."""
    m = _vanilla(3, 11, w_std=0.8)
    T = 12
    x = _x(2, T, 3, 12)
    ref = O.rollout(m, x, 0.0, 3)
    res = O.newton(m, x, 0.0, 3, init=init, fixed_iters=T, history=True)
    for k, zk in enumerate(res["history"]):
        if k == 0:
            continue
        assert np.abs(zk[:, :k] - ref[:, :k]).max() < 1e-12, k
    full = O.newton(m, x, 0.0, 3, init=init, tol=1e-12, max_iter=100)
    assert full["iters"].max() <= T + 1


@pytest.mark.parametrize("gamma", [0.0, 0.5])
def test_damped_newton_prefix_and_fixed_point(gamma):
    """The damped step Delta_t = gamma J~_t Delta_{t-1} - r_t (the safeguard of the GPU
    solve) keeps the fixed point of the GTF residual and the prefix property of the DEER
    update: after k updates z_1..z_k are exact, for every gamma in [0, 1]."""
    m = _vanilla(3, 11, w_std=0.8)
    T = 12
    x = _x(2, T, 3, 12)
    alpha = 0.2
    ref = O.rollout(m, x, alpha, 3)
    res = O.newton(m, x, alpha, 3, fixed_iters=T, history=True, gamma=gamma)
    for k, zk in enumerate(res["history"]):
        if k:
            assert np.abs(zk[:, :k] - ref[:, :k]).max() < 1e-12, k
    assert np.abs(res["z"] - ref).max() < 1e-12
    full = O.newton(m, x, alpha, 3, tol=1e-12, max_iter=100, gamma=gamma)
    assert full["status"] == "ok" and full["iters"].max() <= T + 1


def test_undamped_fixed_point_step_is_local():
    """gamma = 0 is the fixed-point step z_t <- F(z~_{t-1}): a change of the iterate at
    step s changes the next iterate at step s + 1 only (z + (F - z) rounds, hence the
    threshold at step s itself)."""
    m = _vanilla(4, 21)
    x = _x(1, 20, 2, 22)
    z = np.random.default_rng(23).standard_normal((1, 20, 4))
    base = O.newton(m, x, 0.3, 2, init="user", z_init=z, fixed_iters=1, gamma=0.0)["z"]
    for s in (0, 7, 19):
        z2 = z.copy()
        z2[0, s] += 0.5
        moved = O.newton(m, x, 0.3, 2, init="user", z_init=z2, fixed_iters=1, gamma=0.0)["z"]
        diff = np.abs(moved - base).max(axis=2)[0]
        changed = np.nonzero(diff > 1e-12)[0].tolist()
        assert changed == ([s + 1] if s + 1 < 20 else []), (s, changed)


def test_newton_lands_on_fixed_point_once_masks_match():
    """F is affine on each activation cell, so a Newton update linearised at an iterate
    that shares the fixed point's masks is exact: one update from a small perturbation
    of z* returns z* (pins J~_t = J_F(z~) P_alpha: any other matrix leaves an error)."""
    m = _vanilla(6, 13)
    x = _x(2, 40, 4, 14)
    alpha = 0.25
    zs = O.rollout(m, x, alpha, 4)
    _, _, mask_s, zt_s = O.residual_and_masks(m, x, zs, alpha, 4)
    pert = 1e-7 * np.random.default_rng(1).standard_normal(zs.shape)
    z1 = zs + pert
    _, _, mask1, _ = O.residual_and_masks(m, x, z1, alpha, 4)
    assert np.array_equal(mask1, mask_s), "perturbation crossed a kink; choose a smaller one"
    res = O.newton(m, x, alpha, 4, init="user", z_init=z1, fixed_iters=1)
    assert np.abs(res["z"] - zs).max() < 1e-13
    res2 = O.newton(m, x, alpha, 4, init="user", z_init=z1, tol=1e-10)
    assert res2["iters"].tolist() == [2, 2]


# ------------------------------------------------------------------------------------
# P4/P5: alpha = 0 on a linear model; alpha = 1 reproduces the data-driven states
# ------------------------------------------------------------------------------------

def test_alpha0_linear_model_closed_form_and_two_iterations():
    """W = 0: z_t = A^t z_0 + (1 - A^t)/(1 - A) h, and DEER needs exactly 2 updates
    (the first exact, the second verifying; footnote to the runtime section)."""
    M, T = 4, 50
    A = np.array([0.5, 0.7, 0.9, 0.95], np.float32)
    h = np.array([0.1, -0.2, 0.3, 0.05], np.float32)
    m = {"kind": "plrnn", "A": A, "W": np.zeros((M, M), np.float32), "h": h}
    x = _x(2, T, M, 15)
    z0 = x[:, 0].astype(np.float64)
    t = np.arange(1, T + 1)[None, :, None]
    A64, h64 = A.astype(np.float64), h.astype(np.float64)
    closed = A64 ** t * z0[:, None, :] + (1 - A64 ** t) / (1 - A64) * h64
    res = O.newton(m, x, 0.0, M, tol=1e-10)
    assert np.abs(res["z"] - closed).max() < 1e-12
    assert res["iters"].tolist() == [2, 2]
    assert np.abs(O.rollout(m, x, 0.0, M) - closed).max() < 1e-12


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_alpha1_full_observation_closed_form(kind):
    """alpha = 1 and M <= N: z~ = zbar, J~ = 0, so z*_t = F(zbar_{t-1}) in closed form and
    DEER stops after 2 updates."""
    M = 4
    m = _vanilla(M, 16, w_std=1.0) if kind == "plrnn" else _shallow(M, 9, 17)
    x = _x(3, 25, M, 18)
    xb = x.astype(np.float64)
    closed = O.model_map(m, xb[:, :-1])
    res = O.newton(m, x, 1.0, M, tol=1e-10)
    assert np.abs(res["z"] - closed).max() < 1e-13
    assert res["iters"].tolist() == [2, 2, 2]


def test_prop1_contraction_bound():
    """Prop. 1 (M <= N): J~_t = (1 - alpha) J_F, so ||J~_t||_2 <= (1 - alpha) sigma~_max and
    products of k forced Jacobians are bounded by rho^k.  sigma~_max is exact here: a
    vanilla PLRNN with M = 3 has only 2^3 distinct Jacobians."""
    M = 3
    m = _vanilla(M, 19, w_std=1.2)
    sig = max(np.linalg.svd(O.jacobian_dense(m, np.array(mk, bool)), compute_uv=False)[0]
              for mk in itertools.product([0, 1], repeat=M))
    assert sig > 1.0
    alpha = 1.0 - 1.0 / sig + 0.05
    rho = (1.0 - O.alpha_as_gpu(alpha)) * sig
    assert rho < 1.0
    x = _x(1, 80, M, 20)
    z = O.rollout(m, x, alpha, M)
    _, _, mask, _ = O.residual_and_masks(m, x, z, alpha, M)
    Jt = O.forced_jacobians(m, mask[0], O.forcing_weights(M, M, alpha))
    for k in range(80):
        assert np.linalg.svd(Jt[k], compute_uv=False)[0] <= rho * (1 + 1e-12)
    P = np.eye(M)
    for k in range(80):
        P = Jt[k] @ P
        assert np.linalg.norm(P, 2) <= rho ** (k + 1) * (1 + 1e-9)


# ------------------------------------------------------------------------------------
# P8/P9: adjoint and parameter gradients
# ------------------------------------------------------------------------------------

@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_adjoint_equals_dense_adjoint_solve(kind):
    """lam solves R^T lam = dL/dz for R = dR/dz (eq. blockdiag_jacobian, eq. adjoint_eq)."""
    M, N, T, alpha = 4, 2, 14, 0.3
    m = _vanilla(M, 21) if kind == "plrnn" else _shallow(M, 8, 22)
    x = _x(1, T, N, 23)
    z = O.rollout(m, x, alpha, N)
    _, _, mask, _ = O.residual_and_masks(m, x, z, alpha, N)
    J = O.forced_jacobians(m, mask[0], O.forcing_weights(M, N, alpha))
    g = O.mse_seed(z, x)[0]
    lam = O.adjoint(m, x, z, alpha, N)[0]
    assert np.allclose(lam, brute.block_bidiagonal_adjoint_solve(J, g), rtol=1e-12, atol=1e-14)


def _torch_bptt(m, x, alpha, N, T_w=0):
    """Independent reverse-mode AD (torch, float64) through the sequential GTF rollout
    of Alg. 2 and the MSE loss: the BPTT gradient the IFT gradient must equal.  T_w: the
    first T_w forced inputs fully forced, their states left out of the loss."""
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    P = {k: t(v) for k, v in m.items() if k != "kind"}
    xt = torch.tensor(np.asarray(x, np.float64))
    Bn, T1, _ = x.shape
    M = P["A"].shape[0]
    a = torch.zeros(M, dtype=torch.float64)
    a[:N] = float(np.float32(alpha))
    zbar = torch.zeros(Bn, T1, M, dtype=torch.float64)
    zbar[:, :, :N] = xt
    prev = zbar[:, 0]
    loss = 0.0
    aw = a.clone()
    aw[:N] = 1.0
    for k in range(1, T1):
        ak = aw if k - 1 <= T_w else a
        zt = prev if k == 1 else (1 - ak) * prev + ak * zbar[:, k - 1]
        if m["kind"] == "plrnn":
            prev = P["A"] * zt + torch.relu(zt) @ P["W"].T + P["h"]
        else:
            prev = P["A"] * zt + torch.relu(zt @ P["W2"].T + P["h2"]) @ P["W1"].T + P["h1"]
        if k > T_w:
            loss = loss + ((prev[:, :N] - xt[:, k]) ** 2).sum()
    loss = loss / (Bn * N * (T1 - 1 - T_w))
    loss.backward()
    return float(loss.detach()), {k: v.grad.numpy() for k, v in P.items()}


@pytest.mark.parametrize("kind,M,N,alpha", [("plrnn", 5, 3, 0.2), ("plrnn", 3, 3, 0.1), ("shplrnn", 4, 4, 0.15),
                                            ("shplrnn", 6, 2, 0.3)])
def test_ift_gradient_equals_bptt(kind, M, N, alpha):
    """The IFT gradient at the fixed point equals BPTT through the sequential rollout
    (gradients appendix vs Alg. 2)."""
    m = _vanilla(M, 31) if kind == "plrnn" else _shallow(M, 10, 32)
    x = _x(2, 40, N, 33)
    z = O.newton(m, x, alpha, N, tol=1e-13)["z"]
    loss_ref, gref = _torch_bptt(m, x, alpha, N)
    assert np.isclose(O.mse_loss(z, x), loss_ref, rtol=1e-12)
    lam = O.adjoint(m, x, z, alpha, N)
    g = O.param_grads(m, x, z, alpha, N, lam)
    for k, v in gref.items():
        assert np.allclose(g[k], v, rtol=1e-10, atol=1e-13), k


def test_param_grads_central_differences():
    """dL/dtheta of L(z*(theta)) by central differences (float64, h = 1e-6) for a few
    entries of every parameter, at a trajectory with no activation near zero."""
    m = _vanilla(3, 41)
    x = _x(1, 30, 2, 42)
    alpha = 0.2
    z = O.rollout(m, x, alpha, 2)
    _, _, _, zt = O.residual_and_masks(m, x, z, alpha, 2)
    assert np.abs(zt[:, 1:]).min() > 1e-4     # z~_0 = z_0 is data, independent of theta
    g = O.param_grads(m, x, z, alpha, 2, O.adjoint(m, x, z, alpha, 2))
    mf = {k: (np.asarray(v, np.float64) if k != "kind" else v) for k, v in m.items()}
    for name, idx in [("A", (1,)), ("W", (0, 2)), ("W", (2, 1)), ("h", (0,))]:
        hstep = 1e-6
        mp = {k: (v.copy() if k != "kind" else v) for k, v in mf.items()}
        mm = {k: (v.copy() if k != "kind" else v) for k, v in mf.items()}
        mp[name][idx] += hstep
        mm[name][idx] -= hstep
        fd = (O.mse_loss(O.rollout(mp, x, alpha, 2), x) - O.mse_loss(O.rollout(mm, x, alpha, 2), x)) / (2 * hstep)
        assert np.isclose(g[name][idx], fd, rtol=1e-6, atol=1e-10), (name, idx)


def test_fp32_mask_decision_agrees_away_from_ties():
    """The float32 ReLU decision (kernel precision) equals the float64 one wherever the
    pre-activation is not within float32 rounding of zero."""
    for case in [random_plrnn_case(8, 3, 2, 200, 0.2, 50), random_shplrnn_case(6, 20, 6, 2, 100, 0.1, 51)]:
        m = {"kind": case.kind, **case.params}
        z = O.rollout(m, case.x, case.alpha, case.n_obs).astype(np.float32)
        _, _, mask64, zt = O.residual_and_masks(m, case.x, z, case.alpha, case.n_obs)
        u = O.preactivation(m, zt)
        m32 = O.activation_mask_fp32(m, z, case.x, case.alpha, case.n_obs)
        far = np.abs(u) > 1e-5 * (1 + np.abs(u).max())
        assert np.array_equal(m32[far], mask64[far])


# ------------------------------------------------------------------------------------
# P10: diagonal complex SSM
# ------------------------------------------------------------------------------------

def test_diag_scan_closed_forms():
    """Impulse response h_t = lam^(t-1) b_1 and constant input h_t = (1 - lam^t)/(1 - lam) b
    (linear-SSM appendix: dz_t/dz_r = A^(t-r))."""
    rng = np.random.default_rng(60)
    lam = 0.97 * np.exp(1j * rng.uniform(0, np.pi / 10, 5))
    T = 200
    b = np.zeros((1, T, 5), np.complex128)
    b[0, 0] = 1.0 + 0.5j
    h = O.diag_scan(lam, b)
    t = np.arange(T)[:, None]
    assert np.allclose(h[0], lam ** t * (1.0 + 0.5j), rtol=1e-12, atol=1e-14)
    c = rng.standard_normal(5) + 1j * rng.standard_normal(5)
    h = O.diag_scan(lam, np.broadcast_to(c, (1, T, 5)))
    tt = np.arange(1, T + 1)[:, None]
    assert np.allclose(h[0], (1 - lam ** tt) / (1 - lam) * c, rtol=1e-11)
    g = rng.standard_normal((1, T, 5)) + 1j * rng.standard_normal((1, T, 5))
    a = O.diag_scan_reverse(lam, g)
    bb = rng.standard_normal((1, T, 5)) + 1j * rng.standard_normal((1, T, 5))
    # real inner product on C = R^2: <g, S b> = <S^T g, b>
    assert np.isclose(np.real(np.conj(g) * O.diag_scan(lam, bb)).sum(), np.real(np.conj(a) * bb).sum(), rtol=1e-11)


def test_diag_ssm_gradients_match_autograd():
    """Gradients of the diagonal SSM training loss (scan, MLP read-out, MSE) against torch
    autograd with lam and Bc parametrised by their real and imaginary parts."""
    from workloads import diag_ssm_params
    prm = diag_ssm_params(6, 3, 8, 3, np.random.default_rng(70))
    x = _x(2, 50, 3, 71)
    out = O.diag_ssm_step(prm, x)
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    lr, li = t(prm["lam"].real), t(prm["lam"].imag)
    br, bi = t(prm["Bc"].real), t(prm["Bc"].imag)
    Wa, ca, Wb, cb = t(prm["Wa"]), t(prm["ca"]), t(prm["Wb"]), t(prm["cb"])
    xt = torch.tensor(x.astype(np.float64))
    Bn, T1, _ = x.shape
    hr = torch.zeros(Bn, 6, dtype=torch.float64)
    hi = torch.zeros(Bn, 6, dtype=torch.float64)
    loss = 0.0
    for k in range(1, T1):
        u = xt[:, k - 1]
        hr, hi = lr * hr - li * hi + u @ br.T, lr * hi + li * hr + u @ bi.T
        y = torch.relu(hr @ Wa.T + ca) @ Wb.T + cb
        loss = loss + ((y - xt[:, k]) ** 2).sum()
    loss = loss / (Bn * 3 * (T1 - 1))
    loss.backward()
    G = out["grads"]
    assert np.isclose(out["loss"], float(loss.detach()), rtol=1e-12)
    assert np.allclose(G["lam"], lr.grad.numpy() + 1j * li.grad.numpy(), rtol=1e-9, atol=1e-13)
    assert np.allclose(G["Bc"], br.grad.numpy() + 1j * bi.grad.numpy(), rtol=1e-9, atol=1e-13)
    for k, v in [("Wa", Wa), ("ca", ca), ("Wb", Wb), ("cb", cb)]:
        assert np.allclose(G[k], v.grad.numpy(), rtol=1e-9, atol=1e-13), k


def test_readout_with_given_masks_matches_autograd():
    """The mask-conditioned read-out (ReLU decisions supplied from outside, as the GPU parity
    tests do) equals torch autograd of y = Wb (s * m) + cb with that fixed mask m, for a
    random mask; with m = (s > 0) it reproduces the plain read-out."""
    from workloads import diag_ssm_params
    prm = diag_ssm_params(5, 2, 7, 2, np.random.default_rng(80))
    rng = np.random.default_rng(81)
    h = rng.standard_normal((2, 9, 5)) + 1j * rng.standard_normal((2, 9, 5))
    x = _x(2, 9, 2, 82)
    s = O.diag_ssm_readout_preactivation(prm, h)
    base = O.diag_ssm_loss_and_seed(prm, h, x)
    own = O.diag_ssm_loss_and_seed(prm, h, x, mask=s > 0)
    assert base[0] == own[0] and np.array_equal(base[1], own[1])
    m = rng.random(s.shape) < 0.5
    loss, g, gr = O.diag_ssm_loss_and_seed(prm, h, x, mask=m)
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    hr = t(h.real)
    Wa, ca, Wb, cb = t(prm["Wa"]), t(prm["ca"]), t(prm["Wb"]), t(prm["cb"])
    st = hr @ Wa.T + ca
    y = (st * torch.tensor(m, dtype=torch.float64)) @ Wb.T + cb
    L = ((y - torch.tensor(x[:, 1:].astype(np.float64))) ** 2).sum() / (2 * 2 * 9)
    L.backward()
    assert np.isclose(loss, float(L.detach()), rtol=1e-12)
    assert np.allclose(g, hr.grad.numpy(), rtol=1e-10, atol=1e-14)
    for k, v in [("Wa", Wa), ("ca", ca), ("Wb", Wb), ("cb", cb)]:
        assert np.allclose(gr[k], v.grad.numpy(), rtol=1e-10, atol=1e-14), k


# ------------------------------------------------------------------------------------
# quasi-DEER: every forced Jacobian replaced by its diagonal (the diagonal approximation
# discussed with eq. DEER_update; quasi form of the backward recursion, gradients appendix)
# ------------------------------------------------------------------------------------

def _diag_blocks(d):
    """[T, M] diagonals -> [T, M, M] diagonal blocks."""
    return np.einsum("ti,ij->tij", d, np.eye(d.shape[1]))


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_jacobian_diagonal_central_differences(kind):
    """d_i = dF_i / dz~_i, by central differences of F itself (no ReLU ties nearby)."""
    M = 5
    m = _vanilla(M, 41) if kind == "plrnn" else _shallow(M, 9, 42)
    zt = np.random.default_rng(43).standard_normal((6, M))
    d = O.jacobian_diagonal(m, O.activation_mask(m, zt))
    eps = 1e-6
    for i in range(M):
        e = np.zeros(M)
        e[i] = eps
        fd = (O.model_map(m, zt + e)[:, i] - O.model_map(m, zt - e)[:, i]) / (2 * eps)
        assert np.allclose(fd, d[:, i], rtol=1e-7, atol=1e-8), i


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_quasi_equals_deer_when_every_jacobian_is_diagonal(kind):
    """Diagonal W (vanilla), or diagonal W1 and W2 with L = M (shallow), make every J_F
    diagonal: quasi-DEER then takes exactly DEER's steps and has DEER's adjoint."""
    M, N, T, alpha = 4, 2, 40, 0.25
    rng = np.random.default_rng(44)
    A, h = rng.uniform(0.3, 0.8, M), rng.normal(0, 0.1, M)
    if kind == "plrnn":
        m = {"kind": "plrnn", "A": A, "W": np.diag(rng.normal(0, 0.5, M)), "h": h}
    else:
        m = {"kind": "shplrnn", "A": A, "W1": np.diag(rng.normal(0, 0.7, M)), "W2": np.diag(rng.normal(0, 0.7, M)),
             "h1": h, "h2": rng.normal(0, 0.1, M)}
    x = _x(2, T, N, 45)
    full = O.newton(m, x, alpha, N, fixed_iters=6, history=True)
    qd = O.newton(m, x, alpha, N, fixed_iters=6, history=True, quasi=True)
    for a, b in zip(full["history"], qd["history"]):
        assert np.abs(a - b).max() < 1e-12
    z = O.rollout(m, x, alpha, N)
    assert np.allclose(O.adjoint(m, x, z, alpha, N, quasi=True), O.adjoint(m, x, z, alpha, N), rtol=1e-12,
                       atol=1e-15)


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_quasi_update_and_adjoint_are_diagonal_block_solves(kind):
    """One quasi-DEER update solves the block-bidiagonal system with blocks diag(d_t) below
    the identity (eq. blockdiag_jacobian with diagonal Jacobians), and the quasi adjoint
    solves its transpose (LAPACK, dense)."""
    M, N, T, alpha = 4, 2, 12, 0.3
    m = _vanilla(M, 46, w_std=0.6) if kind == "plrnn" else _shallow(M, 7, 47)
    x = _x(1, T, N, 48)
    p = 1.0 - O.forcing_weights(M, N, alpha)
    z_init = O.teacher_states(x, M)[:, 1:]
    res = O.newton(m, x, alpha, N, fixed_iters=1, quasi=True)
    r, _, mask, _ = O.residual_and_masks(m, x, z_init, alpha, N)
    D = _diag_blocks(O.jacobian_diagonal(m, mask[0]) * p)
    assert np.allclose(res["z"][0] - z_init[0], brute.block_bidiagonal_solve(D, -r[0]), rtol=1e-12, atol=1e-14)
    z = O.rollout(m, x, alpha, N)
    _, _, mask, _ = O.residual_and_masks(m, x, z, alpha, N)
    D = _diag_blocks(O.jacobian_diagonal(m, mask[0]) * p)
    lam = O.adjoint(m, x, z, alpha, N, quasi=True)[0]
    assert np.allclose(lam, brute.block_bidiagonal_adjoint_solve(D, O.mse_seed(z, x)[0]), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("kind,M,N,alpha", [("plrnn", 4, 3, 0.2), ("plrnn", 16, 3, 0.2), ("shplrnn", 5, 3, 0.15)])
def test_quasi_converges_to_rollout_with_prefix_exactness(kind, M, N, alpha):
    """The quasi step keeps the zero of the residual, so a converged quasi-DEER iterate is the
    rollout; and with Delta_0 = 0 its first k steps are exact after k updates, like DEER's."""
    m = _vanilla(M, 49, w_std=0.2) if kind == "plrnn" else _shallow(M, 3 * M, 50)
    x = _x(2, 50, N, 51)
    ref = O.rollout(m, x, alpha, N)
    res = O.newton(m, x, alpha, N, tol=1e-13, max_iter=500, quasi=True)
    assert res["status"] == "ok"
    assert np.abs(res["z"] - ref).max() <= 1e-11
    T = 12
    xs = x[:, :T + 1]
    refs = O.rollout(m, xs, alpha, N)
    hist = O.newton(m, xs, alpha, N, fixed_iters=T, history=True, quasi=True)["history"]
    for k in range(1, T + 1):
        assert np.abs(hist[k][:, :k] - refs[:, :k]).max() < 1e-12, k



# ------------------------------------------------------------------------------------
# latent warm-up (Alg. GTF-DEER: P_1 for t <= T_w; the warm-up states left out of the loss)
# ------------------------------------------------------------------------------------

def test_warmup_prefix_is_driven_by_the_data():
    """With every latent observed, the warm-up inputs are the data themselves: z_1 = F(z_0),
    z_t = F(x_{t-1}) for t = 2..T_w + 1; afterwards the forcing is alpha again."""
    M = N = 4
    m = _vanilla(M, 61)
    x = _x(2, 30, N, 62)
    T_w = 10
    z = O.rollout(m, x, 0.3, N, T_w=T_w)
    m64 = {k: (v if k == "kind" else np.asarray(v, np.float64)) for k, v in m.items()}
    assert np.allclose(z[:, 1:T_w + 1], O.model_map(m64, np.asarray(x[:, 1:T_w + 1], np.float64)), atol=1e-13)
    assert not np.allclose(z[:, T_w + 1], O.model_map(m64, np.asarray(x[:, T_w + 1], np.float64)))
    assert np.allclose(O.rollout(m, x, 0.3, N, T_w=0), O.rollout(m, x, 0.3, N))


@pytest.mark.parametrize("kind,M,N,alpha,T_w", [("plrnn", 4, 3, 0.2, 7), ("plrnn", 16, 3, 0.2, 25),
                                                ("shplrnn", 5, 3, 0.15, 12)])
def test_warmup_newton_reaches_rollout(kind, M, N, alpha, T_w):
    m = _vanilla(M, 63) if kind == "plrnn" else _shallow(M, 3 * M, 64)
    x = _x(2, 60, N, 65)
    ref = O.rollout(m, x, alpha, N, T_w=T_w)
    res = O.newton(m, x, alpha, N, tol=1e-13, max_iter=200, T_w=T_w)
    assert res["status"] == "ok"
    assert np.abs(res["z"] - ref).max() <= 1e-11
    q = O.newton(m, x, alpha, N, tol=1e-13, max_iter=500, T_w=T_w, quasi=True)
    assert np.abs(q["z"] - ref).max() <= 1e-11


@pytest.mark.parametrize("kind,M,N,alpha,T_w", [("plrnn", 5, 3, 0.2, 6), ("shplrnn", 4, 4, 0.15, 9)])
def test_warmup_gradient_equals_bptt(kind, M, N, alpha, T_w):
    """IFT gradient with the warm-up (full forcing, warm-up states out of the loss) equals
    reverse-mode AD through the sequential rollout."""
    m = _vanilla(M, 66) if kind == "plrnn" else _shallow(M, 7, 67)
    x = _x(2, 25, N, 68)
    z = O.rollout(m, x, alpha, N, T_w=T_w)
    lam = O.adjoint(m, x, z, alpha, N, T_w=T_w)
    gr = O.param_grads(m, x, z, alpha, N, lam, T_w=T_w)
    loss, ref = _torch_bptt(m, x, alpha, N, T_w=T_w)
    assert abs(O.mse_loss(z, x, T_w=T_w) - loss) <= 1e-12 * max(1.0, abs(loss))
    for k, v in ref.items():
        assert np.allclose(gr[k], v, rtol=1e-9, atol=1e-12), k


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
def test_warmup_as_two_chained_solves(kind):
    """The warm-up part and the rest can be solved one after the other: the prefix with
    alpha = 1, the rest from z_0 := P_1 z_{T_w} + zbar_{T_w}; the adjoint of the rest (MSE seed
    over its own steps) hands J~_{T_w+1}^T lam_{T_w+1} to the prefix as its only cotangent, and
    the parameter gradients add."""
    M, N, alpha, T, T_w = 4, 2, 0.25, 40, 11
    m = _vanilla(M, 69) if kind == "plrnn" else _shallow(M, 6, 70)
    x = _x(2, T, N, 71)
    z = O.rollout(m, x, alpha, N, T_w=T_w)
    x1, x2 = x[:, :T_w + 1], x[:, T_w:]
    z1 = O.rollout(m, x1, 1.0, N)
    zb = np.concatenate([np.asarray(x[:, T_w], np.float64), z1[:, -1, N:]], axis=1)
    z2 = O.rollout(m, x2, alpha, N, z0=zb)
    assert np.allclose(np.concatenate([z1, z2], axis=1), z, atol=1e-13)
    lam = O.adjoint(m, x, z, alpha, N, T_w=T_w)
    gr = O.param_grads(m, x, z, alpha, N, lam, T_w=T_w)
    lam2 = O.adjoint(m, x2, z2, alpha, N, z0=zb)
    # J~_{T_w+1} at the fully forced input zb: P_1 J_F(zb)^T lam2[:, 0]
    m64 = {k: (v if k == "kind" else np.asarray(v, np.float64)) for k, v in m.items()}
    p1 = 1.0 - O.forcing_weights(M, N, 1.0)
    gb = p1 * O.vjp(m64, O.activation_mask(m64, zb), lam2[:, 0])
    g1 = np.zeros_like(z1)
    g1[:, -1] = gb
    lam1 = O.adjoint(m, x1, z1, 1.0, N, g=g1)
    assert np.allclose(np.concatenate([lam1, lam2], axis=1), lam, rtol=1e-12, atol=1e-15)
    g_a = O.param_grads(m, x1, z1, 1.0, N, lam1)
    g_b = O.param_grads(m, x2, z2, alpha, N, lam2, z0=zb)
    for k in gr:
        assert np.allclose(g_a[k] + g_b[k], gr[k], rtol=1e-11, atol=1e-14), k


# ------------------------------------------------------------------------------------
# training step: MAR penalty (eq. mar_loss_latent_initscale) and the Adam update
# ------------------------------------------------------------------------------------

@pytest.mark.parametrize("kind,p", [("plrnn", 1), ("plrnn", 2), ("shplrnn", 1), ("shplrnn", 2)])
def test_mar_penalty_matches_autograd(kind, p):
    M, M_r = 6, 3
    m = _vanilla(M, 81) if kind == "plrnn" else _shallow(M, 5, 82)
    lam_mar, gw, gv = 0.7, 0.3, 0.2
    loss, gr = O.mar_loss_and_grads(m, M_r, lam_mar, p, gw, gv)
    P = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in m.items() if k != "kind"}
    W = P["W"] if kind == "plrnn" else P["W1"]
    h = P["h"] if kind == "plrnn" else P["h1"]
    L = W.shape[1]
    tl = (torch.abs(1 - P["A"][M - M_r:]) ** p).sum() + (torch.abs(h[M - M_r:]) ** p).sum() \
        + gw / L * (torch.abs(W[M - M_r:]) ** p).sum()
    if kind == "shplrnn":
        tl = tl + gv / L * (torch.abs(P["W2"][:, M - M_r:]) ** p).sum()
    tl = lam_mar / M_r * tl
    tl.backward()
    assert abs(loss - float(tl)) < 1e-13
    for k, v in P.items():
        ref = v.grad.numpy() if v.grad is not None else np.zeros(v.shape)
        assert np.allclose(gr[k], ref, rtol=1e-12, atol=1e-15), k


def test_adam_matches_torch_adam():
    rng = np.random.default_rng(83)
    params = {"a": rng.standard_normal(7), "b": rng.standard_normal((3, 4))}
    tp = {k: torch.tensor(v.copy(), requires_grad=True) for k, v in params.items()}
    opt = torch.optim.Adam(list(tp.values()), lr=1e-2, betas=(0.9, 0.99), eps=1e-6)
    state = {}
    for step in range(1, 4):
        grads = {k: rng.standard_normal(v.shape) for k, v in params.items()}
        params, state = O.adam_update(params, grads, state, step, 1e-2, 0.9, 0.99, 1e-6)
        opt.zero_grad()
        for k, v in tp.items():
            v.grad = torch.tensor(grads[k])
        opt.step()
        for k in params:
            assert np.allclose(params[k], tp[k].detach().numpy(), rtol=1e-12, atol=1e-14), (step, k)


def _mar_base(kind, M, L):
    """A model whose MAR penalty is zero term by term: A = 1, every weight and bias 0."""
    if kind == "plrnn":
        return {"kind": "plrnn", "A": np.ones(M, np.float32), "W": np.zeros((M, M), np.float32),
                "h": np.zeros(M, np.float32)}
    return {"kind": "shplrnn", "A": np.ones(M, np.float32), "W1": np.zeros((M, L), np.float32),
            "W2": np.zeros((L, M), np.float32), "h1": np.zeros(M, np.float32), "h2": np.zeros(L, np.float32)}


@pytest.mark.parametrize("p", [1, 2])
@pytest.mark.parametrize("kind,M,L", [("plrnn", 7, 7), ("shplrnn", 5, 9)])
def test_mar_penalty_closed_forms(kind, M, L, p):
    """eq. mar_loss_latent_initscale term by term, on models with a single non-zero entry:
    lambda/M_r [ |1 - A_ii|^p + (1/L) sum_j (gamma_W |W_ij|^p + gamma_V |V_ji|^p) + |h_i|^p ]
    summed over the last M_r latents i only.  The sum runs over the rows of W (M x L) and the
    columns of V (L x M) that belong to a MAR latent; L is the hidden width (M for the vanilla
    PLRNN, which has no V).  Every closed form below is written from the equation, not from the
    oracle; a row/column swap of V, a 1/M instead of 1/L, or a wrong latent range fails one."""
    M_r, lam, gw, gv = 3, 0.7, 0.3, 0.2
    mar = list(range(M - M_r, M))
    free = list(range(M - M_r))
    c = lam / M_r
    wkey, hkey = ("W", "h") if kind == "plrnn" else ("W1", "h1")

    def val(m):
        return O.mar_loss_and_grads(m, M_r, lam, p, gw, gv)[0]

    assert val(_mar_base(kind, M, L)) == 0.0
    for i in mar + free:
        inside = i in mar
        m = _mar_base(kind, M, L)
        m["A"][i] = np.float32(0.25)            # |1 - A| = 0.75
        assert np.isclose(val(m), c * 0.75 ** p if inside else 0.0, rtol=1e-15, atol=0)
        m = _mar_base(kind, M, L)
        m[hkey][i] = np.float32(-1.5)
        assert np.isclose(val(m), c * 1.5 ** p if inside else 0.0, rtol=1e-15, atol=0)
        m = _mar_base(kind, M, L)
        m[wkey][i, L - 1] = np.float32(-2.0)    # W_ij: row i is the latent
        assert np.isclose(val(m), c * gw / L * 2.0 ** p if inside else 0.0, rtol=1e-15, atol=0)
    if kind == "shplrnn":
        for i in mar + free:
            m = _mar_base(kind, M, L)
            m["W2"][L - 2, i] = np.float32(1.25)  # V_ji: column i is the latent
            assert np.isclose(val(m), c * gv / L * 1.25 ** p if i in mar else 0.0, rtol=1e-15, atol=0)
        # V_ij instead of V_ji: a row index that equals a MAR latent index, in a free column
        m = _mar_base(kind, M, L)
        m["W2"][mar[0], free[0]] = np.float32(1.25)
        assert val(m) == 0.0
    # hidden biases h2 never enter the penalty
    if kind == "shplrnn":
        m = _mar_base(kind, M, L)
        m["h2"][:] = 3.0
        assert val(m) == 0.0
    # the terms add: all four at once in one MAR latent
    i = mar[-1]
    m = _mar_base(kind, M, L)
    m["A"][i], m[hkey][i], m[wkey][i, 0] = np.float32(0.5), np.float32(0.5), np.float32(0.5)
    ref = c * (0.5 ** p + 0.5 ** p + gw / L * 0.5 ** p)
    if kind == "shplrnn":
        m["W2"][0, i] = np.float32(0.5)
        ref += c * gv / L * 0.5 ** p
    assert np.isclose(val(m), ref, rtol=1e-15, atol=0)


# ------------------------------------------------------------------------------------
# general observation matrix (eqs. error_forcing, error_forcing_decomp; Alg. GTF-DEER)
# ------------------------------------------------------------------------------------

def _obs(N, M, seed, scale=1.0):
    return (np.random.default_rng(seed).standard_normal((N, M)) * scale / np.sqrt(M)).astype(np.float32)


def test_obs_projectors_closed_forms():
    """B = [I_N 0]: B^+ = B^T and P_alpha = diag(1 - a) (the identity read-out).  Dense B of full
    row rank: B^+ = B^T (B B^T)^-1, P_1 is the orthogonal projector onto the null space of B
    (P_1^2 = P_1 = P_1^T, B P_1 = 0) and P_alpha = P_1 + (1 - alpha) B^+ B; for M <= N with full
    column rank B^+ B = I, so P_alpha = (1 - alpha) I (plain GTF)."""
    M, N, alpha = 6, 3, 0.3
    Bi = np.zeros((N, M), np.float32)
    Bi[:, :N] = np.eye(N)
    Bp, Pa, P1 = O.obs_projectors(Bi, alpha)
    assert np.allclose(Bp, Bi.T, atol=1e-15)
    assert np.allclose(Pa, np.diag(1.0 - O.forcing_weights(M, N, alpha)), atol=1e-15)
    B = _obs(N, M, 5).astype(np.float64)
    Bp, Pa, P1 = O.obs_projectors(B, alpha)
    assert np.allclose(Bp, B.T @ np.linalg.inv(B @ B.T), atol=1e-12)
    assert np.allclose(P1 @ P1, P1, atol=1e-12) and np.allclose(P1, P1.T, atol=1e-12)
    assert np.allclose(B @ P1, 0.0, atol=1e-12)
    a = O.alpha_as_gpu(alpha)
    assert np.allclose(Pa, P1 + (1 - a) * (Bp @ B), atol=1e-12)
    Bt = _obs(5, 4, 6).astype(np.float64)              # M = 4 <= N = 5
    _, Pa2, _ = O.obs_projectors(Bt, alpha)
    assert np.allclose(Pa2, (1 - a) * np.eye(4), atol=1e-12)


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
@pytest.mark.parametrize("T_w", [0, 9])
def test_obs_functions_reduce_to_the_identity_readout(kind, T_w):
    """With B = [I_N 0] every general-B function equals its identity-read-out counterpart,
    which is pinned independently above."""
    M, N, alpha, T = 5, 2, 0.25, 30
    m = _vanilla(M, 91) if kind == "plrnn" else _shallow(M, 7, 92)
    x = _x(2, T, N, 93)
    Bi = np.zeros((N, M), np.float32)
    Bi[:, :N] = np.eye(N)
    z = O.rollout(m, x, alpha, N, T_w=T_w)
    assert np.allclose(O.rollout_obs(m, x, Bi, alpha, T_w=T_w), z, rtol=1e-13, atol=1e-14)
    assert np.allclose(O.mse_seed_obs(z, x, Bi, T_w), O.mse_seed(z, x, T_w), atol=1e-15)
    assert abs(O.mse_loss_obs(z, x, Bi, T_w) - O.mse_loss(z, x, T_w)) < 1e-14
    lam = O.adjoint(m, x, z, alpha, N, T_w=T_w)
    assert np.allclose(O.adjoint_obs(m, x, z, Bi, alpha, T_w=T_w), lam, rtol=1e-12, atol=1e-15)
    g1 = O.param_grads(m, x, z, alpha, N, lam, T_w=T_w)
    g2 = O.param_grads_obs(m, x, z, Bi, alpha, lam, T_w=T_w)
    for k in g1:
        assert np.allclose(g1[k], g2[k], rtol=1e-12, atol=1e-15), k


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
@pytest.mark.parametrize("T_w", [0, 7])
def test_obs_newton_converges_to_the_rollout_with_prefix_exactness(kind, T_w):
    """Dense B (N < M): the Newton iterate reaches the sequential rollout (the unique zero of the
    residual), and after k updates its first k states are exact (Delta_0 = 0 and the
    block-bidiagonal structure of the forced Jacobians)."""
    M, N, alpha, T = 5, 2, 0.3, 16
    m = _vanilla(M, 94, w_std=0.25) if kind == "plrnn" else _shallow(M, 6, 95)
    x = _x(2, T, N, 96)
    B = _obs(N, M, 97)
    ref = O.rollout_obs(m, x, B, alpha, T_w=T_w)
    out = O.newton_obs(m, x, B, alpha, tol=1e-13, max_iter=T + 2, T_w=T_w, history=True)
    assert out["status"] == "ok"
    assert np.abs(out["z"] - ref).max() <= 1e-11 * max(1.0, np.abs(ref).max())
    for k, zk in enumerate(out["history"][:T + 1]):
        assert np.allclose(zk[:, :k], ref[:, :k], rtol=1e-10, atol=1e-11), k


def _torch_rollout_obs(m, x, B, alpha, T_w, z0):
    """The forward model of Alg. GTF-DEER in torch (float64), B a leaf tensor: pinv, forced
    inputs z~ = z + a_k B^+ (x_k - B z), F, and the loss over t > T_w."""
    Bp = torch.linalg.pinv(B)
    X = torch.tensor(np.asarray(x, np.float64))
    Bn, T1, _ = X.shape
    T = T1 - 1
    a = float(np.float32(alpha))
    zprev = X[:, 0] @ Bp.T if z0 is None else torch.tensor(np.asarray(z0, np.float64))
    zs = []
    for t in range(1, T + 1):
        k = t - 1
        if k == 0:
            zt = zprev
        else:
            ak = 1.0 if k <= T_w else a
            zt = zprev + ak * ((X[:, k] - zprev @ B.T) @ Bp.T)
        if m["kind"] == "plrnn":
            zprev = m["A"] * zt + torch.relu(zt) @ m["W"].T + m["h"]
        else:
            zprev = m["A"] * zt + torch.relu(zt @ m["W2"].T + m["h2"]) @ m["W1"].T + m["h1"]
        zs.append(zprev)
    Z = torch.stack(zs, dim=1)
    N = B.shape[0]
    loss = ((Z[:, T_w:] @ B.T - X[:, 1 + T_w:]) ** 2).sum() / (Bn * N * (T - T_w))
    return loss


@pytest.mark.parametrize("kind", ["plrnn", "shplrnn"])
@pytest.mark.parametrize("T_w,given_z0,M,N", [(0, False, 5, 2), (5, False, 5, 2), (0, True, 5, 2), (0, False, 3, 5),
                                              (4, False, 3, 5)])
def test_obs_gradients_match_autograd_through_the_rollout(kind, T_w, given_z0, M, N):
    """The IFT gradients (adjoint recursion, parameter sums and dL/dB from the differential of
    the pseudo-inverse) equal reverse-mode AD through the sequential rollout with B as a
    parameter (torch.linalg.pinv differentiated by torch), at the rollout's fixed point.  Wide B
    (N < M) and tall B (N > M, where B^+ B = I and the (I - B B^+) terms of the differential
    are the ones that do not vanish)."""
    alpha, T = 0.3, 24
    m = _vanilla(M, 98, w_std=0.25) if kind == "plrnn" else _shallow(M, 6, 99)
    x = _x(2, T, N, 100)
    B = _obs(N, M, 101).astype(np.float64)
    z0 = np.random.default_rng(102).standard_normal((2, M)) if given_z0 else None
    z = O.rollout_obs(m, x, B, alpha, z0=z0, T_w=T_w)
    lam = O.adjoint_obs(m, x, z, B, alpha, z0=z0, T_w=T_w)
    gr = O.param_grads_obs(m, x, z, B, alpha, lam, z0=z0, T_w=T_w)
    gB = O.obs_grad(m, x, z, B, alpha, lam, z0=z0, T_w=T_w)
    P = {k: torch.tensor(np.asarray(v, np.float64), requires_grad=True) for k, v in m.items() if k != "kind"}
    Bt = torch.tensor(B, requires_grad=True)
    loss = _torch_rollout_obs({"kind": kind, **P}, x, Bt, alpha, T_w, z0)
    assert abs(float(loss) - O.mse_loss_obs(z, x, B, T_w)) < 1e-13
    loss.backward()
    for k, v in P.items():
        assert np.allclose(gr[k], v.grad.numpy(), rtol=1e-9, atol=1e-12), k
    assert np.allclose(gB, Bt.grad.numpy(), rtol=1e-9, atol=1e-12)


def test_obs_gradient_matches_central_differences():
    """dL/dB against central differences of the loss of the rollout (float64, step 1e-6), away
    from ReLU kinks; a second pin that does not use torch's pinv derivative."""
    M, N, alpha, T = 4, 2, 0.35, 20
    m = _vanilla(M, 103, w_std=0.25)
    x = _x(1, T, N, 104)
    B = _obs(N, M, 105).astype(np.float64)
    z = O.rollout_obs(m, x, B, alpha)
    lam = O.adjoint_obs(m, x, z, B, alpha)
    gB = O.obs_grad(m, x, z, B, alpha, lam)
    eps = 1e-6
    fd = np.zeros_like(B)
    for n in range(N):
        for j in range(M):
            Bp_, Bm_ = B.copy(), B.copy()
            Bp_[n, j] += eps
            Bm_[n, j] -= eps
            lp = O.mse_loss_obs(O.rollout_obs(m, x, Bp_, alpha), x, Bp_)
            lm = O.mse_loss_obs(O.rollout_obs(m, x, Bm_, alpha), x, Bm_)
            fd[n, j] = (lp - lm) / (2 * eps)
    assert np.allclose(gB, fd, rtol=1e-6, atol=1e-9)
