"""Quasi-DEER (every forced Jacobian replaced by its diagonal; vanilla PLRNN) on the GPU
against the float64 oracle, through the C ABI.

Tolerance 1e-4 normwise relative for float32 states, adjoints and gradients.  Newton
iterates are compared where the ReLU decisions of both sides cannot differ: the first update
from the teacher states, and one update from an iterate given to both; converged solves are
compared with the sequential rollout (the zero of the residual, independent of the path)."""
import os

import numpy as np
import pytest

import oracle as O
import workloads as W
from gpu_util import oracle_model, rel_inf, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402

TOL = 1e-4
SIZES = [(1, 1, 1, 1), (3, 3, 1, 5), (16, 3, 2, 1000), (17, 5, 3, 333), (24, 24, 1, 4099), (33, 8, 2, 700),
         (64, 64, 2, 2050)]


def _case(M, N, B, T, alpha, seed):
    return W.random_plrnn_case(M, N, B, T, alpha, seed, w_norm=0.2, a_range=(0.3, 0.75))


@pytest.mark.parametrize("M,N,B,T", SIZES)
def test_quasi_first_update(M, N, B, T):
    c = _case(M, N, B, T, 0.2, 300 + M + T)
    m = oracle_model(c)
    say("deer_solve_quasi first update", M, N, B, T)
    res = D.deer_solve_quasi(m, c.x, c.alpha, N, fixed_iters=1)
    ref = O.newton(m, c.x, c.alpha, N, fixed_iters=1, quasi=True)
    assert rel_inf(res["z"].cpu().numpy(), ref["z"]) < TOL


@pytest.mark.parametrize("M,N,B,T", SIZES[2:])
def test_quasi_update_from_a_given_iterate(M, N, B, T):
    c = _case(M, N, B, T, 0.2, 310 + M + T)
    m = oracle_model(c)
    say("deer_solve_quasi three updates", M, N, B, T)
    z3 = D.deer_solve_quasi(m, c.x, c.alpha, N, fixed_iters=3)["z"]
    zin = z3.cpu().numpy()
    say("deer_solve_quasi one update from z3", M, N, B, T)
    res = D.deer_solve_quasi(m, c.x, c.alpha, N, fixed_iters=1, init="user", z=z3)
    ref = O.newton(m, c.x, c.alpha, N, fixed_iters=1, init="user", z_init=zin, quasi=True)
    assert rel_inf(res["z"].cpu().numpy(), ref["z"]) < TOL


@pytest.mark.parametrize("M,N,B,T,alpha", [(3, 3, 1, 300, 0.1), (16, 3, 2, 1000, 0.2), (8, 2, 3, 2049, 0.2),
                                           (64, 64, 2, 600, 0.05)])
def test_quasi_solve_converges_to_rollout(M, N, B, T, alpha):
    c = _case(M, N, B, T, alpha, 320 + M)
    m = oracle_model(c)
    say("deer_solve_quasi to tolerance", M, N, B, T)
    res = D.deer_solve_quasi(m, c.x, alpha, N, tol=1e-5, max_iter=2000)
    assert res["status"] == 0
    ref = O.rollout(m, c.x, alpha, N)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    full = D.deer_solve(m, c.x, alpha, N, tol=1e-5)
    print(f"[gpu-case] quasi updates {res['iters']} vs full-Jacobian updates {full['iters']}", flush=True)
    assert min(res["iters"]) >= min(full["iters"])


def test_quasi_safeguard_lands_on_rollout():
    """A small step bound rejects updates and damps d (gamma d); the fixed point is unchanged."""
    M, N, B, T = 16, 3, 2, 500
    c = _case(M, N, B, T, 0.2, 330)
    m = oracle_model(c)
    say("deer_solve_quasi with rejections")
    res = D.deer_solve_quasi(m, c.x, c.alpha, N, tol=1e-5, max_iter=3000, step_bound=0.05)
    assert res["status"] == 0
    assert rel_inf(res["z"].cpu().numpy(), O.rollout(m, c.x, c.alpha, N)) < TOL


@pytest.mark.parametrize("M,N,B,T", SIZES)
@pytest.mark.parametrize("user_g", [False, True])
def test_quasi_adjoint_and_gradients(M, N, B, T, user_g):
    c = _case(M, N, B, T, 0.2, 340 + M + T)
    m = oracle_model(c)
    z32 = O.rollout(m, c.x, c.alpha, N).astype(np.float32)
    g = np.random.default_rng(M + T).standard_normal((B, T, M)).astype(np.float32) if user_g else None
    say("deer_adjoint_quasi", M, N, B, T, user_g)
    out = D.deer_adjoint_quasi(m, c.x, z32, c.alpha, N, g=g)
    lam = O.adjoint(m, c.x, z32, c.alpha, N, g=g, mask_precision="float32", quasi=True)
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    gr = O.param_grads(m, c.x, z32, c.alpha, N, lam, mask_precision="float32")
    for k, v in out["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k
    out2 = D.deer_adjoint_quasi(m, c.x, z32, c.alpha, N, g=g, want_lam=False)
    for k, v in out2["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k


@pytest.mark.parametrize("M,N,B,T,alpha,T_w,bound", [(16, 3, 4, 4096, 0.2, 0, 0.0), (8, 2, 3, 2049, 0.2, 0, 0.0),
                                                     (24, 24, 2, 1500, 0.1, 300, 0.0), (33, 8, 2, 700, 0.2, 0, 0.05),
                                                     (64, 64, 2, 2050, 0.05, 0, 0.0), (3, 3, 1, 5, 0.1, 0, 0.0),
                                                     (16, 3, 2, 500, 0.2, 100, 0.05), (50, 7, 5, 333, 0.2, 40, 0.0),
                                                     (1, 1, 1, 1, 0.2, 0, 0.0), (4, 2, 3, 2, 0.2, 1, 0.0)])
def test_quasi_fused_and_separate_passes_agree(M, N, B, T, alpha, T_w, bound):
    """The adaptive loop's quasi-DEER pass in one kernel (fix-up of an update, chunk aggregates
    of the next, pass-end control; chunk counts padded to whole groups) and in separate kernels
    (DEER_QUASI_FUSED=0): both land on the rollout, in the oracle's number of quasi-Newton
    updates up to one; ragged and padding chunks, several groups per sequence, all three lane
    widths, latent warm-up and forced rejections (damped coefficients)."""
    c = _case(M, N, B, T, alpha, 360 + M + T)
    m = oracle_model(c)
    ref = O.rollout(m, c.x, alpha, N, T_w=T_w)
    want = None
    if bound == 0.0:
        want = O.newton(m, c.x, alpha, N, tol=1e-5, max_iter=T + 2, T_w=T_w, quasi=True)["iters"].tolist()
    its = {}
    try:
        for fuse in ("1", "0"):
            os.environ["DEER_QUASI_FUSED"] = fuse
            say("deer_solve_quasi fused" if fuse == "1" else "deer_solve_quasi separate", M, N, B, T, alpha, T_w, bound)
            res = D.deer_solve_quasi(m, c.x, alpha, N, tol=1e-5, max_iter=T + 2, step_bound=bound, T_w=T_w)
            assert res["status"] == 0, (fuse, res)
            assert rel_inf(res["z"].cpu().numpy(), ref) < TOL, fuse
            assert all(n < 1e-5 for n in res["norms"]), fuse
            its[fuse] = res["iters"]
    finally:
        os.environ.pop("DEER_QUASI_FUSED", None)
    print(f"[gpu-case] quasi updates fused {its['1']} separate {its['0']} oracle {want}", flush=True)
    assert max(abs(a - b) for a, b in zip(its["1"], its["0"])) <= 1
    if want is not None:
        assert max(abs(a - b) for a, b in zip(its["1"], want)) <= 1, (its["1"], want)


@pytest.mark.parametrize("fuse", ["1", "0"])
def test_quasi_nonfinite_and_not_converged(fuse):
    """A NaN input ends its sequence as non-finite after the damped retries, and an update cap
    of one leaves every sequence unconverged after one update, in the one-kernel pass and in
    the separate kernels."""
    c = _case(8, 3, 2, 200, 0.2, 17)
    m = oracle_model(c)
    x = c.x.copy()
    x[1, 50, 0] = np.nan
    try:
        os.environ["DEER_QUASI_FUSED"] = fuse
        say("deer_solve_quasi NaN input", fuse)
        res = D.deer_solve_quasi(m, x, 0.2, 3, tol=1e-5, check=False)
        assert res["status"] == 3                      # DEER_ERR_NONFINITE
        say("deer_solve_quasi max_iter=1", fuse)
        res = D.deer_solve_quasi(m, c.x, 0.2, 3, tol=1e-5, max_iter=1, check=False)
        assert res["status"] == 2                      # DEER_ERR_NOT_CONVERGED
        assert res["iters"] == [1, 1]
    finally:
        os.environ.pop("DEER_QUASI_FUSED", None)


def test_quasi_workload2_full_size():
    """The M = 16 workload (16 Lorenz-63 sequences of 16384 steps, alpha = 0.2, tolerance
    1e-5) with quasi-DEER: the solve lands on the rollout and the adjoint and gradients at
    that trajectory match the oracle's quasi recursion.  Quasi-DEER needs thousands of
    updates here (one more leading step is exact per update, so at most T + 1)."""
    c = W.make_config(2)
    m = oracle_model(c)
    say("deer_solve_quasi workload 2")
    res = D.deer_solve_quasi(m, c.x, c.alpha, c.n_obs, tol=c.tol, max_iter=c.T + 2)
    assert res["status"] == 0
    print(f"[gpu-case] quasi updates per sequence: {res['iters']}", flush=True)
    ref = O.rollout(m, c.x, c.alpha, c.n_obs)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    z32 = ref.astype(np.float32)
    say("deer_adjoint_quasi workload 2")
    out = D.deer_adjoint_quasi(m, c.x, z32, c.alpha, c.n_obs)
    lam = O.adjoint(m, c.x, z32, c.alpha, c.n_obs, mask_precision="float32", quasi=True)
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    gr = O.param_grads(m, c.x, z32, c.alpha, c.n_obs, lam, mask_precision="float32")
    for k, v in out["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k


# ---- shallow PLRNN (the model of the paper's quasi-DEER ablation: M = 5, L = 50) ----------

SH_SIZES = [(5, 50, 3, 1, 300), (3, 7, 3, 2, 129), (8, 32, 2, 2, 700), (32, 256, 32, 1, 1024)]


def _sh_case(M, L, N, B, T, alpha, seed):
    return W.random_shplrnn_case(M, L, N, B, T, alpha, seed, w_norm=0.2, a_range=(0.3, 0.75))


@pytest.mark.parametrize("M,L,N,B,T", SH_SIZES)
def test_quasi_shallow_first_update_and_rollout(M, L, N, B, T):
    c = _sh_case(M, L, N, B, T, 0.15, 400 + M + L)
    m = oracle_model(c)
    say("deer_solve_quasi shallow first update", M, L, N, B, T)
    res = D.deer_solve_quasi(m, c.x, c.alpha, N, fixed_iters=1)
    ref = O.newton(m, c.x, c.alpha, N, fixed_iters=1, quasi=True)
    assert rel_inf(res["z"].cpu().numpy(), ref["z"]) < TOL
    say("deer_solve_quasi shallow to tolerance", M, L, N, B, T)
    res = D.deer_solve_quasi(m, c.x, c.alpha, N, tol=1e-5, max_iter=T + 2)
    assert res["status"] == 0
    assert rel_inf(res["z"].cpu().numpy(), O.rollout(m, c.x, c.alpha, N)) < TOL
    print(f"[gpu-case] shallow quasi updates {res['iters']}", flush=True)


@pytest.mark.parametrize("M,L,N,B,T", SH_SIZES)
@pytest.mark.parametrize("user_g", [False, True])
def test_quasi_shallow_adjoint_and_gradients(M, L, N, B, T, user_g):
    c = _sh_case(M, L, N, B, T, 0.15, 410 + M + L)
    m = oracle_model(c)
    z32 = O.rollout(m, c.x, c.alpha, N).astype(np.float32)
    g = np.random.default_rng(M + L).standard_normal((B, T, M)).astype(np.float32) if user_g else None
    say("deer_adjoint_quasi shallow", M, L, N, B, T, user_g)
    out = D.deer_adjoint_quasi(m, c.x, z32, c.alpha, N, g=g)
    lam = O.adjoint(m, c.x, z32, c.alpha, N, g=g, mask_precision="float32", quasi=True)
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    gr = O.param_grads(m, c.x, z32, c.alpha, N, lam, mask_precision="float32")
    for k, v in out["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k
    out2 = D.deer_adjoint_quasi(m, c.x, z32, c.alpha, N, g=g, want_lam=False)
    for k, v in out2["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k
