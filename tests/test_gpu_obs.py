"""General observation matrix B (dense P_alpha = I - alpha B^+ B, forcing targets B^+ x, joint
latent warm-up, dL/dB) on the GPU against the float64 oracle, through the C ABI.

The forced inputs involve a matrix-vector product, so the GPU's float32 ReLU decisions are not
reproducible bit for bit by a float64 oracle.  As for the shallow model's decisions: masks are
compared outside a tie band (|u| > 1e-5 max|u|; in-band differences are counted and printed);
solves are compared with the sequential rollout (F is continuous, so an in-band decision moves
the solution by O(band) only); adjoints and gradients with the oracle's recursion taken with
the GPU's own decisions at the same trajectory (plrnn_jacobian_ex returns the decisions of the
kernels the adjoint runs)."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from gpu_util import masks_to_bool, oracle_model, rel_inf, say, tie_band_check

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402
from paper_2605_12683_amd import _binding as Bnd  # noqa: E402

TOL = 1e-4
BAND = 1e-5


def _obs(N, M, seed):
    return (np.random.default_rng(seed).standard_normal((N, M)) / np.sqrt(M)).astype(np.float32)


def _case(kind, M, L, N, B, T, seed):
    """A contracting model and data of N observed dimensions."""
    if kind == "plrnn":
        c = W.random_plrnn_case(M, min(N, M), B, T, 0.2, seed, w_norm=0.3, a_range=(0.3, 0.6))
    else:
        c = W.random_shplrnn_case(M, L, min(N, M), B, T, 0.2, seed, w_norm=0.3, a_range=(0.3, 0.6))
    x = np.random.default_rng(seed + 7).standard_normal((B, T + 1, N)).astype(np.float32)
    return oracle_model(c), x


def _no_ties(m, zt):
    u = O.preactivation(m, zt)
    au = np.abs(u)
    if au.size and au.min() <= BAND * au.max():
        pytest.fail(f"a ReLU decision lies in the tie band (min |u| = {au.min():.3g}); choose another seed")


def _masks_outside_band(gpu_mask, m, zt, what):
    """GPU decisions equal the float64 ones wherever |u| > BAND max|u|, and few differ inside."""
    return tie_band_check(gpu_mask, O.preactivation(m, zt), BAND, what)


CASES = [("plrnn", 5, 0, 2, 2, 60), ("plrnn", 16, 0, 3, 3, 700), ("plrnn", 33, 0, 7, 2, 300),
         ("plrnn", 64, 0, 16, 1, 400), ("plrnn", 3, 0, 5, 2, 80), ("shplrnn", 5, 12, 2, 2, 90),
         ("shplrnn", 32, 64, 8, 2, 500), ("shplrnn", 4, 20, 6, 1, 64)]


@pytest.mark.parametrize("kind,M,L,N,B,T", CASES)
@pytest.mark.parametrize("T_w", [0, 1, 17])
def test_obs_solve_matches_rollout(kind, M, L, N, B, T, T_w):
    m, x = _case(kind, M, L, N, B, T, 300 + M + N + T_w)
    Bm = _obs(N, M, 400 + M)
    ref = O.rollout_obs(m, x, Bm, 0.2, T_w=T_w)
    say("deer_solve obs", kind, M, L, N, B, T, T_w)
    res = D.deer_solve(m, x, 0.2, N, tol=1e-6, obs=Bm, T_w=T_w, want_masks=True)
    assert res["status"] == Bnd.DEER_OK
    z = res["z"].cpu().numpy()
    assert rel_inf(z, ref) < TOL
    mk = masks_to_bool(res["masks"].cpu().numpy(), L if kind == "shplrnn" else M)
    zt = O.obs_forced_states(z.astype(np.float64), x, Bm, 0.2, T_w=T_w)
    _masks_outside_band(mk, m, zt, "solve masks")


@pytest.mark.parametrize("kind,M,L,N", [("plrnn", 6, 0, 3), ("shplrnn", 5, 16, 2)])
@pytest.mark.parametrize("k", [1, 3])
def test_obs_fixed_updates_match_newton_iterates(kind, M, L, N, k):
    """A fixed number of updates from the teacher states B^+ x equals the oracle's k-th iterate."""
    m, x = _case(kind, M, L, N, 2, 200, 500 + M)
    Bm = _obs(N, M, 501)
    ref = O.newton_obs(m, x, Bm, 0.2, fixed_iters=k, history=True)
    for zk in ref["history"][:-1]:
        _no_ties(m, O.obs_forced_states(zk, x, Bm, 0.2))
    say("deer_solve obs fixed", kind, M, L, N, k)
    res = D.deer_solve(m, x, 0.2, N, fixed_iters=k, obs=Bm)
    assert rel_inf(res["z"].cpu().numpy(), ref["z"]) < TOL


def test_obs_identity_readout_equals_the_tuned_path():
    """B = [I_N 0] through the general path gives the solve and gradients of the identity
    read-out kernels."""
    c = W.random_plrnn_case(16, 3, 2, 500, 0.2, 600, w_norm=0.3, a_range=(0.3, 0.6))
    m = oracle_model(c)
    Bi = np.zeros((3, 16), np.float32)
    Bi[:, :3] = np.eye(3)
    say("deer_solve obs identity")
    a = D.deer_solve(m, c.x, 0.2, 3, tol=1e-6)
    b = D.deer_solve(m, c.x, 0.2, 3, tol=1e-6, obs=Bi)
    assert rel_inf(b["z"].cpu().numpy(), a["z"].cpu().numpy()) < TOL
    z32 = O.rollout(m, c.x, 0.2, 3).astype(np.float32)
    ga = D.deer_adjoint(m, c.x, z32, 0.2, 3)
    gb = D.deer_adjoint(m, c.x, z32, 0.2, 3, obs=Bi)
    assert rel_inf(gb["lam"].cpu().numpy(), ga["lam"].cpu().numpy()) < TOL
    for k in ("A", "W", "h"):
        assert rel_inf(gb["grads"][k].cpu().numpy(), ga["grads"][k].cpu().numpy()) < TOL, k


@pytest.mark.parametrize("kind,M,L,N,B,T", CASES)
@pytest.mark.parametrize("T_w,given", [(0, False), (11, False), (0, True)])
def test_obs_adjoint_and_gradients(kind, M, L, N, B, T, T_w, given):
    """lam, the parameter gradients and dL/dB at the fixed point, with the MSE seed (dL/dB then
    includes the MSE's direct term) or with a given cotangent and initial state."""
    m, x = _case(kind, M, L, N, B, T, 700 + M + N + T_w)
    Bm = _obs(N, M, 800 + M)
    rng = np.random.default_rng(900 + M)
    z0 = rng.standard_normal((B, M)).astype(np.float32) if given else None
    g = (rng.standard_normal((B, T, M)) * 1e-3).astype(np.float32) if given else None
    z32 = O.rollout_obs(m, x, Bm, 0.2, z0=z0, T_w=T_w).astype(np.float32)
    say("plrnn_jacobian obs", kind, M, L, N, B, T, T_w, given)
    jac = D.plrnn_jacobian(m, x, z32, 0.2, N, z0=z0, want=("F", "r", "masks"), obs=Bm, T_w=T_w)
    mk = masks_to_bool(jac["masks"].cpu().numpy(), L if kind == "shplrnn" else M)
    zt = O.obs_forced_states(z32, x, Bm, 0.2, z0=z0, T_w=T_w)
    _masks_outside_band(mk, m, zt, "adjoint masks")
    F = O.model_map(m, zt)
    assert rel_inf(jac["F"].cpu().numpy(), F) < TOL
    assert np.abs(jac["r"].cpu().numpy() - (z32 - F)).max() <= 1e-5 * max(1.0, np.abs(F).max())
    lam = O.adjoint_obs(m, x, z32, Bm, 0.2, z0=z0, g=g, T_w=T_w, mask=mk)
    gr = O.param_grads_obs(m, x, z32, Bm, 0.2, lam, z0=z0, T_w=T_w, mask=mk)
    gB = O.obs_grad(m, x, z32, Bm, 0.2, lam, z0=z0, T_w=T_w, mask=mk, with_mse=not given)
    say("deer_adjoint obs", kind, M, L, N, B, T, T_w, given)
    out = D.deer_adjoint(m, x, z32, 0.2, N, z0=z0, g=g, T_w=T_w, obs=Bm)
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    for k, v in gr.items():
        assert rel_inf(out["grads"][k].cpu().numpy(), v) < TOL, k
    assert rel_inf(out["grads"]["obs"].cpu().numpy(), gB) < TOL


def test_obs_rank_deficient_is_nonfinite():
    """A B without full row rank has no well-defined forcing here: the projectors are NaN and the
    solve reports a non-finite update."""
    m, x = _case("plrnn", 6, 0, 3, 1, 40, 950)
    Bm = _obs(3, 6, 951)
    Bm[2] = Bm[0]
    say("deer_solve obs rank-deficient")
    res = D.deer_solve(m, x, 0.2, 3, obs=Bm, check=False)
    assert res["status"] == Bnd.DEER_ERR_NONFINITE
