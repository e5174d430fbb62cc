"""Stored-Jacobian dense scan and the shallow PLRNN on the GPU against the float64 oracle."""
import os

import numpy as np
import pytest

import oracle as O
import workloads as W
from gpu_util import masks_to_bool, oracle_model, rel_inf, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402
from paper_2605_12683_amd import _binding as Bnd  # noqa: E402

TOL = 1e-4


@pytest.fixture(autouse=True)
def _no_chunk_override():
    os.environ.pop("DEER_CHUNK", None)
    yield
    os.environ.pop("DEER_CHUNK", None)


def _rand_scan(B, T, M, seed):
    rng = np.random.default_rng(seed)
    J = (rng.standard_normal((B, T, M, M)) * (0.9 / np.sqrt(M) / 2)).astype(np.float32)
    b = rng.standard_normal((B, T, M)).astype(np.float32)
    return J, b


@pytest.mark.parametrize("B,T,M,chunk", [(1, 1, 1, 0), (2, 2, 3, 0), (3, 100, 16, 0), (2, 1000, 20, 0),
                                         (1, 777, 32, 64), (2, 300, 64, 0), (2, 513, 5, 17), (1, 4000, 64, 0)])
@pytest.mark.parametrize("rev,tr", [(False, False), (True, True), (False, True), (True, False)])
def test_deer_scan_dense(B, T, M, chunk, rev, tr):
    """The bare scan in both directions with each step's matrix or its transpose,
    y_t = op(J_t) y_{t-1} + b_t or y_{t-1} = op(J_t) y_t + b_{t-1}, equals the sequential recurrence."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    J, b = _rand_scan(B, T, M, B * T + M)
    say("deer_scan dense", B, T, M, chunk, rev, tr)
    y = D.deer_scan(Bnd.DEER_SCAN_DENSE, torch.tensor(J), torch.tensor(b), reverse=rev, transpose=tr).cpu().numpy()
    Jd = J.astype(np.float64)
    # the oracle's reverse recursion applies J^T; hand it J^T to get J
    Jop = Jd if rev == tr else np.ascontiguousarray(np.swapaxes(Jd, -1, -2))
    if rev:
        ref = O.reverse_affine_recurrence(lambda k, w: np.einsum("bi,bij->bj", w, Jop[:, k]), b.astype(np.float64))
    else:
        ref = O.affine_recurrence(lambda k, v: np.einsum("bij,bj->bi", Jop[:, k], v), b.astype(np.float64))
    assert rel_inf(y, ref) < TOL


def test_dense_scan_transpose_identity():
    """<g, S b> = <S^T g, b> between the forward and the reverse GPU scans (any size)."""
    J, b = _rand_scan(4, 5000, 32, 9)
    g = np.random.default_rng(10).standard_normal(b.shape).astype(np.float32)
    say("deer_scan dense transpose identity")
    y = D.deer_scan(Bnd.DEER_SCAN_DENSE, torch.tensor(J), torch.tensor(b)).double()
    lt = D.deer_scan(Bnd.DEER_SCAN_DENSE, torch.tensor(J), torch.tensor(g), reverse=True).double()
    lhs = float((torch.tensor(g, device="cuda").double() * y).sum())
    rhs = float((lt * torch.tensor(b, device="cuda").double()).sum())
    assert abs(lhs - rhs) <= 1e-4 * max(abs(lhs), 1.0)


def _case(M, L, N, B, T, alpha, seed):
    return W.random_shplrnn_case(M, L, N, B, T, alpha, seed, w_norm=0.3, a_range=(0.3, 0.65))


@pytest.mark.parametrize("M,L,N,T", [(1, 7, 1, 40), (4, 12, 4, 100), (5, 20, 2, 64), (16, 64, 16, 130),
                                     (32, 256, 32, 70), (33, 100, 33, 50), (64, 128, 64, 40)])
def test_shallow_jacobian_masks_bitexact(M, L, N, T):
    c = _case(M, L, N, 2, T, 0.2, 500 + M)
    m = oracle_model(c)
    z = np.random.default_rng(2).standard_normal((2, T, M)).astype(np.float32)
    say("plrnn_jacobian shallow", M, L, N, T)
    out = D.plrnn_jacobian(m, c.x, z, c.alpha, N, want=("F", "r", "masks"), dense_J=True)
    ref = O.jacobian_at(m, c.x, z, c.alpha, N, mask_precision="float32",
                        dense_index=[(b, t) for b in range(2) for t in range(T)])
    got = masks_to_bool(out["masks"].cpu().numpy(), L)
    assert np.array_equal(got, ref["mask"])
    assert rel_inf(out["F"].cpu().numpy(), ref["F"]) < 1e-5
    assert rel_inf(out["r"].cpu().numpy(), ref["r"]) < 1e-5
    assert rel_inf(out["J"].cpu().numpy().reshape(-1, M, M), ref["J"]) < 1e-5


@pytest.mark.parametrize("M,L,N,B,T,alpha,chunk", [(4, 12, 4, 2, 300, 0.1, 0), (5, 20, 2, 2, 200, 0.3, 33),
                                                   (16, 64, 16, 2, 500, 0.1, 0), (32, 256, 32, 2, 400, 0.1, 0),
                                                   (20, 40, 5, 3, 300, 0.2, 64), (64, 128, 64, 1, 100, 0.1, 0),
                                                   (1, 7, 1, 2, 50, 0.2, 0)])
def test_shallow_solve_and_adjoint(M, L, N, B, T, alpha, chunk):
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    c = _case(M, L, N, B, T, alpha, 400 + M)
    m = oracle_model(c)
    say("deer_solve shallow", M, L, N, B, T, alpha, chunk)
    res = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=100)
    assert res["status"] == 0, res
    ref = O.rollout(m, c.x, alpha, N)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    z32 = ref.astype(np.float32)
    say("deer_adjoint shallow", M, L, N, B, T, alpha, chunk)
    out = D.deer_adjoint(m, c.x, z32, alpha, N)
    lam = O.adjoint(m, c.x, z32, alpha, N, mask_precision="float32")
    gr = O.param_grads(m, c.x, z32, alpha, N, lam, mask_precision="float32")
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    for k in ("A", "W1", "W2", "h1", "h2"):
        assert rel_inf(out["grads"][k].cpu().numpy(), gr[k]) < TOL, k


@pytest.mark.parametrize("path", ["fused", "fixed-order residual", "stored Jacobian"])
def test_shallow_nonfinite_and_not_converged(path):
    """A NaN input ends its sequence as non-finite after the damped retries, and an update cap of
    one leaves both sequences unconverged after one update: with the pass-end control in the
    Jacobian-vector fix-up (the default), with the fixed-order residual (k_seq_ctl), and on the
    stored-Jacobian path."""
    env = {"fused": {}, "fixed-order residual": {"DEER_SH_RESMFMA": "0"},
           "stored Jacobian": {"DEER_SH_FUSED": "0"}}[path]
    c = _case(6, 20, 3, 2, 300, 0.2, 23)
    m = oracle_model(c)
    x = c.x.copy()
    x[1, 70, 1] = np.nan
    try:
        os.environ.update(env)
        say("shallow NaN input", path)
        res = D.deer_solve(m, x, 0.2, 3, tol=1e-5, check=False)
        assert res["status"] == 3                      # DEER_ERR_NONFINITE
        say("shallow max_iter=1", path)
        res = D.deer_solve(m, c.x, 0.2, 3, tol=1e-5, max_iter=1, check=False)
        assert res["status"] == 2                      # DEER_ERR_NOT_CONVERGED
        assert res["iters"] == [1, 1]
        say("shallow to tolerance", path)
        res = D.deer_solve(m, c.x, 0.2, 3, tol=1e-5, max_iter=100)
        assert res["status"] == 0
        assert rel_inf(res["z"].cpu().numpy(), O.rollout(m, c.x, 0.2, 3)) < TOL
    finally:
        for k in env:
            os.environ.pop(k, None)


@pytest.mark.parametrize("M,L,N,B,T,chunk,bound", [(16, 64, 16, 3, 300, 0, 0.05), (20, 40, 5, 3, 200, 32, 0.2)])
def test_shallow_safeguard_rejections_reach_rollout(M, L, N, B, T, chunk, bound):
    """Rejected updates retried with the damped stored Jacobians gamma J~ still reach the
    rollout."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    c = _case(M, L, N, B, T, 0.1, 700 + M)
    m = oracle_model(c)
    say("deer_solve shallow safeguard", M, L, N, B, T, chunk, bound)
    plain = D.deer_solve(m, c.x, 0.1, N, tol=1e-5, max_iter=100)
    res = D.deer_solve(m, c.x, 0.1, N, tol=1e-5, max_iter=5000, step_bound=bound)
    assert res["status"] == 0, res
    assert rel_inf(res["z"].cpu().numpy(), O.rollout(m, c.x, 0.1, N)) < TOL
    assert sum(res["iters"]) > sum(plain["iters"])


def test_config3_reduced():
    """Workload 3 (shallow PLRNN M=32, L=256, Lorenz-96) with T reduced to 4096."""
    c = W.make_config(3, B=2, T=4096)
    m = oracle_model(c)
    say("deer_solve config3 reduced")
    res = D.deer_solve(m, c.x, c.alpha, c.n_obs, tol=c.tol)
    assert res["status"] == 0
    ref = O.rollout(m, c.x, c.alpha, c.n_obs)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    z32 = ref.astype(np.float32)
    out = D.deer_adjoint(m, c.x, z32, c.alpha, c.n_obs)
    lam = O.adjoint(m, c.x, z32, c.alpha, c.n_obs, mask_precision="float32")
    gr = O.param_grads(m, c.x, z32, c.alpha, c.n_obs, lam, mask_precision="float32")
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    for k in ("A", "W1", "W2", "h1", "h2"):
        assert rel_inf(out["grads"][k].cpu().numpy(), gr[k]) < TOL, k


@pytest.mark.parametrize("M,L,N,B,T,alpha,chunk", [(32, 256, 32, 3, 700, 0.1, 0), (32, 256, 8, 2, 1000, 0.1, 37),
                                                   (5, 20, 2, 2, 333, 0.3, 33), (16, 384, 16, 2, 300, 0.1, 0),
                                                   (64, 128, 64, 2, 257, 0.1, 0), (64, 50, 3, 1, 400, 0.15, 0),
                                                   (1, 7, 1, 2, 50, 0.2, 0), (24, 48, 24, 3, 129, 0.2, 16),
                                                   (40, 100, 10, 5, 211, 0.2, 0)])
def test_shallow_fused_and_stored_updates_agree(M, L, N, B, T, alpha, chunk):
    """The Newton update and the adjoint without a stored Jacobian (J~_t rebuilt from the
    hidden masks inside the chunk products, Jacobian-vector products in the fix-ups) and the
    stored-Jacobian ones: both solves reach the sequential rollout, in the same number of
    updates up to one (the two round differently), also with forced rejections (damped gamma
    J~); both adjoints and all gradients equal the oracle's.  Covers ragged last chunks,
    sequences that converge at different updates, and every register-tile variant."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    c = _case(M, L, N, B, T, alpha, 900 + M + L)
    m = oracle_model(c)
    ref = O.rollout(m, c.x, alpha, N)
    z32 = ref.astype(np.float32)
    lam = O.adjoint(m, c.x, z32, alpha, N, mask_precision="float32")
    gr = O.param_grads(m, c.x, z32, alpha, N, lam, mask_precision="float32")
    out = {}
    # stored J~; without a stored J~ and the fixed-order residual; the default (matrix-core
    # residual in the Newton passes)
    paths = {"0": ("0", "1"), "1x": ("1", "0"), "1": ("1", "1")}
    try:
        for path, (fz, rm) in paths.items():
            os.environ["DEER_SH_FUSED"] = fz
            os.environ["DEER_SH_RESMFMA"] = rm
            say("deer_solve shallow path", path, M, L, N, B, T, alpha, chunk)
            res = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=200)
            assert res["status"] == 0, (path, res)
            assert rel_inf(res["z"].cpu().numpy(), ref) < TOL, path
            say("deer_solve shallow path with rejections", path)
            rj = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=5000, step_bound=0.05)
            assert rj["status"] == 0, (path, rj)
            assert rel_inf(rj["z"].cpu().numpy(), ref) < TOL, path
            out[path] = (list(res["iters"]), list(rj["iters"]))
            say("deer_adjoint shallow path", path)
            adj = D.deer_adjoint(m, c.x, z32, alpha, N)
            assert rel_inf(adj["lam"].cpu().numpy(), lam) < TOL, path
            for k in ("A", "W1", "W2", "h1", "h2"):
                assert rel_inf(adj["grads"][k].cpu().numpy(), gr[k]) < TOL, (path, k)
    finally:
        os.environ.pop("DEER_SH_FUSED", None)
        os.environ.pop("DEER_SH_RESMFMA", None)
    for p2 in ("1x", "1"):
        for a, b in zip(out["0"][0], out[p2][0]):
            assert abs(a - b) <= 1, out
