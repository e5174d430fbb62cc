"""Latent warm-up on the GPU (the first T_w forced inputs with alpha = 1, the warm-up states
left out of the loss) against the float64 oracle: solves against the warm-up rollout, adjoints
and gradients against the oracle's recursion at the same float32 trajectory, for GTF-DEER and
quasi-DEER, vanilla and shallow PLRNNs."""
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

TOL = 1e-4
_ENV = ("DEER_CHUNK", "DEER_GROUP_MAPS", "DEER_PASS_FUSION", "DEER_FIX_MFMA", "DEER_SH_FUSED", "DEER_SH_RESMFMA")


@pytest.fixture(autouse=True)
def _no_overrides():
    for k in _ENV:
        os.environ.pop(k, None)
    yield
    for k in _ENV:
        os.environ.pop(k, None)
CASES = [("plrnn", 16, 0, 3, 2, 700, 100), ("plrnn", 3, 0, 3, 1, 300, 1), ("plrnn", 24, 0, 24, 3, 1000, 999),
         ("plrnn", 64, 0, 64, 2, 513, 200), ("shplrnn", 5, 50, 3, 2, 600, 128), ("shplrnn", 32, 256, 32, 1, 800, 50)]


def _case(kind, M, L, N, B, T, seed):
    if kind == "plrnn":
        return W.random_plrnn_case(M, N, B, T, 0.2, seed, w_norm=0.2, a_range=(0.3, 0.75))
    return W.random_shplrnn_case(M, L, N, B, T, 0.15, seed, w_norm=0.2, a_range=(0.3, 0.75))


@pytest.mark.parametrize("kind,M,L,N,B,T,T_w", CASES)
@pytest.mark.parametrize("quasi", [False, True])
def test_warmup_solve_and_adjoint(kind, M, L, N, B, T, T_w, quasi):
    c = _case(kind, M, L, N, B, T, 500 + M + T_w)
    m = oracle_model(c)
    solve = D.deer_solve_quasi if quasi else D.deer_solve
    adjoint = D.deer_adjoint_quasi if quasi else D.deer_adjoint
    say("warm-up solve", kind, M, L, N, B, T, T_w, quasi)
    res = solve(m, c.x, c.alpha, N, tol=1e-5, max_iter=T + 2, T_w=T_w)
    assert res["status"] == 0, res["status"]
    ref = O.rollout(m, c.x, c.alpha, N, T_w=T_w)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    z32 = ref.astype(np.float32)
    say("warm-up adjoint", kind, M, L, N, B, T, T_w, quasi)
    out = adjoint(m, c.x, z32, c.alpha, N, T_w=T_w)
    lam = O.adjoint(m, c.x, z32, c.alpha, N, mask_precision="float32", quasi=quasi, T_w=T_w)
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    gr = O.param_grads(m, c.x, z32, c.alpha, N, lam, mask_precision="float32", T_w=T_w)
    for k, v in out["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k


def test_warmup_with_given_cotangent_and_initial_state():
    c = _case("plrnn", 8, 0, 2, 2, 400, 520)
    m = oracle_model(c)
    z0 = np.random.default_rng(1).standard_normal((2, 8)).astype(np.float32)
    T_w = 37
    say("warm-up solve with z0")
    res = D.deer_solve(m, c.x, c.alpha, 2, z0=z0, tol=1e-5, T_w=T_w)
    ref = O.rollout(m, c.x, c.alpha, 2, z0=z0, T_w=T_w)
    assert res["status"] == 0 and rel_inf(res["z"].cpu().numpy(), ref) < TOL
    z32 = ref.astype(np.float32)
    g = np.random.default_rng(2).standard_normal(z32.shape).astype(np.float32)
    say("warm-up adjoint with g and z0")
    out = D.deer_adjoint(m, c.x, z32, c.alpha, 2, z0=z0, g=g, T_w=T_w)
    lam = O.adjoint(m, c.x, z32, c.alpha, 2, z0=z0, g=g, mask_precision="float32", T_w=T_w)
    assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
    gr = O.param_grads(m, c.x, z32, c.alpha, 2, lam, z0=z0, mask_precision="float32", T_w=T_w)
    for k, v in out["grads"].items():
        assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k


# Vanilla PLRNN: the warm-up is part of the one Newton iteration (the kernels take the forcing
# strength per step: alpha_s = 1 and P_1 for s <= T_w).  M <= 16: T_w at the first step, inside a
# chunk and a tile, on a chunk boundary (T_w + 1 divisible by the chunk length) and next to the
# end; chunk layouts through the per-step slow paths (ragged tiles), composed wave maps, group
# maps and the fused pass kernel; every latent observed; M = 3 (the one-launch kernels step
# aside).  M > 16: 32- and 64-wide kernels, M not a multiple of 4, ragged chunks, every latent
# observed (the uniform-forcing M = 64 kernel steps aside).
JOINT = [(16, 3, 2, 700, 100, 0), (16, 3, 2, 2048, 511, 16), (16, 3, 2, 2048, 700, 16), (12, 4, 2, 4096, 1, 32),
         (12, 4, 2, 4096, 4094, 32), (7, 3, 3, 640, 77, 40), (5, 2, 3, 1000, 333, 25), (16, 16, 2, 513, 200, 0),
         (3, 3, 1, 300, 17, 0), (24, 24, 3, 1000, 999, 0), (33, 5, 2, 700, 333, 37), (40, 10, 2, 300, 1, 0),
         (64, 64, 2, 513, 200, 0), (61, 7, 2, 400, 150, 64)]


def _joint_case(M, N, B, T, T_w, chunk, seed):
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    os.environ["DEER_GROUP_MAPS"] = "1"   # where 32 divides the chunk count, whatever the size
    return W.random_plrnn_case(M, N, B, T, 0.2, seed, w_norm=0.2, a_range=(0.3, 0.75))


@pytest.mark.parametrize("M,N,B,T,T_w,chunk", JOINT)
def test_warmup_one_iteration_newton_iterates(M, N, B, T, T_w, chunk):
    """The k-th Newton iterate of the joint iteration equals the oracle's (Alg. GTF-DEER with
    P_1 for t <= T_w), for k = 1 and 3: the per-step forcing in the residual, the chunk products,
    the local solutions and the fix-up."""
    c = _joint_case(M, N, B, T, T_w, chunk, 4100 + M + T_w)
    m = oracle_model(c)
    for k in (1, 3):
        say("warm-up one iteration, fixed updates", M, N, B, T, T_w, chunk, k)
        res = D.deer_solve(m, c.x, c.alpha, N, fixed_iters=k, T_w=T_w, want_masks=True)
        ref = O.newton(m, c.x, c.alpha, N, fixed_iters=k, T_w=T_w)
        assert res["status"] == 0 and res["iters"] == [k] * B
        z = res["z"].cpu().numpy()
        assert rel_inf(z, ref["z"]) < TOL, k
        fp32 = O.activation_mask_fp32(m, z, c.x, c.alpha, N, None, T_w)
        assert np.array_equal(masks_to_bool(res["masks"].cpu().numpy(), M), fp32)


@pytest.mark.parametrize("M,N,B,T,T_w,chunk", JOINT)
def test_warmup_one_iteration_counts_and_adjoint(M, N, B, T, T_w, chunk):
    """Solved to tolerance the joint iteration reaches the warm-up rollout in the oracle's number
    of updates (up to one), with the fused pass kernel and with separate kernels (M <= 16), with
    the matrix-core and the lane-per-latent fix-up (M > 16); the adjoint and gradients (MSE over
    the states after the warm-up, and a given cotangent) match the oracle's joint recursion."""
    c = _joint_case(M, N, B, T, T_w, chunk, 4200 + M + T_w)
    m = oracle_model(c)
    ref = O.rollout(m, c.x, c.alpha, N, T_w=T_w)
    want = O.newton(m, c.x, c.alpha, N, tol=1e-5, T_w=T_w)["iters"].tolist()
    for fuse in ("1", "0"):
        os.environ["DEER_PASS_FUSION"] = fuse
        os.environ["DEER_FIX_MFMA"] = fuse
        say("warm-up one iteration to tolerance", M, N, B, T, T_w, chunk, fuse)
        res = D.deer_solve(m, c.x, c.alpha, N, tol=1e-5, max_iter=200, T_w=T_w)
        assert res["status"] == 0, res
        assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
        assert max(abs(a - b) for a, b in zip(res["iters"], want)) <= 1, (res["iters"], want)
    z32 = ref.astype(np.float32)
    g = np.random.default_rng(M + T_w).standard_normal(z32.shape).astype(np.float32)
    for gg in (None, g):
        say("warm-up one iteration adjoint", M, N, B, T, T_w, chunk, gg is None)
        out = D.deer_adjoint(m, c.x, z32, c.alpha, N, g=gg, T_w=T_w)
        lam = O.adjoint(m, c.x, z32, c.alpha, N, g=gg, mask_precision="float32", T_w=T_w)
        assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL
        gr = O.param_grads(m, c.x, z32, c.alpha, N, lam, mask_precision="float32", T_w=T_w)
        for k, v in out["grads"].items():
            assert rel_inf(v.cpu().numpy(), gr[k]) < TOL, k


# Shallow PLRNN: the warm-up inside the one Newton iteration on every path: the Jacobians rebuilt
# from the masks (P_1 in the warm-up steps of the chunk products and Jacobian-vector fix-ups) with
# the matrix-core or the fixed-order residual, the stored Jacobians (formed per step range), and
# M > 64 (the wide kernels).  Cases: (M, L, N, B, T, T_w, chunk, check the 1st and 2nd iterates).
SH_JOINT = [(5, 50, 3, 2, 600, 128, 0, True), (32, 256, 32, 1, 800, 50, 0, False),
            (20, 40, 5, 3, 300, 77, 64, True), (16, 64, 16, 2, 500, 1, 0, True),
            (64, 128, 64, 1, 300, 150, 0, True), (100, 64, 20, 1, 200, 60, 0, True)]
SH_PATHS = {"stored": ("0", "1"), "fixed-order residual": ("1", "0"), "matrix-core residual": ("1", "1")}


@pytest.mark.parametrize("M,L,N,B,T,T_w,chunk,iterates", SH_JOINT)
def test_shallow_warmup_one_iteration(M, L, N, B, T, T_w, chunk, iterates):
    """The oracle's joint iteration (Alg. GTF-DEER with P_1 for t <= T_w): its first Newton
    iterates, its update counts (up to one) and its fixed point, then the adjoint and the
    gradients, on every shallow path."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    c = W.random_shplrnn_case(M, L, N, B, T, 0.15, 4300 + M + T_w, w_norm=0.2, a_range=(0.3, 0.75))
    m = oracle_model(c)
    ref = O.rollout(m, c.x, c.alpha, N, T_w=T_w)
    want = O.newton(m, c.x, c.alpha, N, tol=1e-5, T_w=T_w)["iters"].tolist()
    firsts = {k: O.newton(m, c.x, c.alpha, N, fixed_iters=k, T_w=T_w)["z"] for k in (1, 2)} if iterates else {}
    z32 = ref.astype(np.float32)
    lam = O.adjoint(m, c.x, z32, c.alpha, N, mask_precision="float32", T_w=T_w)
    gr = O.param_grads(m, c.x, z32, c.alpha, N, lam, mask_precision="float32", T_w=T_w)
    try:
        for path, (fz, rm) in SH_PATHS.items():
            os.environ["DEER_SH_FUSED"] = fz
            os.environ["DEER_SH_RESMFMA"] = rm
            for k, zk in firsts.items():
                say("shallow warm-up one iteration, fixed updates", path, M, L, N, B, T, T_w, k)
                res = D.deer_solve(m, c.x, c.alpha, N, fixed_iters=k, T_w=T_w)
                assert res["status"] == 0 and res["iters"] == [k] * B
                assert rel_inf(res["z"].cpu().numpy(), zk) < TOL, (path, k)
            say("shallow warm-up one iteration to tolerance", path, M, L, N, B, T, T_w)
            res = D.deer_solve(m, c.x, c.alpha, N, tol=1e-5, max_iter=200, T_w=T_w)
            assert res["status"] == 0, (path, res)
            assert rel_inf(res["z"].cpu().numpy(), ref) < TOL, path
            assert max(abs(a - b) for a, b in zip(res["iters"], want)) <= 1, (path, res["iters"], want)
            say("shallow warm-up one iteration adjoint", path)
            out = D.deer_adjoint(m, c.x, z32, c.alpha, N, T_w=T_w)
            assert rel_inf(out["lam"].cpu().numpy(), lam) < TOL, path
            for key, v in out["grads"].items():
                assert rel_inf(v.cpu().numpy(), gr[key]) < TOL, (path, key)
    finally:
        os.environ.pop("DEER_SH_FUSED", None)
        os.environ.pop("DEER_SH_RESMFMA", None)


@pytest.mark.parametrize("kind,M,L,N,B,T,T_w", [("plrnn", 16, 0, 3, 2, 300, 60), ("plrnn", 40, 0, 40, 2, 200, 1),
                                                ("shplrnn", 5, 50, 3, 2, 250, 100)])
def test_quasi_warmup_one_iteration(kind, M, L, N, B, T, T_w):
    """Quasi-DEER takes the warm-up inside its one iteration as well (diagonal coefficients with
    P_1 for t <= T_w): the oracle's first quasi-Newton iterates and its update counts (up to one)."""
    c = _case(kind, M, L, N, B, T, 4400 + M + T_w)
    m = oracle_model(c)
    for k in (1, 2):
        say("quasi warm-up one iteration, fixed updates", kind, M, L, N, B, T, T_w, k)
        res = D.deer_solve_quasi(m, c.x, c.alpha, N, fixed_iters=k, T_w=T_w)
        ref = O.newton(m, c.x, c.alpha, N, fixed_iters=k, T_w=T_w, quasi=True)
        assert res["status"] == 0 and res["iters"] == [k] * B
        assert rel_inf(res["z"].cpu().numpy(), ref["z"]) < TOL, k
    say("quasi warm-up one iteration to tolerance", kind, M, L, N, B, T, T_w)
    res = D.deer_solve_quasi(m, c.x, c.alpha, N, tol=1e-5, max_iter=T + 2, T_w=T_w)
    want = O.newton(m, c.x, c.alpha, N, tol=1e-5, max_iter=T + 2, T_w=T_w, quasi=True)["iters"].tolist()
    assert res["status"] == 0, res
    assert max(abs(a - b) for a, b in zip(res["iters"], want)) <= 1, (res["iters"], want)
