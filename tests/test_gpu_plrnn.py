"""Vanilla PLRNN GTF-DEER on the GPU against the float64 oracle (through the C ABI).

Tolerance: 1e-4 normwise relative error for float32 states, adjoints and gradients;
bit-exact ReLU masks when both sides take the decision in float32 on the same input.
"""
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


@pytest.fixture(autouse=True)
def _no_chunk_override():
    for k in ("DEER_CHUNK", "DEER_GROUP_MAPS", "DEER_PASS_FUSION"):
        os.environ.pop(k, None)
    yield
    for k in ("DEER_CHUNK", "DEER_GROUP_MAPS", "DEER_PASS_FUSION"):
        os.environ.pop(k, None)


def _case(M, N, B, T, alpha, seed, w_std=None):
    """A random vanilla PLRNN; by default a contraction (A in [0.3, 0.75], ||W||_2 = 0.2) so
    that the trajectory stays O(1) for any M and N."""
    if w_std is not None:
        return W.random_plrnn_case(M, N, B, T, alpha, seed, w_std=w_std)
    return W.random_plrnn_case(M, N, B, T, alpha, seed, w_norm=0.2, a_range=(0.3, 0.75))


@pytest.mark.parametrize("M,N,T", [(1, 1, 50), (3, 3, 100), (16, 3, 257), (17, 5, 130), (33, 33, 64), (64, 64, 100)])
def test_jacobian_masks_residual(M, N, T):
    c = _case(M, N, 2, T, 0.2, 100 + M)
    m = oracle_model(c)
    z = np.random.default_rng(1).standard_normal((2, T, M)).astype(np.float32)
    say("plrnn_jacobian", M, N, T)
    out = D.plrnn_jacobian(m, c.x, z, c.alpha, N, want=("F", "r", "masks"), dense_J=True)
    torch.cuda.synchronize()
    ref = O.jacobian_at(m, c.x, z, c.alpha, N, mask_precision="float32",
                        dense_index=[(b, t) for b in range(2) for t in range(T)])
    got_mask = masks_to_bool(out["masks"].cpu().numpy(), M)
    assert np.array_equal(got_mask, ref["mask"])
    assert rel_inf(out["F"].cpu().numpy(), ref["F"]) < 1e-5
    assert rel_inf(out["r"].cpu().numpy(), ref["r"]) < 1e-5
    assert rel_inf(out["J"].cpu().numpy().reshape(-1, M, M), ref["J"]) < 1e-6


def test_config1_fixed_five_iterations():
    """Workload 1 (vanilla PLRNN M=3, T=1024): exactly 5 Newton updates from the teacher states."""
    c = W.make_config(1)
    m = oracle_model(c)
    say("deer_solve config1 fixed 5")
    res = D.deer_solve(m, c.x, c.alpha, c.n_obs, fixed_iters=5)
    ref = O.newton(m, c.x, c.alpha, c.n_obs, fixed_iters=5)
    assert res["status"] == 0
    assert rel_inf(res["z"].cpu().numpy(), ref["z"]) < TOL
    assert res["iters"] == [5]


@pytest.mark.parametrize("M,N,B,T,k", [(1, 1, 1, 1, 1), (2, 1, 3, 17, 3), (3, 3, 1, 1024, 5), (4, 4, 2, 4096, 4),
                                     (3, 2, 2, 300, 7), (4, 2, 1, 255, 2)])
@pytest.mark.parametrize("user_z0", [False, True])
def test_small_solve_in_one_launch(M, N, B, T, k, user_z0):
    """Small models with a fixed number of updates run the whole solve in one workgroup per
    sequence (chunk maps, two-level carries, in-place fix-up): the oracle's k-th Newton iterate,
    and the general path's (DEER_SMALL=0), with the masks at the result."""
    c = _case(M, N, B, T, 0.2, 200 + M + T)
    m = oracle_model(c)
    z0 = np.random.default_rng(M).standard_normal((B, M)).astype(np.float32) if user_z0 else None
    say("deer_solve small one-launch", M, N, B, T, k, user_z0)
    res = D.deer_solve(m, c.x, c.alpha, N, fixed_iters=k, z0=z0, want_masks=True)
    ref = O.newton(m, c.x, c.alpha, N, fixed_iters=k, z0=z0)
    assert res["status"] == 0 and res["iters"] == [k] * B
    z = res["z"].cpu().numpy()
    assert rel_inf(z, ref["z"]) < TOL
    assert np.all(np.abs(np.asarray(res["norms"]) - ref["norms"]) <= 1e-4 * (1.0 + np.abs(ref["norms"])))
    fp32 = O.activation_mask_fp32(m, z, c.x, c.alpha, N, z0)
    assert np.array_equal(masks_to_bool(res["masks"].cpu().numpy(), M), fp32)
    os.environ["DEER_SMALL"] = "0"
    try:
        say("deer_solve general path", M, N, B, T, k, user_z0)
        gen = D.deer_solve(m, c.x, c.alpha, N, fixed_iters=k, z0=z0)
    finally:
        os.environ.pop("DEER_SMALL", None)
    assert rel_inf(z, gen["z"].cpu().numpy()) < TOL


@pytest.mark.parametrize("M,N,B,T,alpha,chunk", [
    (3, 3, 1, 300, 0.1, 0), (3, 3, 2, 300, 0.1, 17), (16, 3, 3, 1000, 0.2, 0), (16, 3, 2, 777, 0.2, 64),
    (20, 4, 2, 513, 0.3, 100), (32, 32, 2, 600, 0.1, 0), (40, 10, 2, 300, 0.3, 33), (64, 64, 2, 400, 0.05, 0),
    (64, 64, 3, 1000, 0.05, 128), (5, 2, 4, 64, 0.5, 64), (16, 16, 1, 1, 0.2, 0), (8, 8, 2, 2, 0.2, 0),
    # chunk counts divisible by 4 (composed wave maps for M <= 16): full tiles, a ragged second
    # tile, and chunks shorter than a tile
    (16, 3, 2, 512, 0.2, 16), (7, 3, 3, 640, 0.3, 40), (16, 3, 2, 1000, 0.2, 25),
    # chunk counts divisible by 32 (group maps walked by the fix-up): one, two and four groups
    (5, 2, 3, 1024, 0.3, 16), (16, 3, 2, 2048, 0.2, 16), (12, 4, 2, 4096, 0.2, 32)])
def test_solve_reaches_rollout(M, N, B, T, alpha, chunk):
    """Converged GTF-DEER equals the sequential GTF rollout (unique zero of the residual)."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    os.environ["DEER_GROUP_MAPS"] = "1"   # where 32 divides the chunk count, whatever the size
    c = _case(M, N, B, T, alpha, 200 + M + T)
    m = oracle_model(c)
    say("deer_solve", M, N, B, T, alpha, chunk)
    res = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=100, want_masks=True)
    assert res["status"] == 0, res
    ref = O.rollout(m, c.x, alpha, N)
    z = res["z"].cpu().numpy()
    assert rel_inf(z, ref) < TOL
    assert all(1 <= k <= 100 for k in res["iters"])
    assert all(n < 1e-5 for n in res["norms"])
    # masks at the returned z: equal to the fixed point's outside a tie band
    _, _, _, zt = O.residual_and_masks(m, c.x, ref, alpha, N)
    got = masks_to_bool(res["masks"].cpu().numpy(), M)
    far = np.abs(zt) > 1e-4 * np.abs(zt).max()
    assert np.array_equal(got[far], (zt > 0)[far])


@pytest.mark.parametrize("M,N,B,T,alpha,chunk,bound", [(16, 3, 2, 2048, 0.2, 16, 0.0), (12, 4, 2, 4096, 0.2, 32, 0.0),
                                                       (16, 3, 3, 512, 0.2, 16, 0.3), (9, 9, 2, 2048, 0.15, 64, 0.0)])
def test_fused_and_separate_pass_kernels_agree(M, N, B, T, alpha, chunk, bound):
    """Where every sequence is whole blocks of 32 chunks of whole tiles, one kernel per pass
    runs the fix-up of an update and the forward pass of the next; DEER_PASS_FUSION=0 keeps
    them apart.  Both reach the rollout, with the same iteration counts up to one."""
    os.environ["DEER_CHUNK"] = str(chunk)
    os.environ["DEER_GROUP_MAPS"] = "1"
    c = _case(M, N, B, T, alpha, 700 + M + T)
    m = oracle_model(c)
    ref = O.rollout(m, c.x, alpha, N)
    out = {}
    for fuse in ("1", "0"):
        os.environ["DEER_PASS_FUSION"] = fuse
        say("deer_solve fused" if fuse == "1" else "deer_solve separate", M, N, B, T, alpha, chunk, bound)
        res = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=5000, step_bound=bound)
        assert res["status"] == 0, res
        assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
        assert all(n < 1e-5 for n in res["norms"])
        out[fuse] = res["iters"]
    assert max(abs(a - b) for a, b in zip(out["1"], out["0"])) <= 1


@pytest.mark.parametrize("M,N,B,T,alpha,chunk,bound", [(64, 64, 3, 2000, 0.1, 0, 0.0), (64, 32, 2, 777, 0.2, 0, 0.0),
                                                         (33, 5, 2, 513, 0.2, 37, 0.0), (20, 20, 5, 300, 0.2, 0, 0.0),
                                                         (48, 7, 2, 700, 0.15, 64, 0.05), (61, 61, 17, 129, 0.1, 16, 0.0)])
def test_fixup_matrix_core_and_vector_paths_agree(M, N, B, T, alpha, chunk, bound):
    """M in 17..64: the forward fix-up on the matrix cores (16 chains as columns, W diag(p) row
    tiles per wave, Delta through LDS) and the lane-per-latent one both reach the rollout, in the
    same number of updates up to one; ragged chunks, M not a multiple of 4, many sequences
    converging at different updates, and forced rejections (damped gamma J~)."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    c = _case(M, N, B, T, alpha, 5100 + M + B)
    m = oracle_model(c)
    ref = O.rollout(m, c.x, alpha, N)
    its = {}
    try:
        for path in ("0", "1"):
            os.environ["DEER_FIX_MFMA"] = path
            say("fixup path", path, M, N, B, T, alpha, chunk, bound)
            res = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=3000, step_bound=bound)
            assert res["status"] == 0, (path, res)
            assert rel_inf(res["z"].cpu().numpy(), ref) < TOL, path
            its[path] = list(res["iters"])
    finally:
        os.environ.pop("DEER_FIX_MFMA", None)
    if bound == 0.0:
        for a, b in zip(its["0"], its["1"]):
            assert abs(a - b) <= 1, its


@pytest.mark.parametrize("M,N,B,T,alpha,chunk,bound", [(16, 3, 4, 300, 0.2, 0, 0.05), (16, 3, 3, 300, 0.2, 16, 0.3),
                                                       (32, 8, 3, 300, 0.1, 16, 0.1), (64, 64, 2, 200, 0.05, 0, 0.1),
                                                       (5, 2, 5, 120, 0.3, 7, 0.02), (16, 3, 3, 512, 0.2, 16, 0.3)])
def test_safeguard_rejections_reach_rollout(M, N, B, T, alpha, chunk, bound):
    """A small step bound makes the solver reject updates and retry them damped (the scan
    uses gamma J~ with gamma < 1, down to the fixed-point step); the iterates alternate
    between two buffers with per-sequence copy-back.  The result is still the rollout, and
    more passes than plain Newton's show that the safeguard ran."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    os.environ["DEER_GROUP_MAPS"] = "1"
    c = _case(M, N, B, T, alpha, 600 + M + T)
    m = oracle_model(c)
    say("deer_solve safeguard", M, N, B, T, alpha, chunk, bound)
    plain = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=100)
    res = D.deer_solve(m, c.x, alpha, N, tol=1e-5, max_iter=5000, step_bound=bound)
    assert res["status"] == 0, res
    ref = O.rollout(m, c.x, alpha, N)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    assert sum(res["iters"]) > sum(plain["iters"])
    assert all(n < 1e-5 for n in res["norms"])


def test_iteration_counts_match_oracle():
    c = _case(16, 3, 4, 800, 0.2, 7)
    m = oracle_model(c)
    say("deer_solve iteration counts")
    res = D.deer_solve(m, c.x, 0.2, 3, tol=1e-5)
    ref = O.newton(m, c.x, 0.2, 3, tol=1e-5)
    assert max(abs(a - b) for a, b in zip(res["iters"], ref["iters"].tolist())) <= 1


def test_consecutive_solves_share_the_host_block():
    """Solves in a row on one host thread: the pinned host block (flags, results, pass mark)
    grows with B and is reused; M <= 16 (passes marked by the forward pass) and M > 16 (an
    event per batch) alternate.  Each result must be the rollout with oracle-like counts."""
    for k, (M, N, B, T) in enumerate([(16, 3, 2, 300), (16, 3, 37, 200), (20, 4, 3, 250), (8, 3, 3, 400),
                                      (16, 3, 64, 128), (5, 2, 1, 90)]):
        c = _case(M, N, B, T, 0.2, 900 + k)
        m = oracle_model(c)
        say("deer_solve in a row", M, N, B, T)
        res = D.deer_solve(m, c.x, 0.2, N, tol=1e-5, max_iter=100)
        assert res["status"] == 0, res
        assert rel_inf(res["z"].cpu().numpy(), O.rollout(m, c.x, 0.2, N)) < TOL
        ref = O.newton(m, c.x, 0.2, N, tol=1e-5)
        assert max(abs(a - b) for a, b in zip(res["iters"], ref["iters"].tolist())) <= 1
        assert all(n < 1e-5 for n in res["norms"])
    # the iteration cap after a grown block: the control block is read back instead
    c = _case(16, 3, 2, 300, 0.2, 950)
    res = D.deer_solve(oracle_model(c), c.x, 0.2, 3, tol=1e-5, max_iter=2, check=False)
    assert res["status"] == 2 and res["iters"] == [2, 2]


def test_alpha1_full_observation_two_updates():
    """alpha = 1, M <= N: z* = F(zbar) in closed form; the GPU stops after 2 updates."""
    c = _case(6, 6, 3, 500, 1.0, 11, w_std=0.8)
    m = oracle_model(c)
    say("deer_solve alpha=1")
    res = D.deer_solve(m, c.x, 1.0, 6, tol=1e-5)
    closed = O.model_map(m, c.x[:, :-1].astype(np.float64))
    assert rel_inf(res["z"].cpu().numpy(), closed) < 1e-6
    assert res["iters"] == [2, 2, 2]


def test_alpha0_linear_model_two_updates():
    M, T = 8, 700
    rng = np.random.default_rng(3)
    m = {"kind": "plrnn", "A": rng.uniform(0.5, 0.9, M).astype(np.float32), "W": np.zeros((M, M), np.float32),
         "h": rng.normal(0, 0.1, M).astype(np.float32)}
    x = rng.standard_normal((2, T + 1, M)).astype(np.float32)
    say("deer_solve alpha=0 linear")
    res = D.deer_solve(m, x, 0.0, M, tol=1e-6)
    assert res["iters"] == [2, 2]
    assert rel_inf(res["z"].cpu().numpy(), O.rollout(m, x, 0.0, M)) < 1e-5


def test_user_init_and_z0():
    c = _case(16, 3, 2, 400, 0.2, 13)
    m = oracle_model(c)
    z0 = np.random.default_rng(5).standard_normal((2, 16)).astype(np.float32)
    ref = O.rollout(m, c.x, 0.2, 3, z0=z0)
    zinit = torch.tensor(ref.astype(np.float32) + 0.1, device="cuda")
    say("deer_solve user init + z0")
    res = D.deer_solve(m, c.x, 0.2, 3, z0=z0, init="user", z=zinit, tol=1e-6)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    res = D.deer_solve(m, c.x, 0.2, 3, z0=z0, init="zero", tol=1e-6)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL


def test_nonfinite_and_not_converged():
    c = _case(8, 3, 2, 200, 0.2, 17)
    m = oracle_model(c)
    x = c.x.copy()
    x[1, 50, 0] = np.nan
    say("deer_solve NaN input")
    res = D.deer_solve(m, x, 0.2, 3, tol=1e-5, check=False)
    assert res["status"] == 3                      # DEER_ERR_NONFINITE
    say("deer_solve max_iter=1")
    res = D.deer_solve(m, c.x, 0.2, 3, tol=1e-5, max_iter=1, check=False)
    assert res["status"] == 2                      # DEER_ERR_NOT_CONVERGED
    assert res["iters"] == [1, 1]


@pytest.mark.parametrize("M,N,B,T,alpha,chunk", [(3, 3, 1, 300, 0.1, 0), (16, 3, 3, 1000, 0.2, 0),
                                                 (16, 3, 2, 777, 0.2, 64), (20, 4, 2, 513, 0.3, 100),
                                                 (64, 64, 2, 400, 0.05, 0), (40, 10, 2, 300, 0.3, 33),
                                                 (8, 8, 1, 1, 0.2, 0), (16, 3, 2, 512, 0.2, 16),
                                                 (7, 3, 3, 640, 0.3, 40), (16, 3, 2, 1000, 0.2, 25),
                                                 (16, 16, 3, 256, 0.1, 32)])
def test_adjoint_and_grads(M, N, B, T, alpha, chunk):
    """lam and dL/dtheta at the same float32 trajectory (the oracle's fixed point rounded to
    float32); both sides take the ReLU decision in float32."""
    if chunk:
        os.environ["DEER_CHUNK"] = str(chunk)
    c = _case(M, N, B, T, alpha, 300 + M + T)
    m = oracle_model(c)
    z32 = O.rollout(m, c.x, alpha, N).astype(np.float32)
    say("deer_adjoint", M, N, B, T, alpha, chunk)
    out = D.deer_adjoint(m, c.x, z32, alpha, N)
    lam_ref = O.adjoint(m, c.x, z32, alpha, N, mask_precision="float32")
    g_ref = O.param_grads(m, c.x, z32, alpha, N, lam_ref, mask_precision="float32")
    assert rel_inf(out["lam"].cpu().numpy(), lam_ref) < TOL
    for k in ("A", "W", "h"):
        assert rel_inf(out["grads"][k].cpu().numpy(), g_ref[k]) < TOL, k


@pytest.mark.parametrize("M,N,B,T", [(1, 1, 1, 1), (2, 1, 3, 17), (3, 3, 1, 1024), (4, 4, 2, 4096),
                                   (3, 2, 2, 300), (4, 2, 1, 255), (3, 3, 1, 9)])
@pytest.mark.parametrize("mode", ["seed", "user_g_z0", "grads_only"])
def test_small_adjoint_in_one_launch(M, N, B, T, mode):
    """Small models take the adjoint in one workgroup per sequence (chunk maps of the
    transposed Jacobians, two-level carries from the last chunk, re-walk with the gradient
    partials): lam and dL/dtheta against the oracle, and against the general path
    (DEER_SMALL=0); B = 1 writes the gradients without the batch reduction."""
    alpha = 0.2
    c = _case(M, N, B, T, alpha, 400 + M + T)
    m = oracle_model(c)
    rng = np.random.default_rng(M + T)
    z0 = rng.standard_normal((B, M)).astype(np.float32) if mode == "user_g_z0" else None
    z32 = O.rollout(m, c.x, alpha, N, z0=z0).astype(np.float32)
    g = rng.standard_normal(z32.shape).astype(np.float32) if mode == "user_g_z0" else None
    want_lam = mode != "grads_only"
    say("deer_adjoint small one-launch", M, N, B, T, mode)
    out = D.deer_adjoint(m, c.x, z32, alpha, N, z0=z0, g=g, want_lam=want_lam)
    lam_ref = O.adjoint(m, c.x, z32, alpha, N, z0=z0, g=g, mask_precision="float32")
    g_ref = O.param_grads(m, c.x, z32, alpha, N, lam_ref, z0=z0, mask_precision="float32")
    if want_lam:
        assert rel_inf(out["lam"].cpu().numpy(), lam_ref) < TOL
    for k in ("A", "W", "h"):
        assert rel_inf(out["grads"][k].cpu().numpy(), g_ref[k]) < TOL, k
    os.environ["DEER_SMALL"] = "0"
    try:
        say("deer_adjoint general path", M, N, B, T, mode)
        gen = D.deer_adjoint(m, c.x, z32, alpha, N, z0=z0, g=g, want_lam=want_lam)
    finally:
        os.environ.pop("DEER_SMALL", None)
    if want_lam:
        assert rel_inf(out["lam"].cpu().numpy(), gen["lam"].cpu().numpy()) < TOL
    for k in ("A", "W", "h"):
        assert rel_inf(out["grads"][k].cpu().numpy(), gen["grads"][k].cpu().numpy()) < TOL, k


def test_adjoint_user_cotangent():
    c = _case(16, 3, 2, 300, 0.2, 19)
    m = oracle_model(c)
    z32 = O.rollout(m, c.x, 0.2, 3).astype(np.float32)
    g = np.random.default_rng(2).standard_normal(z32.shape).astype(np.float32)
    say("deer_adjoint user g")
    out = D.deer_adjoint(m, c.x, z32, 0.2, 3, g=g)
    lam_ref = O.adjoint(m, c.x, z32, 0.2, 3, g=g, mask_precision="float32")
    assert rel_inf(out["lam"].cpu().numpy(), lam_ref) < TOL


def test_config2_full_size():
    """Workload 2 at full size (M=16, N=3, T=16384, B=16): solve, then adjoint + gradients."""
    c = W.make_config(2)
    m = oracle_model(c)
    say("deer_solve config2 full")
    res = D.deer_solve(m, c.x, c.alpha, c.n_obs, tol=c.tol)
    assert res["status"] == 0
    ref = O.rollout(m, c.x, c.alpha, c.n_obs)
    assert rel_inf(res["z"].cpu().numpy(), ref) < TOL
    z32 = ref.astype(np.float32)
    say("deer_adjoint config2 full")
    out = D.deer_adjoint(m, c.x, z32, c.alpha, c.n_obs)
    lam_ref = O.adjoint(m, c.x, z32, c.alpha, c.n_obs, mask_precision="float32")
    assert rel_inf(out["lam"].cpu().numpy(), lam_ref) < TOL
    g_ref = O.param_grads(m, c.x, z32, c.alpha, c.n_obs, lam_ref, mask_precision="float32")
    for k in ("A", "W", "h"):
        assert rel_inf(out["grads"][k].cpu().numpy(), g_ref[k]) < TOL, k
