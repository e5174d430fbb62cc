"""Full-size parity of the benchmarked workloads, in the launch configuration bench.py times.

Workload 5 (vanilla PLRNN M=64, T=131072, B=32), workload 3 (shallow PLRNN M=32, L=256,
T=65536, B=8) and workload 4 (diagonal SSM N=64, T=2^20, B=4) against the float64 oracle
on every output; workloads 1 and 2 are covered at full size in test_gpu_plrnn.py.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W
from gpu_util import masks_to_bool, oracle_model, rel_inf, say, tie_band_check

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402

TOL = 1e-4


def _blas_threads():
    try:
        from threadpoolctl import threadpool_limits
        return threadpool_limits(8)
    except Exception:
        return None


@pytest.mark.parametrize("cfg", [5, 3])
def test_plrnn_workload_full(cfg):
    """Solve to tol 1e-5, compare every state with the sequential rollout; then the adjoint
    and all parameter gradients at the oracle's fixed point rounded to float32."""
    _blas_threads()
    c = W.make_config(cfg)
    m = oracle_model(c)
    say("deer_solve full workload", cfg, c.name)
    res = D.deer_solve(m, c.x, c.alpha, c.n_obs, tol=c.tol, want_masks=True)
    assert res["status"] == 0, res["status"]
    z_gpu = res["z"].cpu().numpy()
    masks = res["masks"].cpu().numpy()
    del res
    ref = O.rollout(m, c.x, c.alpha, c.n_obs)
    assert rel_inf(z_gpu, ref) < TOL
    # masks at the returned z equal the fixed point's wherever the decision is not a tie
    _, _, _, zt = O.residual_and_masks(m, c.x, ref, c.alpha, c.n_obs)
    u = O.preactivation(m, zt)
    H = u.shape[2]
    got = masks_to_bool(masks, H)
    tie_band_check(got, u, 1e-4, "solve masks")
    del zt, u, got, z_gpu
    z32 = ref.astype(np.float32)
    del ref
    say("deer_adjoint full workload", cfg)
    out = D.deer_adjoint(m, c.x, z32, c.alpha, c.n_obs)
    lam_gpu = out["lam"].cpu().numpy()
    grads = {k: v.cpu().numpy() for k, v in out["grads"].items()}
    del out
    lam = O.adjoint(m, c.x, z32, c.alpha, c.n_obs, mask_precision="float32")
    assert rel_inf(lam_gpu, lam) < TOL
    gr = O.param_grads(m, c.x, z32, c.alpha, c.n_obs, lam, mask_precision="float32")
    for k, v in grads.items():
        assert rel_inf(v, gr[k]) < TOL, k


def test_diag_workload_full():
    """Workload 4, the step bench.py times: fused-projection forward scan, read-out loss and
    cotangent (ReLU decisions taken from the GPU, checked against float64 outside a tie
    band), reverse scan of the real cotangent with dlambda / dBc, against the oracle."""
    _blas_threads()
    c = W.make_config(4)
    p = c.params
    m = {"kind": "diag_ssm", "lam": p["lam"], "Bc": p["Bc"]}
    ro = {k: p[k] for k in ("Wa", "ca", "Wb", "cb")}
    say("deer_solve diag full")
    res = D.deer_solve(m, c.x, 0.0, 0)
    h_gpu = res["z"]
    say("deer_readout_loss diag full")
    r = D.deer_readout_loss(ro, h_gpu, c.x, want_masks=True)
    say("deer_adjoint diag full (real g)")
    out = D.deer_adjoint(m, c.x, h_gpu, 0.0, 0, g=r["g"])
    say("deer_adjoint diag full (real g, gradients only: the step bench.py times)")
    out_g = D.deer_adjoint(m, c.x, h_gpu, 0.0, 0, g=r["g"], want_lam=False)
    h = O.diag_scan(p["lam"], O.diag_ssm_inputs(p, c.x))
    hg = h_gpu.cpu().numpy()
    assert rel_inf(hg[..., 0] + 1j * hg[..., 1], h) < TOL
    del hg
    H = p["Wa"].shape[0]
    w = r["masks"].cpu().numpy().astype(np.uint32)
    mask = (((w[..., :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(w.shape[:-1] + (-1,))[..., :H]
            .astype(bool))
    del w
    s = O.diag_ssm_readout_preactivation(p, h)
    tie_band_check(mask, s, 1e-5, "read-out masks")
    del s
    loss, g, gr = O.diag_ssm_loss_and_seed(p, h, c.x, mask=mask)
    del mask
    assert abs(float(r["loss"].cpu()[0]) - loss) <= 1e-5 * loss
    assert rel_inf(r["g"].cpu().numpy(), g) < TOL
    for k in ("Wa", "ca", "Wb", "cb"):
        assert rel_inf(r["grads"][k].cpu().numpy(), gr[k]) < TOL, k
    a = O.diag_scan_reverse(p["lam"], g)
    del g
    ag = out["lam"].cpu().numpy()
    assert rel_inf(ag[..., 0] + 1j * ag[..., 1], a) < TOL
    del ag
    pg = O.diag_ssm_param_grads(a, h, c.x)
    dl = out["grads"]["lam"].cpu().numpy()
    dB = out["grads"]["Bc"].cpu().numpy()
    assert rel_inf(dl[..., 0] + 1j * dl[..., 1], pg["lam"]) < TOL
    assert rel_inf(dB[..., 0] + 1j * dB[..., 1], pg["Bc"]) < TOL
    dl = out_g["grads"]["lam"].cpu().numpy()
    dB = out_g["grads"]["Bc"].cpu().numpy()
    assert rel_inf(dl[..., 0] + 1j * dl[..., 1], pg["lam"]) < TOL
    assert rel_inf(dB[..., 0] + 1j * dB[..., 1], pg["Bc"]) < TOL
