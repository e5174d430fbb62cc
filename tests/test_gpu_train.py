"""The training step (solve, MSE over the post-warm-up states plus MAR, its gradient, one Adam
update in place) on the GPU against the float64 oracle, through the C ABI: the trajectory, the
loss, the total gradient, and two consecutive Adam updates (the oracle's Adam applied to the
GPU's gradients, so the update itself is checked without the sign sensitivity of Adam's first
steps)."""
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


def _case(kind, M, L, N, B, T, seed):
    if kind == "plrnn":
        return W.random_plrnn_case(M, N, B, T, 0.2, seed, w_norm=0.2, a_range=(0.3, 0.75))
    return W.random_shplrnn_case(M, L, N, B, T, 0.15, seed, w_norm=0.2, a_range=(0.3, 0.75))


@pytest.mark.parametrize("kind,M,L,N,B,T,T_w,quasi,p", [
    ("plrnn", 16, 0, 3, 2, 600, 0, False, 2), ("plrnn", 8, 0, 4, 2, 500, 50, False, 1),
    ("shplrnn", 5, 50, 3, 2, 400, 32, False, 2), ("plrnn", 16, 0, 3, 2, 300, 0, True, 1),
    ("shplrnn", 6, 20, 2, 1, 256, 0, True, 2)])
def test_train_steps(kind, M, L, N, B, T, T_w, quasi, p):
    c = _case(kind, M, L, N, B, T, 600 + M + T)
    m_np = oracle_model(c)
    model = D._Model(m_np)
    M_r, lam_mar = max(1, M // 2), 0.5
    Lw = L if kind == "shplrnn" else M
    gw, gv = 1.0 / (3 * Lw), 1.0 / (3 * M)
    hp = dict(lr=1e-2, beta1=0.9, beta2=0.99, eps=1e-6, mar_lambda=lam_mar, mar_units=M_r, mar_p=p, mar_gamma_w=gw,
              mar_gamma_v=gv, quasi=quasi, T_w=T_w, max_iter=T + 2, want_grads=True)
    params = {k: np.asarray(v, np.float64) for k, v in m_np.items() if k != "kind"}
    state, ostate = None, {}
    for step in (1, 2):
        cur = {"kind": kind, **{k: v.astype(np.float32) for k, v in params.items()}}
        say("deer_train_step", kind, M, L, N, B, T, T_w, quasi, p, step)
        out = D.deer_train_step(model, c.x, c.alpha, N, step=step, state=state, **hp)
        state = out["state"]
        assert out["status"] == 0
        ref = O.rollout(cur, c.x, c.alpha, N, T_w=T_w)
        z = out["z"].cpu().numpy()
        assert rel_inf(z, ref) < TOL
        lam = O.adjoint(cur, c.x, z, c.alpha, N, mask_precision="float32", quasi=quasi, T_w=T_w)
        gr = O.param_grads(cur, c.x, z, c.alpha, N, lam, mask_precision="float32", T_w=T_w)
        mar_loss, mar_gr = O.mar_loss_and_grads(cur, M_r, lam_mar, p, gw, gv)
        loss = O.mse_loss(z, c.x, T_w=T_w) + mar_loss
        assert abs(float(out["loss"].cpu()[0]) - loss) <= 1e-5 * abs(loss)
        ggpu = {k: v.cpu().numpy().astype(np.float64) for k, v in out["grads"].items()}
        for k, v in ggpu.items():
            assert rel_inf(v, gr[k] + mar_gr[k]) < TOL, (step, k)
        params, ostate = O.adam_update(params, ggpu, ostate, step, 1e-2, 0.9, 0.99, 1e-6)
        for k, v in params.items():
            got = model.t[k].cpu().numpy()
            assert np.allclose(got, v, rtol=1e-5, atol=1e-6), (step, k)
