"""Robustness of the workspace contract and of the results, through the C ABI.

* NaN-poisoned workspace: every entry point is run with its workspace filled with 0xFF bytes
  (NaN as a float, -1 as an integer) and with a zero-filled one; the outputs must be equal bit for
  bit, so no kernel reads scratch it has not written in the same call.
* Bitwise rerun determinism: the same call twice gives the same bits.  The one exception is the
  reverse diagonal scan that stores the adjoint (decoupled look-back, whose combination order
  depends on timing): its adjoint is compared to float32 rounding instead.
"""
import ctypes

import numpy as np
import pytest

import workloads as W
from gpu_util import oracle_model, rel_inf, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402
from paper_2605_12683_amd import _binding as Bnd  # noqa: E402


def _ws(nbytes, fill):
    w = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")
    w.fill_(fill)
    return w


def _np(v):
    if isinstance(v, torch.Tensor):
        return v.detach().cpu().numpy()
    return np.asarray(v)


def _same_bits(a, b, what):
    assert set(a) == set(b), what
    for k in a:
        x, y = _np(a[k]), _np(b[k])
        assert x.shape == y.shape, (what, k)
        assert x.tobytes() == y.tobytes(), (what, k, float(np.abs(x.astype(np.float64) - y).max()))


def _ws_bytes(model, forcing_alpha, n, B, T, op, quasi=0, T_w=0, obs=None):
    lib = D.load()
    m = D._model(model)
    od = D._dev(obs)
    f = Bnd.deer_forcing(float(forcing_alpha), int(n), int(T_w), D._ptr(od))
    return lib.deer_workspace_bytes_ex(ctypes.byref(m.c), ctypes.byref(f), B, T, op, quasi)


def _plrnn_run(m, x, alpha, N, fill, *, fixed=0, quasi=False, obs=None):
    B, T = x.shape[0], x.shape[1] - 1
    q = 1 if quasi else 0
    ws_s = _ws(_ws_bytes(m, alpha, N, B, T, Bnd.DEER_OP_SOLVE, q, obs=obs), fill)
    ws_a = _ws(_ws_bytes(m, alpha, N, B, T, Bnd.DEER_OP_ADJOINT, q, obs=obs), fill)
    kw = {"obs": obs} if obs is not None else {}
    solve = D.deer_solve_quasi if quasi else D.deer_solve
    adjoint = D.deer_adjoint_quasi if quasi else D.deer_adjoint
    res = solve(m, x, alpha, N, tol=1e-5, fixed_iters=fixed, ws=ws_s, want_masks=True, **kw)
    adj = adjoint(m, x, res["z"], alpha, N, ws=ws_a, **kw)
    torch.cuda.synchronize()
    out = {"z": res["z"], "masks": res["masks"], "iters": np.array(res["iters"]), "lam": adj["lam"]}
    out.update({"g_" + k: v for k, v in adj["grads"].items()})
    return out


PLRNN_CASES = {
    "vanilla_M16_fused": lambda: (W.random_plrnn_case(16, 3, 4, 4096, 0.2, 11, w_norm=0.3, a_range=(0.3, 0.7)), {}),
    "vanilla_M64": lambda: (W.random_plrnn_case(64, 8, 2, 2048, 0.1, 12, w_norm=0.3, a_range=(0.3, 0.7)), {}),
    "vanilla_M3_small": lambda: (W.make_config(1), {"fixed": 5}),
    "shallow_M32_L64": lambda: (W.random_shplrnn_case(32, 64, 8, 2, 1024, 0.2, 13, w_norm=0.3,
                                                      a_range=(0.3, 0.65)), {}),
    # width 128: 188 chunks, carries in two levels (group maps composed on the matrix cores)
    "shallow_M128_L50": lambda: (W.random_shplrnn_case(128, 50, 3, 1, 1500, 0.15, 15, w_norm=0.3,
                                                       a_range=(0.3, 0.65)), {}),
    "quasi_M16": lambda: (W.random_plrnn_case(16, 3, 2, 512, 0.2, 14, w_norm=0.3, a_range=(0.3, 0.7)),
                          {"quasi": True}),
}


@pytest.mark.parametrize("name", list(PLRNN_CASES))
def test_poisoned_workspace_and_rerun_are_bitwise_equal(name):
    c, kw = PLRNN_CASES[name]()
    m = oracle_model(c)
    say("robust", name, "zero workspace")
    a = _plrnn_run(m, c.x, c.alpha, c.n_obs, 0, **kw)
    say("robust", name, "NaN-poisoned workspace")
    b = _plrnn_run(m, c.x, c.alpha, c.n_obs, 255, **kw)
    say("robust", name, "rerun")
    r = _plrnn_run(m, c.x, c.alpha, c.n_obs, 0, **kw)
    _same_bits(a, b, name + " poisoned")
    _same_bits(a, r, name + " rerun")
    assert np.isfinite(_np(a["z"])).all() and np.isfinite(_np(a["lam"])).all()


def test_observation_matrix_path_poisoned_and_rerun():
    c = W.random_plrnn_case(8, 3, 2, 600, 0.2, 15, w_norm=0.3, a_range=(0.3, 0.7))
    m = oracle_model(c)
    obs = (np.random.default_rng(16).standard_normal((3, 8)) / np.sqrt(8)).astype(np.float32)
    say("robust obs")
    a = _plrnn_run(m, c.x, c.alpha, 3, 0, obs=obs)
    b = _plrnn_run(m, c.x, c.alpha, 3, 255, obs=obs)
    r = _plrnn_run(m, c.x, c.alpha, 3, 0, obs=obs)
    _same_bits(a, b, "obs poisoned")
    _same_bits(a, r, "obs rerun")


def _diag_run(c, fill, want_lam):
    p = c.params
    model = D._Model({"kind": "diag_ssm", "lam": p["lam"], "Bc": p["Bc"]})
    readout = D._Readout({k: p[k] for k in ("Wa", "ca", "Wb", "cb")})
    B, T, M = c.B, c.T, c.M
    ws_s = _ws(D.deer_workspace_bytes(model, B, T, Bnd.DEER_OP_SOLVE), fill)
    ws_a = _ws(D.deer_workspace_bytes(model, B, T, Bnd.DEER_OP_ADJOINT), fill)
    ws_r = _ws(D.deer_readout_workspace_bytes(readout, B, T, M), fill)
    res = D.deer_solve(model, c.x, 0.0, 0, ws=ws_s)
    r = D.deer_readout_loss(readout, res["z"], c.x, ws=ws_r)
    adj = D.deer_adjoint(model, c.x, res["z"], 0.0, 0, g=r["g"], ws=ws_a, want_lam=want_lam)
    torch.cuda.synchronize()
    out = {"h": res["z"], "g": r["g"], "loss": r["loss"]}
    out.update({"rg_" + k: v for k, v in r["grads"].items()})
    out.update({"g_" + k: v for k, v in adj["grads"].items()})
    if want_lam:
        out["lam"] = adj["lam"]
    return out


def test_diag_ssm_poisoned_and_rerun():
    """Forward scan, read-out and the reverse scan with the gradients only: bitwise; the adjoint
    stored by the look-back scan: to rounding (its summation order depends on timing)."""
    c = W.make_config(4, B=2, T=20000)
    say("robust diag gradients only")
    a = _diag_run(c, 0, False)
    b = _diag_run(c, 255, False)
    r = _diag_run(c, 0, False)
    _same_bits(a, b, "diag poisoned")
    _same_bits(a, r, "diag rerun")
    say("robust diag with the adjoint stored")
    la = _diag_run(c, 0, True)
    lb = _diag_run(c, 255, True)
    for k in la:
        assert rel_inf(_np(lb[k]), _np(la[k])) < 1e-5, k


@pytest.mark.parametrize("M", [32, 128])
@pytest.mark.parametrize("rev,tr", [(False, False), (True, True)])
def test_dense_scan_poisoned_and_rerun(rev, tr, M):
    rng = np.random.default_rng(17)
    B, T = 2, 3000
    J = torch.tensor((rng.standard_normal((B, T, M, M)) * (0.45 / np.sqrt(M))).astype(np.float32), device="cuda")
    bb = torch.tensor(rng.standard_normal((B, T, M)).astype(np.float32), device="cuda")
    n = D.deer_scan_workspace_bytes(Bnd.DEER_SCAN_DENSE, B, T, M, reverse=rev, transpose=tr)
    say("robust dense scan", rev, tr, M)
    outs = [D.deer_scan(Bnd.DEER_SCAN_DENSE, J, bb, reverse=rev, transpose=tr, ws=_ws(n, f)) for f in (0, 255, 0)]
    torch.cuda.synchronize()
    _same_bits({"y": outs[0]}, {"y": outs[1]}, "scan poisoned")
    _same_bits({"y": outs[0]}, {"y": outs[2]}, "scan rerun")
