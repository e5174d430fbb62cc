"""Diagonal complex SSM scans on the GPU against the complex128 oracle (through the C ABI)."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from gpu_util import rel_inf, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402

TOL = 1e-4


def _c(a):
    return np.asarray(a[..., 0], np.float64) + 1j * np.asarray(a[..., 1], np.float64)


def _rand(B, T, M, seed):
    rng = np.random.default_rng(seed)
    lam = (rng.uniform(0.9, 0.999, M) * np.exp(1j * rng.uniform(0, np.pi / 10, M))).astype(np.complex64)
    b = (rng.standard_normal((B, T, M)) + 1j * rng.standard_normal((B, T, M))).astype(np.complex64)
    return lam, b


@pytest.mark.parametrize("B,T,M", [(1, 1, 1), (1, 5, 3), (2, 1023, 16), (1, 1024, 17), (3, 1025, 64),
                                   (2, 5000, 40), (1, 70000, 8)])
@pytest.mark.parametrize("rev", [False, True])
def test_deer_scan_diag(B, T, M, rev):
    lam, b = _rand(B, T, M, B * T + M)
    say("deer_scan diag", B, T, M, rev)
    y = D.deer_scan(D._b.DEER_SCAN_DIAG_C64, torch.tensor(lam), torch.tensor(b), reverse=rev)
    ref = O.diag_scan_reverse(lam, b) if rev else O.diag_scan(lam, b)
    assert rel_inf(_c(y.cpu().numpy()), ref) < TOL


def test_diag_solve_fused_projection_and_adjoint():
    """Workload-4 model at reduced T: fused b_t = Bc x_{t-1}, forward scan, reverse scan of a
    given cotangent, dlam and dBc."""
    c = W.make_config(4, B=2, T=5000)
    p = c.params
    m = {"kind": "diag_ssm", "lam": p["lam"], "Bc": p["Bc"]}
    say("deer_solve diag fused")
    res = D.deer_solve(m, c.x, 0.0, 0)
    h = _c(res["z"].cpu().numpy())
    ref = O.diag_ssm_step(p, c.x)
    assert rel_inf(h, ref["h"]) < TOL
    g = ref["g"].astype(np.complex64)          # dL/dRe h from the oracle's read-out
    say("deer_adjoint diag")
    hd = res["z"]
    out = D.deer_adjoint(m, c.x, hd, 0.0, 0, g=torch.tensor(g))
    assert rel_inf(_c(out["lam"].cpu().numpy()), ref["a"]) < TOL
    assert rel_inf(_c(out["grads"]["lam"].cpu().numpy()), ref["grads"]["lam"]) < TOL
    assert rel_inf(_c(out["grads"]["Bc"].cpu().numpy()), ref["grads"]["Bc"]) < TOL
