"""deer_scan_noalloc (scratch in the library's static device array, no workspace argument)
against deer_scan with a caller-supplied workspace, through the C ABI: two calls in a row, the
second with a smaller input, in every layout and orientation; and sizes beyond the array are
refused before any device work."""
import numpy as np
import pytest

from gpu_util import rel_inf, say

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2605_12683_amd as D  # noqa: E402
from paper_2605_12683_amd import _binding as Bnd  # noqa: E402

TOL = 1e-4


def _inputs(layout, B, T, M, seed):
    rng = np.random.default_rng(seed)
    if layout == Bnd.DEER_SCAN_DENSE:
        J = (rng.standard_normal((B, T, M, M)) * (0.45 / np.sqrt(M))).astype(np.float32)
        b = rng.standard_normal((B, T, M)).astype(np.float32)
        return torch.tensor(J, device="cuda"), torch.tensor(b, device="cuda")
    lam = (rng.uniform(0.9, 0.999, M) * np.exp(1j * rng.uniform(0, np.pi / 10, M))).astype(np.complex64)
    b = (rng.standard_normal((B, T, M)) + 1j * rng.standard_normal((B, T, M))).astype(np.complex64)
    return D._dev(lam), D._dev(b)


@pytest.mark.parametrize("layout,sizes", [
    (Bnd.DEER_SCAN_DENSE, [(3, 3000, 32), (2, 700, 16)]),
    (Bnd.DEER_SCAN_DENSE, [(2, 2000, 64), (1, 33, 5)]),
    (Bnd.DEER_SCAN_DIAG_C64, [(2, 70000, 64), (1, 1025, 17)]),
])
@pytest.mark.parametrize("rev,tr", [(False, False), (True, True), (False, True), (True, False)])
def test_noalloc_scan_matches_workspace_scan(layout, sizes, rev, tr):
    for k, (B, T, M) in enumerate(sizes):
        J, b = _inputs(layout, B, T, M, 7 + 13 * k + B * T + M)
        need = D.deer_scan_workspace_bytes(layout, B, T, M, reverse=rev, transpose=tr)
        assert 0 < need <= D.deer_noalloc_scratch_bytes()
        say("deer_scan_noalloc", layout, B, T, M, rev, tr, "call", k + 1)
        y = torch.full_like(b, float("nan"))
        D.deer_scan_noalloc(layout, J, b, y, reverse=rev, transpose=tr)
        ref = D.deer_scan(layout, J, b, reverse=rev, transpose=tr)
        torch.cuda.synchronize()
        yn, rn = y.cpu().numpy().astype(np.float64), ref.cpu().numpy().astype(np.float64)
        assert np.isfinite(yn).all()
        assert rel_inf(yn, rn) <= TOL, (B, T, M, rel_inf(yn, rn))


def test_noalloc_refuses_sizes_beyond_the_scratch():
    B, T, M = 64, 1 << 16, 64
    need = D.deer_scan_workspace_bytes(Bnd.DEER_SCAN_DENSE, B, T, M)
    assert need > D.deer_noalloc_scratch_bytes()
    lib = D.load()
    say("deer_scan_noalloc refusal", B, T, M)
    tiny = torch.zeros(4, device="cuda")
    st = lib.deer_scan_noalloc(Bnd.DEER_SCAN_DENSE, 0, 0, B, T, M, D._ptr(tiny), D._ptr(tiny), D._ptr(tiny[2:]),
                               D._stream())
    assert st == Bnd.DEER_ERR_INVALID_ARG
    assert b"scratch" in lib.deer_last_error()
    assert lib.deer_scan_noalloc(7, 0, 0, 1, 10, 4, D._ptr(tiny), D._ptr(tiny), D._ptr(tiny[2:]),
                                 D._stream()) == Bnd.DEER_ERR_INVALID_ARG
