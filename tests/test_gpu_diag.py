"""Diagonal complex SSM scans on the GPU against the complex128 oracle (through the C ABI)."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from gpu_util import rel_inf, say, tie_band_check

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
@pytest.mark.parametrize("rev,tr", [(False, False), (True, True), (False, True), (True, False)])
def test_deer_scan_diag(B, T, M, rev, tr):
    """Both directions with lambda or its transpose conj(lambda) (C read as R^2)."""
    lam, b = _rand(B, T, M, B * T + M)
    say("deer_scan diag", B, T, M, rev, tr)
    y = D.deer_scan(D._b.DEER_SCAN_DIAG_C64, torch.tensor(lam), torch.tensor(b), reverse=rev, transpose=tr)
    # the oracle's reverse scan multiplies by conj(lam); the forward one by lam
    lop = lam if rev == tr else np.conj(lam)
    ref = O.diag_scan_reverse(lop, b) if rev else O.diag_scan(lop, b)
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


@pytest.mark.parametrize("B,T,M,K", [(1, 1, 1, 1), (1, 5, 3, 2), (2, 511, 16, 3), (1, 1025, 17, 4),
                                     (3, 2049, 64, 3), (2, 5000, 70, 1), (1, 70000, 8, 2)])
def test_diag_fused_projection_and_fused_gradients(B, T, M, K):
    """Forward scan with b_t = Bc x_{t-1} formed on the fly (segment path), then the reverse
    scan of a random cotangent with dlam and dBc accumulated inside it; with and without the
    adjoint itself stored."""
    rng = np.random.default_rng(B * T + M + K)
    lam = (rng.uniform(0.9, 0.999, M) * np.exp(1j * rng.uniform(0, np.pi / 10, M))).astype(np.complex64)
    Bc = ((rng.standard_normal((M, K)) + 1j * rng.standard_normal((M, K))) / np.sqrt(2 * K)).astype(np.complex64)
    x = rng.standard_normal((B, T + 1, K)).astype(np.float32)
    m = {"kind": "diag_ssm", "lam": lam, "Bc": Bc}
    say("deer_solve diag fused", B, T, M, K)
    res = D.deer_solve(m, x, 0.0, 0)
    h_ref = O.diag_scan(lam, O.diag_ssm_inputs({"Bc": Bc}, x))
    assert rel_inf(_c(res["z"].cpu().numpy()), h_ref) < TOL
    g = (rng.standard_normal((B, T, M)) + 1j * rng.standard_normal((B, T, M))).astype(np.complex64)
    gt = torch.tensor(np.stack([g.real, g.imag], -1))
    say("deer_adjoint diag fused grads", B, T, M, K)
    out = D.deer_adjoint(m, x, res["z"], 0.0, 0, g=gt)
    a_ref = O.diag_scan_reverse(lam, g)
    assert rel_inf(_c(out["lam"].cpu().numpy()), a_ref) < TOL
    gr = O.diag_ssm_param_grads(a_ref, h_ref, x)
    dl = out["grads"]["lam"].cpu().numpy()
    dB = out["grads"]["Bc"].cpu().numpy()
    assert rel_inf(_c(dl), gr["lam"]) < TOL
    assert rel_inf(_c(dB), gr["Bc"]) < TOL
    # gradients only: the segment walk (one read of g and h, carries applied afterwards)
    out2 = D.deer_adjoint(m, x, res["z"], 0.0, 0, g=gt, want_lam=False)
    assert out2["lam"] is None
    assert rel_inf(_c(out2["grads"]["lam"].cpu().numpy()), gr["lam"]) < TOL
    assert rel_inf(_c(out2["grads"]["Bc"].cpu().numpy()), gr["Bc"]) < TOL


@pytest.mark.parametrize("B,T,M,K", [(2, 4096, 64, 3), (1, 70000, 8, 2), (3, 1537, 33, 4), (1, 600, 64, 1),
                                     (2, 512, 16, 3), (1, 513, 64, 3)])
@pytest.mark.parametrize("mfma", ["1", "0"])
def test_diag_forward_segment_aggregates(B, T, M, K, mfma, monkeypatch):
    """Forward scan: the segment aggregates from the matrix-core product of the powers
    lam^{63-k} with the transposed inputs (combined with lam^{64 (7 - a)} Bc), and from the
    lane-per-channel walk, both against the sequential oracle; full and partial last segments,
    |lam| close to 1."""
    monkeypatch.setenv("DEER_DIAG_AGG_MFMA", mfma)
    rng = np.random.default_rng(7 * T + M + K)
    lam = (rng.uniform(0.99, 0.9999, M) * np.exp(1j * rng.uniform(0, np.pi / 4, M))).astype(np.complex64)
    Bc = ((rng.standard_normal((M, K)) + 1j * rng.standard_normal((M, K))) / np.sqrt(2 * K)).astype(np.complex64)
    x = rng.standard_normal((B, T + 1, K)).astype(np.float32)
    m = {"kind": "diag_ssm", "lam": lam, "Bc": Bc}
    say("deer_solve diag segment aggregates", B, T, M, K, mfma)
    res = D.deer_solve(m, x, 0.0, 0)
    h_ref = O.diag_scan(lam, O.diag_ssm_inputs({"Bc": Bc}, x))
    assert rel_inf(_c(res["z"].cpu().numpy()), h_ref) < TOL


@pytest.mark.parametrize("B,T,M,K,g_real,seg", [(1, 1, 1, 1, True, 0), (1, 5, 3, 2, False, 0),
                                                (2, 511, 16, 3, True, 64), (1, 1025, 17, 4, False, 128),
                                                (3, 2049, 64, 3, True, 192), (2, 5000, 70, 1, True, 0),
                                                (1, 70000, 8, 2, False, 0), (2, 4097, 130, 3, True, 256),
                                                (1, 64, 64, 3, True, 64), (1, 65, 64, 3, False, 64)])
def test_diag_gradients_segment_walk(B, T, M, K, g_real, seg, monkeypatch):
    """Reverse scan with dlam and dBc when the adjoint itself is not stored: every segment is
    walked once from a zero state and the carries are applied to its sums afterwards.  Short
    forced segment lengths give many segments, a partial last segment and segments shorter
    than a register batch; the cotangent is real (the read-out's dL/dRe h) or complex."""
    if seg:
        monkeypatch.setenv("DEER_DIAG_RSEG", str(seg))
    rng = np.random.default_rng(7 * B + T + M + K)
    lam = (rng.uniform(0.9, 0.999, M) * np.exp(1j * rng.uniform(0, np.pi / 10, M))).astype(np.complex64)
    Bc = ((rng.standard_normal((M, K)) + 1j * rng.standard_normal((M, K))) / np.sqrt(2 * K)).astype(np.complex64)
    x = rng.standard_normal((B, T + 1, K)).astype(np.float32)
    m = {"kind": "diag_ssm", "lam": lam, "Bc": Bc}
    say("deer_solve diag fused", B, T, M, K)
    res = D.deer_solve(m, x, 0.0, 0)
    h32 = _c(res["z"].cpu().numpy())
    if g_real:
        g = rng.standard_normal((B, T, M)).astype(np.float32)
        gt = torch.tensor(g)
    else:
        g = (rng.standard_normal((B, T, M)) + 1j * rng.standard_normal((B, T, M))).astype(np.complex64)
        gt = torch.tensor(np.stack([g.real, g.imag], -1))
    say("deer_adjoint diag segment walk", B, T, M, K, g_real, seg)
    out = D.deer_adjoint(m, x, res["z"], 0.0, 0, g=gt, want_lam=False)
    assert out["lam"] is None
    # the oracle reads the same float32 forward states the GPU reads
    a_ref = O.diag_scan_reverse(lam, g.astype(np.complex128))
    gr = O.diag_ssm_param_grads(a_ref, h32, x)
    assert rel_inf(_c(out["grads"]["lam"].cpu().numpy()), gr["lam"]) < TOL
    assert rel_inf(_c(out["grads"]["Bc"].cpu().numpy()), gr["Bc"]) < TOL


def _readout_params(M, H, No, rng):
    return {"Wa": (rng.standard_normal((H, M)) / np.sqrt(M)).astype(np.float32),
            "ca": (0.1 * rng.standard_normal(H)).astype(np.float32),
            "Wb": (rng.standard_normal((No, H)) / np.sqrt(H)).astype(np.float32),
            "cb": (0.1 * rng.standard_normal(No)).astype(np.float32)}


def _bits(words, H):
    w = words.astype(np.uint32)
    bits = (w[..., :, None] >> np.arange(32, dtype=np.uint32)) & 1
    return bits.reshape(w.shape[:-1] + (-1,))[..., :H].astype(bool)


@pytest.mark.parametrize("B,T,M,H,No", [(1, 1, 1, 1, 1), (2, 37, 64, 128, 3), (1, 1000, 17, 50, 2),
                                        (3, 5000, 64, 128, 4), (2, 300, 64, 16, 3), (1, 70, 40, 100, 1)])
def test_readout_loss_g_and_grads(B, T, M, H, No):
    """Read-out MLP on the matrix cores: the ReLU decisions equal the float64 ones outside a
    tie band; loss, g = dL/dRe h and the read-out gradients equal the float64 oracle taken
    with the GPU's decisions."""
    rng = np.random.default_rng(B * T + M + H + No)
    prm = _readout_params(M, H, No, rng)
    h = (rng.standard_normal((B, T, M)) + 1j * rng.standard_normal((B, T, M))).astype(np.complex64)
    x = rng.standard_normal((B, T + 1, No)).astype(np.float32)
    say("deer_readout_loss", B, T, M, H, No)
    out = D.deer_readout_loss(prm, torch.tensor(h), x, want_masks=True)
    got = _bits(out["masks"].cpu().numpy(), H)
    s = O.diag_ssm_readout_preactivation(prm, h)
    tie_band_check(got, s, 1e-5, "read-out masks")
    loss, g, gr = O.diag_ssm_loss_and_seed(prm, h, x, mask=got)
    assert abs(float(out["loss"].cpu()[0]) - loss) <= 1e-5 * abs(loss)
    assert rel_inf(out["g"].cpu().numpy(), g) < TOL
    for k in ("Wa", "ca", "Wb", "cb"):
        assert rel_inf(out["grads"][k].cpu().numpy(), gr[k]) < TOL, k
    # without gradients / masks / loss the cotangent is bit-identical
    out2 = D.deer_readout_loss(prm, torch.tensor(h), x, want_grads=False, want_loss=False)
    assert np.array_equal(out2["g"].cpu().numpy(), out["g"].cpu().numpy())


def test_diag_training_step_with_readout():
    """Workload-4 model at reduced T, the whole step: forward scan with the fused projection,
    read-out loss and cotangent, reverse scan of the real cotangent with dlam, dBc."""
    c = W.make_config(4, B=2, T=3000)
    p = c.params
    m = {"kind": "diag_ssm", "lam": p["lam"], "Bc": p["Bc"]}
    ro = {k: p[k] for k in ("Wa", "ca", "Wb", "cb")}
    say("diag step: solve")
    res = D.deer_solve(m, c.x, 0.0, 0)
    say("diag step: read-out")
    r = D.deer_readout_loss(ro, res["z"], c.x, want_masks=True)
    say("diag step: adjoint (real g)")
    out = D.deer_adjoint(m, c.x, res["z"], 0.0, 0, g=r["g"])
    h = O.diag_scan(p["lam"], O.diag_ssm_inputs(p, c.x))
    assert rel_inf(_c(res["z"].cpu().numpy()), h) < TOL
    mask = _bits(r["masks"].cpu().numpy(), p["Wa"].shape[0])
    loss, g, gr = O.diag_ssm_loss_and_seed(p, h, c.x, mask=mask)
    assert abs(float(r["loss"].cpu()[0]) - loss) <= 1e-5 * loss
    assert rel_inf(r["g"].cpu().numpy(), g) < TOL
    a = O.diag_scan_reverse(p["lam"], g.astype(np.complex128))
    assert rel_inf(_c(out["lam"].cpu().numpy()), a) < TOL
    pg = O.diag_ssm_param_grads(a, h, c.x)
    assert rel_inf(_c(out["grads"]["lam"].cpu().numpy()), pg["lam"]) < TOL
    assert rel_inf(_c(out["grads"]["Bc"].cpu().numpy()), pg["Bc"]) < TOL
    for k in ("Wa", "ca", "Wb", "cb"):
        assert rel_inf(r["grads"][k].cpu().numpy(), gr[k]) < TOL, k
