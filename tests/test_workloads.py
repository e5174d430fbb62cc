"""The seeded input generators: shapes, determinism and the stated recipe."""
import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("i", [1, 2, 3, 4, 5])
def test_config_shapes_and_dtypes(i):
    c = W.make_config(i, B=2, T=300)
    assert c.x.shape == (2, 301, c.n_obs) and c.x.dtype == np.float32
    for v in c.params.values():
        assert v.dtype in (np.float32, np.complex64)
    if c.kind == "plrnn":
        assert c.params["W"].shape == (c.M, c.M)
    if c.kind == "shplrnn":
        assert c.params["W1"].shape == (c.M, c.L) and c.params["W2"].shape == (c.L, c.M)
    if c.kind == "diag_ssm":
        lam = c.params["lam"]
        assert np.all((np.abs(lam) >= 0.9 - 1e-6) & (np.abs(lam) <= 0.999 + 1e-6))
        assert np.all((np.angle(lam) >= -1e-7) & (np.angle(lam) <= np.pi / 10 + 1e-6))


def test_deterministic_and_sequence_independent():
    a = W.make_config(2, B=3, T=500)
    b = W.make_config(2, B=3, T=500)
    assert np.array_equal(a.x, b.x)
    for k in a.params:
        assert np.array_equal(a.params[k], b.params[k])
    c = W.make_config(2, B=1, T=500)
    assert np.array_equal(c.x[0], a.x[0])          # sequence b depends only on its own seed


def test_standardised_with_noise():
    c = W.make_config(2, B=2, T=20000)
    m = c.x.astype(np.float64).mean(axis=1)
    s = c.x.astype(np.float64).std(axis=1)
    assert np.all(np.abs(m) < 0.01) and np.all(np.abs(s - 1) < 0.01)


def test_drift_is_triangle_wave():
    tw = W.triangle_wave(20000, 5000.0, 0.0)
    assert np.isclose(tw.max(), 1.0) and np.isclose(tw.min(), -1.0, atol=1e-3)
    assert np.allclose(tw[:5000], tw[5000:10000])


def test_parameter_distributions():
    c = W.make_config(5)
    assert 0.5 <= c.params["A"].min() and c.params["A"].max() <= 0.9
    assert abs(c.params["W"].std() - 0.05) < 0.005
    c3 = W.make_config(3, B=1, T=10)
    assert abs(c3.params["W1"].std() - 1 / 16) < 0.005
