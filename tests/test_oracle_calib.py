"""Pins of the ridge calibration (App. A) against library solvers and
closed-form cases."""
import numpy as np

import workloads as W
from oracle import calib, method


def _stats_from(Z, y, chunks=4):
    st = calib.ExpertStats(Z.shape[1])
    for part in np.array_split(np.arange(len(y)), chunks):
        st.update(Z[part], y[part])
    return st


def test_ridge_small_lambda_equals_least_squares():
    g = np.random.default_rng(0)
    n, d = 400, 16
    Z = g.standard_normal((n, d))
    y = Z @ g.standard_normal(d) + 0.3 + 0.1 * g.standard_normal(n)
    st = _stats_from(Z, y)
    a, b = calib.ridge_direct(st, 1e-10)
    X = np.hstack([Z, np.ones((n, 1))])
    coef, *_ = np.linalg.lstsq(X, y, rcond=None)
    # the Gram is held in fp32 (App. A), so agreement is to fp32 level
    np.testing.assert_allclose(a, coef[:d], rtol=1e-4, atol=1e-5)
    assert abs(b - coef[d]) < 1e-4


def test_eig_path_equals_direct_solve_for_every_lambda():
    g = np.random.default_rng(1)
    n, d = 300, 24
    Z = g.standard_normal((n, d))
    y = Z @ g.standard_normal(d) + g.standard_normal(n)
    st = _stats_from(Z, y)
    for lam in calib.LAMBDAS:
        f = calib.ridge_fit(st, lambdas=[lam])
        a, b = calib.ridge_direct(st, lam)
        np.testing.assert_allclose(f["a"], a, rtol=1e-8, atol=1e-10)
        assert abs(f["b_raw"] - b) < 1e-8


def test_streaming_equals_batch_statistics():
    g = np.random.default_rng(2)
    Z = g.standard_normal((250, 8))
    y = g.standard_normal(250)
    s1, s7 = _stats_from(Z, y, 1), _stats_from(Z, y, 7)
    assert s1.n == s7.n == 250
    np.testing.assert_allclose(s1.sz, s7.sz, rtol=1e-12)
    np.testing.assert_allclose(s1.q, s7.q, rtol=1e-12)
    np.testing.assert_allclose(s1.G, s7.G, rtol=1e-5)


def test_noise_free_linear_target_is_recovered():
    g = np.random.default_rng(3)
    n, d = 500, 10
    Z = g.standard_normal((n, d))
    a_true = g.standard_normal(d)
    y = Z @ a_true - 1.5
    f = calib.ridge_fit(_stats_from(Z, y))
    assert f["lam"] == calib.LAMBDAS[0]          # evidence prefers no shrinkage
    np.testing.assert_allclose(f["a"], a_true, rtol=1e-4, atol=1e-5)
    assert abs(f["b"] - (-1.5)) < 1e-4            # zero residual: no correction


def test_pure_noise_target_is_shrunk():
    g = np.random.default_rng(4)
    n, d = 200, 40
    Z = g.standard_normal((n, d)) * 0.05
    y = g.standard_normal(n)
    f = calib.ridge_fit(_stats_from(Z, y))
    assert f["lam"] >= 1.0
    assert np.linalg.norm(f["a"]) < 5.0


def test_lognormal_bias_correction_restores_mean_energy():
    # log-energy with Gaussian residual: exp(b) must match the mean energy
    g = np.random.default_rng(5)
    n, d = 20000, 4
    Z = g.standard_normal((n, d)) * 0.01
    s = 0.5
    y = 2.0 + s * g.standard_normal(n)
    f = calib.ridge_fit(_stats_from(Z, y))
    mean_energy = np.mean(np.exp(y))
    assert abs(np.exp(f["b"]) / mean_energy - 1) < 0.02


def test_tiny_layer_fit_runs_and_predicts_positive_costs():
    inp = W.layer_inputs("tiny")
    sh = inp["shape"]
    ex = method.Experts(inp["w13"], inp["w2"], False)
    z = W.calibration_tokens(sh)
    A, b, info = calib.fit_predictor(z, inp["w_router"], inp["b_router"],
                                     sh.K, ex)
    assert A.shape == (16, 256) and b.shape == (16,)
    assert sum(i["n"] for i in info) == 2 * len(z)
    assert np.all(np.isfinite(A)) and np.all(np.isfinite(b))
