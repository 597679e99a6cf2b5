"""Pins of the oracle's zero-order (ES) gradient estimator (Sec. 2.2):
exact recovery of the gradient of a quadratic with an orthonormal antithetic
sample set, the plain estimator's exact value for a linear function, a library
matrix product as a special case, and convergence to the smoothed gradient."""
import numpy as np

import oracle
from workloads import normal


def _quadratic(n, seed):
    rng = np.random.default_rng(seed)
    A = rng.normal(size=(n, n))
    A = A @ A.T / n
    b = rng.normal(size=n)
    return (lambda x: 0.5 * x @ A @ x + b @ x + 3.0), (lambda x: A @ x + b)


def test_antithetic_recovers_quadratic_gradient_exactly():
    # f(t + s z) - f(t - s z) = 2 s grad(t).z for any quadratic, and with the
    # sample set z_i = sqrt(n) e_i, (1/N) sum z_i z_i^T = I: the estimate is
    # exactly grad(t), whatever s.
    n = 16
    f, grad = _quadratic(n, 1)
    theta = normal(n, 1.0, "es", "p0").astype(np.float64)
    Z = np.sqrt(n) * np.eye(n)
    for sigma in (1e-2, 0.3, 2.0):
        pts = oracle.es_perturb(theta, Z, sigma, antithetic=True)
        fv = np.array([f(x) for x in pts])
        w = fv[:n] - fv[n:]
        g = oracle.es_estimate(Z, w, 1.0 / (2 * n * sigma))
        assert np.max(np.abs(g - grad(theta))) < 1e-10 * np.max(np.abs(grad(theta)))


def test_plain_estimator_linear_function_closed_form():
    # for f(x) = a.x + c the plain estimate is (1/(N s)) sum_i (a.(t + s z_i) + c) z_i
    #   = (a.t + c)/(N s) sum_i z_i + (1/N) sum_i (a.z_i) z_i,  written out with numpy
    n, N, sigma = 40, 25, 0.1
    a = normal(n, 1.0, "es", "grad").astype(np.float64)
    theta = normal(n, 1.0, "es", "p0", 2).astype(np.float64)
    Z = np.stack([normal(n, 1.0, "es", "misc", 10 + i) for i in range(N)]).astype(np.float64)
    pts = oracle.es_perturb(theta, Z, sigma)
    assert np.allclose(pts, theta + sigma * Z, rtol=0, atol=1e-15)
    fv = pts @ a + 0.5
    g = oracle.es_estimate(Z, fv, 1.0 / (N * sigma))
    expect = (a @ theta + 0.5) / (N * sigma) * Z.sum(0) + (Z @ a) @ Z / N
    assert np.max(np.abs(g - expect)) < 1e-11 * np.max(np.abs(expect))


def test_estimate_is_a_weighted_row_sum():
    # special case that reduces to a library routine: scale * (w @ Z)
    N, n = 37, 1001
    Z = np.stack([normal(n, 1.0, "es", "misc", 100 + i) for i in range(N)]).astype(np.float64)
    w = normal(N, 3.0, "es", "cot_p").astype(np.float64)
    g = oracle.es_estimate(Z, w, 0.25)
    assert np.max(np.abs(g - 0.25 * (w @ Z))) <= 1e-13 * np.max(oracle.es_estimate_mag(Z, w, 0.25))
    assert np.all(np.abs(g) <= oracle.es_estimate_mag(Z, w, 0.25) * (1 + 1e-12))


def test_antithetic_estimate_converges_to_smoothed_gradient():
    # for a quadratic the smoothed gradient equals the gradient; with Gaussian
    # samples the antithetic estimate is unbiased with error ~ 1/sqrt(N)
    n, N, sigma = 8, 20000, 0.05
    f, grad = _quadratic(n, 3)
    theta = normal(n, 1.0, "es", "p0", 3).astype(np.float64)
    Z = np.random.default_rng(5).normal(size=(N, n))
    pts = oracle.es_perturb(theta, Z, sigma, antithetic=True)
    fv = np.array([f(x) for x in pts])
    g = oracle.es_estimate(Z, fv[:N] - fv[N:], 1.0 / (2 * N * sigma))
    err = np.linalg.norm(g - grad(theta)) / np.linalg.norm(grad(theta))
    assert err < 5 * np.sqrt(n / N) * 3
