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


# ------------------------------------------------------------------ seeded noise
# The noise is drawn from Philox-4x64-10 through the Box-Muller transform.  The
# generator is pinned bit for bit to numpy's independent implementation, the
# transform to its closed-form values, and the composed noise to the normal
# distribution and to the structure a counter-based design guarantees.

def _numpy_philox_block(counter, key):
    """numpy's Philox advances its 256-bit counter before each block, so the
    block at counter c is its first output when started at c - 1."""
    c = [int(x) for x in counter]
    v = (c[0] | c[1] << 64 | c[2] << 128 | c[3] << 192) - 1
    start = np.array([(v >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    gen = np.random.Philox(counter=start, key=np.array(key, dtype=np.uint64))
    return gen.random_raw(4).astype(np.uint64)


def test_philox_matches_numpy_bit_for_bit():
    rng = np.random.default_rng(2211)
    cases = [([1, 0, 0, 0], [0, 0]), ([0, 1, 0, 0], [0, 0]), ([0, 0, 0, 1], [2**64 - 1, 2**64 - 1]),
             ([2**64 - 1, 2**64 - 1, 2**64 - 1, 2**64 - 1], [12345, 67890])]
    for _ in range(200):
        cases.append(([int(x) for x in rng.integers(0, 2**64, size=4, dtype=np.uint64)],
                      [int(x) for x in rng.integers(0, 2**64, size=2, dtype=np.uint64)]))
    for ctr, key in cases:
        assert np.array_equal(oracle.philox4x64_10(ctr, key), _numpy_philox_block(ctr, key)), (ctr, key)
    # consecutive blocks of one numpy stream are consecutive counters (with the
    # carry from word 0 into word 1)
    gen = np.random.Philox(counter=np.array([2**64 - 3, 5, 0, 0], dtype=np.uint64),
                           key=np.array([7, 9], dtype=np.uint64))
    raw = gen.random_raw(16).astype(np.uint64).reshape(4, 4)
    for b, ctr in enumerate(([2**64 - 2, 5, 0, 0], [2**64 - 1, 5, 0, 0], [0, 6, 0, 0], [1, 6, 0, 0])):
        assert np.array_equal(oracle.philox4x64_10(ctr, [7, 9]), raw[b]), b


def _word(lo, hi):
    return (int(hi) << 32) | int(lo)


def test_box_muller_closed_forms():
    # u1 = 1 gives r = 0: both normals are exactly zero
    assert oracle.box_muller(_word(0xFFFFFFFF, 0x12345678)) == (0.0, 0.0)
    for k in (1, 2, 7, 24):
        lo = ((1 << (24 - k)) - 1) << 8  # u1 = 2^-k exactly
        r = np.sqrt(2.0 * k * np.log(2.0))
        for hi, za, zb in ((0, r, 0.0),                      # u2 = 0
                           (1 << 29, r / np.sqrt(2), r / np.sqrt(2)),  # u2 = 1/8
                           (1 << 30, 0.0, r),                # u2 = 1/4
                           (1 << 31, -r, 0.0),               # u2 = 1/2
                           (3 << 30, 0.0, -r)):              # u2 = 3/4
            ga, gb = oracle.box_muller(_word(lo, hi))
            assert abs(ga - za) <= 1e-14 * r and abs(gb - zb) <= 1e-14 * r, (k, hi, ga, gb, za, zb)
            # the low 8 bits of each half do not enter the 24-bit uniforms
            assert oracle.box_muller(_word(lo | 0xFF, hi | 0xFF)) == (ga, gb)


def test_gaussian_noise_is_standard_normal():
    from scipy import stats
    N, n = 64, (1 << 14) + 5
    z = oracle.es_gaussian_noise(N, n, 20221112).reshape(-1)
    M = z.size
    assert abs(z.mean()) < 5 / np.sqrt(M)
    assert abs(z.var() - 1.0) < 5 * np.sqrt(2.0 / M)
    assert stats.kstest(z, "norm").pvalue > 1e-4
    # the two normals of one word, and neighbouring words, are uncorrelated
    pairs = z[: M // 2 * 2].reshape(-1, 2)
    assert abs(np.corrcoef(pairs[:, 0], pairs[:, 1])[0, 1]) < 5 / np.sqrt(M / 2)
    assert abs(np.corrcoef(z[:-2], z[2:])[0, 1]) < 5 / np.sqrt(M)
    # the tails: P(|z| > 3) = 0.0026998
    assert abs(np.mean(np.abs(z) > 3.0) - 0.0026998) < 5 * np.sqrt(0.0027 / M)


def test_gaussian_noise_is_a_function_of_seed_sample_and_element():
    a = oracle.es_gaussian_noise(9, 101, 5)
    assert np.array_equal(oracle.es_gaussian_noise(9, 37, 5), a[:, :37])   # element j does not depend on n
    assert np.array_equal(oracle.es_gaussian_noise(4, 101, 5), a[:4])     # sample i does not depend on N
    b = oracle.es_gaussian_noise(9, 101, 6)
    assert not np.any(a == b)
    assert not np.any(a[0] == a[1])


def test_weights_recover_linear_and_quadratic_gradients_exactly():
    # with the symmetric sample set {+sqrt(n) e_j} u {-sqrt(n) e_j}, sum_i z_i = 0
    # and (1/N) sum_i z_i z_i^T = I, so each method's weights and scale must
    # return the gradient of a linear function exactly, and antithetic that of
    # a quadratic
    n = 12
    a = normal(n, 1.0, "es", "grad", 7).astype(np.float64)
    theta = normal(n, 1.0, "es", "p0", 7).astype(np.float64)
    Z = np.sqrt(n) * np.concatenate([np.eye(n), -np.eye(n)])
    N = Z.shape[0]
    lin = lambda x: x @ a + 0.75  # noqa: E731
    f_quad, grad_quad = _quadratic(n, 9)
    for sigma in (1e-2, 0.5):
        plus = oracle.es_perturb(theta, Z, sigma, antithetic=True)
        for method, f, want in (("plain", lin, a), ("baseline", lin, a), ("antithetic", lin, a),
                                ("antithetic", f_quad, grad_quad(theta))):
            fv = np.array([f(x) for x in (plus if method == "antithetic" else plus[:N])])
            w, scale = oracle.es_weights(fv, method, sigma, f0=f(theta))
            g = oracle.es_estimate(Z, w, scale)
            assert np.max(np.abs(g - want)) < 1e-9 * np.max(np.abs(want)), (method, sigma)
    # baseline and plain differ by the f0 term only
    fv = np.array([lin(x) for x in oracle.es_perturb(theta, Z, 0.1)])
    assert np.allclose(oracle.es_weights(fv, "baseline", 0.1, f0=2.0)[0], fv - 2.0, rtol=0, atol=0)
    assert oracle.es_weights(fv, "plain", 0.1)[1] == 1.0 / (N * 0.1)
    assert oracle.es_weights(np.concatenate([fv, fv]), "antithetic", 0.1)[1] == 1.0 / (2 * N * 0.1)


def test_noise_radius_is_the_pair_radius():
    # r^2 = za^2 + zb^2 for the two normals of one word, and |z| <= r
    N, n = 5, 64
    z = oracle.es_gaussian_noise(N, n, 77)
    r = oracle.es_gaussian_noise_radius(N, n, 77)
    assert np.allclose(r[:, 0::2] ** 2, z[:, 0::2] ** 2 + z[:, 1::2] ** 2, rtol=1e-13, atol=0)
    assert np.array_equal(r[:, 0::2], r[:, 1::2])
    assert np.all(np.abs(z) <= r * (1 + 1e-15))
    assert np.array_equal(oracle.es_gaussian_noise_radius(N, 13, 77), r[:, :13])


def test_noise_at_chosen_columns_is_the_same_noise():
    N, n, seed = 3, 77, 2**63 + 5
    z = oracle.es_gaussian_noise(N, n, seed)
    r = oracle.es_gaussian_noise_radius(N, n, seed)
    cols = [76, 0, 9, 8, 7, 40, 9]
    zc, rc = oracle.es_gaussian_noise_cols(N, cols, seed)
    assert np.array_equal(zc, z[:, cols]) and np.array_equal(rc, r[:, cols])
