"""Pins the oracle's Kumaraswamy inverse-CDF sampler and its pathwise
derivatives against closed forms, library special cases and statistics."""
import numpy as np
import pytest
from scipy import special, stats

import oracle
from oracle.sampler import kumaraswamy_cdf, kumaraswamy_icdf, pathwise, uniform_from_words

RNG = np.random.default_rng(7)


def _grid_u(n):
    w = RNG.integers(0, 2**32, n, dtype=np.uint64).astype(np.uint32)
    return uniform_from_words(w)


def test_cdf_round_trip():
    u = np.concatenate([_grid_u(20000), [2.0**-24, 1 - 2.0**-24, 0.5]])
    a = RNG.uniform(1, 6, u.size)
    b = RNG.uniform(1, 6, u.size)
    x = kumaraswamy_icdf(u, a, b)
    assert np.all((x > 0) & (x < 1))
    assert np.max(np.abs(kumaraswamy_cdf(x, a, b) - u)) < 1e-12


def test_unit_shape_is_identity():
    u = _grid_u(5000)
    assert np.array_equal(kumaraswamy_icdf(u, 1.0, 1.0), u)


@pytest.mark.parametrize("b", [1.0, 1.7, 3.0, 5.5])
def test_a1_is_beta_1_b(b):
    u = _grid_u(3000)
    np.testing.assert_allclose(kumaraswamy_icdf(u, 1.0, b), stats.beta.ppf(u, 1.0, b), rtol=1e-10, atol=1e-14)


@pytest.mark.parametrize("a", [1.0, 2.5, 4.0, 6.0])
def test_b1_is_beta_a_1(a):
    u = _grid_u(3000)
    np.testing.assert_allclose(kumaraswamy_icdf(u, a, 1.0), stats.beta.ppf(u, a, 1.0), rtol=1e-10, atol=1e-14)


def test_median():
    for a, b in [(2, 5), (1.5, 3), (5.9, 1.1), (1.0, 6.0)]:
        assert abs(kumaraswamy_icdf(0.5, a, b) - (1 - 2.0 ** (-1.0 / b)) ** (1.0 / a)) < 1e-15


@pytest.mark.parametrize("theta", [(2.0, 5.0, 1.5, 3.0), (4.2, 1.3, 1.1, 5.7)])
def test_moments_and_ks_from_philox_draws(theta):
    E = 200_000
    s = oracle.sample(np.array([theta]), E, seed=11, return_all=True)
    x = s["x"]
    for j in range(2):
        a, b = theta[2 * j], theta[2 * j + 1]
        for n in (1, 2, 3):
            m = b * special.beta(1 + n / a, b)
            xs = x[:, j] ** n
            assert abs(xs.mean() - m) < 5 * xs.std() / np.sqrt(E), (j, n)
        ks = stats.kstest(x[:, j], lambda t: kumaraswamy_cdf(t, a, b))
        assert ks.pvalue > 1e-4


def test_theta_index_and_word_index_mapping():
    theta = np.array([[1.0, 1.0, 2.0, 3.0], [3.0, 2.0, 1.0, 1.0]])
    E = 50
    s = oracle.sample(theta, E, seed=5, counter_base=1000, return_all=True)
    ids = 1000 + np.arange(2 * E, dtype=np.uint64)
    w = oracle.event_words(5, ids)
    u = uniform_from_words(w)
    # event k of sample i uses theta[i]; coordinate j uses word j
    np.testing.assert_array_equal(s["x"][:E, 0], u[:E, 0])
    np.testing.assert_array_equal(s["x"][E:, 1], u[E:, 1])
    np.testing.assert_allclose(kumaraswamy_cdf(s["x"][:E, 1], 2, 3), u[:E, 1], atol=1e-13)
    np.testing.assert_allclose(kumaraswamy_cdf(s["x"][E:, 0], 3, 2), u[E:, 0], atol=1e-13)


def test_pathwise_vs_finite_differences():
    u = _grid_u(4000)
    u = u[(u > 1e-3) & (u < 1 - 1e-3)]      # float64 differences lose digits at the ends
    a = RNG.uniform(1, 6, u.size)
    b = RNG.uniform(1, 6, u.size)
    x = kumaraswamy_icdf(u, a, b)
    da, db = pathwise(x, a, b)
    h = 1e-6
    fa = (kumaraswamy_icdf(u, a + h, b) - kumaraswamy_icdf(u, a - h, b)) / (2 * h)
    fb = (kumaraswamy_icdf(u, a, b + h) - kumaraswamy_icdf(u, a, b - h)) / (2 * h)
    np.testing.assert_allclose(da, fa, rtol=1e-5, atol=1e-9)
    np.testing.assert_allclose(db, fb, rtol=1e-5, atol=1e-9)
    assert np.all(da >= 0) and np.all(db <= 0)


@pytest.mark.parametrize("u", [2.0**-24, 1e-5, 0.5, 1 - 1e-5, 1 - 2.0**-24])
def test_pathwise_vs_arbitrary_precision_derivative(u):
    """Edge cells of the u grid: derivatives of the quantile taken numerically in 40-digit arithmetic."""
    import mpmath
    mpmath.mp.dps = 40
    for a, b in [(1.0, 1.0), (6.0, 6.0), (1.0, 6.0), (6.0, 1.0), (3.3, 2.2)]:
        q = lambda aa, bb: (1 - (1 - mpmath.mpf(u)) ** (1 / bb)) ** (1 / aa)
        ea = float(mpmath.diff(lambda t: q(t, b), a))
        eb = float(mpmath.diff(lambda t: q(a, t), b))
        da, db = pathwise(kumaraswamy_icdf(u, a, b), a, b)
        assert abs(da - ea) <= 1e-7 * abs(ea) and abs(db - eb) <= 1e-7 * abs(eb), (a, b)


def test_pathwise_vs_chain_rule_form():
    u = _grid_u(4000)
    a = RNG.uniform(1, 6, u.size)
    b = RNG.uniform(1, 6, u.size)
    x = kumaraswamy_icdf(u, a, b)
    da, db = pathwise(x, a, b)
    ell = np.log1p(-u)
    s = np.exp(ell / b)
    g = -np.expm1(ell / b)
    lam = np.log(g)
    np.testing.assert_allclose(da, -x * lam / a**2, rtol=1e-9, atol=1e-15)
    np.testing.assert_allclose(db, x * s * ell / (a * b**2 * g), rtol=1e-7, atol=1e-15)


def test_pathwise_unit_theta_closed_form():
    u = _grid_u(4000)
    da, db = pathwise(u, 1.0, 1.0)
    np.testing.assert_allclose(da, -u * np.log(u), rtol=1e-12)
    np.testing.assert_allclose(db, (1 - u) * np.log1p(-u), rtol=1e-9)


@pytest.mark.parametrize("theta", [(2.0, 5.0, 1.5, 3.0), (1.2, 1.4, 5.0, 2.2)])
def test_pathwise_mean_is_derivative_of_mean(theta):
    """E[dx/dtheta] = d E[x] / dtheta, with E[x] = b B(1 + 1/a, b); the
    derivative via digamma: dm/da = -m/a^2 [psi(1+1/a) - psi(1+b+1/a)],
    dm/db = m [1/b + psi(b) - psi(1+b+1/a)] with psi(b) - psi(1+b) = -1/b folded in."""
    E = 200_000
    s = oracle.sample(np.array([theta]), E, seed=21, return_all=True)
    for j in range(2):
        a, b = theta[2 * j], theta[2 * j + 1]
        m = b * special.beta(1 + 1 / a, b)
        dma = -(m / a**2) * (special.digamma(1 + 1 / a) - special.digamma(1 + b + 1 / a))
        dmb = m * (1.0 / b + special.digamma(b) - special.digamma(1 + b + 1 / a))
        # cross-check the digamma forms by differencing the closed-form mean
        h = 1e-6
        mean = lambda aa, bb: bb * special.beta(1 + 1 / aa, bb)
        assert abs(dma - (mean(a + h, b) - mean(a - h, b)) / (2 * h)) < 1e-7
        assert abs(dmb - (mean(a, b + h) - mean(a, b - h)) / (2 * h)) < 1e-7
        for est, ref in ((s["dxda"][:, j], dma), (s["dxdb"][:, j], dmb)):
            assert abs(est.mean() - ref) < 5 * est.std() / np.sqrt(E)


def test_hd8_features_and_jacobian():
    x = kumaraswamy_icdf(_grid_u(600).reshape(200, 3), 2.0, 3.0)
    f = oracle.features_hd8(x)
    np.testing.assert_allclose(np.exp(f[:, 6]), x[:, 0], rtol=1e-14)
    np.testing.assert_allclose(-np.expm1(f[:, 7]), x[:, 2], rtol=1e-12)
    np.testing.assert_allclose(f[:, 3], x[:, 0] * x[:, 1], rtol=1e-15)
    J = oracle.features_hd8_jacobian(x)
    h = 1e-7
    for j in range(3):
        e = np.zeros(3)
        e[j] = h
        fd = (oracle.features_hd8(x + e) - oracle.features_hd8(x - e)) / (2 * h)
        np.testing.assert_allclose(J[:, :, j], fd, rtol=1e-6, atol=1e-8)
