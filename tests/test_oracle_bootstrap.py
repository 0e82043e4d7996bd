"""Pins of the oracle's bootstrap draw (Sec. IV-B: sub-samples drawn with
replacement), by properties that do not retype its formula."""
import numpy as np
import pytest

import oracle
from oracle.bootstrap import bootstrap, bootstrap_indices, STREAM_BOOTSTRAP
from oracle.philox import philox4x32_10


def test_indices_in_range_and_deterministic():
    for n in (1, 2, 7, 1000, 12345, 1 << 32):
        idx = bootstrap_indices(n, 5000, seed=11, step=3)
        assert idx.dtype == np.int64 and idx.min() >= 0 and idx.max() < n
        assert np.array_equal(idx, bootstrap_indices(n, 5000, seed=11, step=3))


def test_power_of_two_rows_take_the_top_bits():
    """For n = 2^k the map floor(w n / 2^32) is the top k bits of the word."""
    n_out = 4096
    i = np.arange(n_out, dtype=np.uint64)
    ctr = np.stack([i, np.zeros_like(i), np.full_like(i, STREAM_BOOTSTRAP), np.full_like(i, 9)], axis=1)
    w0 = philox4x32_10(ctr, (5, 0))[:, 0]
    for k in (0, 1, 5, 16, 31):
        assert np.array_equal(bootstrap_indices(1 << k, n_out, seed=5, step=9), (w0 >> (32 - k)).astype(np.int64))


def test_with_replacement_statistics():
    """Drawing m = n rows with replacement leaves 1 - (1 - 1/n)^n of them
    distinct (-> 1 - 1/e); the count of one row is Binomial(m, 1/n)."""
    n = 200_000
    idx = bootstrap_indices(n, n, seed=2024, step=0)
    frac = np.unique(idx).size / n
    expect = 1 - (1 - 1 / n) ** n
    sd = np.sqrt(n * expect * (1 - expect)) / n     # a loose scale for the fluctuation
    assert abs(frac - expect) < 6 * sd
    counts = np.bincount(idx, minlength=n)
    # Binomial(n, 1/n) ~ Poisson(1): P(0) = e^-1, P(1) = e^-1, P(2) = e^-1/2
    for c, p in ((0, np.exp(-1)), (1, np.exp(-1)), (2, np.exp(-1) / 2)):
        f = np.mean(counts == c)
        assert abs(f - p) < 6 * np.sqrt(p * (1 - p) / n), (c, f, p)


def test_uniform_over_rows():
    n, m = 10, 200_000
    counts = np.bincount(bootstrap_indices(n, m, seed=1, step=1), minlength=n)
    chi2 = np.sum((counts - m / n) ** 2 / (m / n))
    assert chi2 < 40.0          # 9 degrees of freedom: P(chi2 > 40) < 1e-5


def test_steps_and_seeds_draw_independent_subsamples():
    n, m = 1 << 20, 50_000
    a = bootstrap_indices(n, m, seed=7, step=0)
    b = bootstrap_indices(n, m, seed=7, step=1)
    c = bootstrap_indices(n, m, seed=8, step=0)
    # agreement of two independent uniform draws over n rows: about m/n per position
    for x, y in ((a, b), (a, c), (b, c)):
        assert np.count_nonzero(x == y) < 10


def test_gather_returns_the_drawn_rows():
    rng = np.random.default_rng(0)
    data = rng.standard_normal((1000, 3))
    out, idx = bootstrap(data, 777, seed=3, step=5)
    assert out.shape == (777, 3) and np.array_equal(out, data[idx])


def test_rejects_too_many_rows():
    with pytest.raises(ValueError):
        bootstrap_indices((1 << 32) + 1, 10, seed=0, step=0)


def test_row_order_is_the_same_multiset():
    """Row order lists every drawn row as often as it was drawn, ascending, and
    its rows are the data rows of those indices (checked by counting, not by
    re-sorting)."""
    rng = np.random.default_rng(5)
    data = rng.standard_normal((997, 3))
    x, idx = oracle.bootstrap_row_order(data, 1500, 9, 2)
    _, draws = oracle.bootstrap(data, 1500, 9, 2)
    assert (np.diff(idx) >= 0).all()
    np.testing.assert_array_equal(np.bincount(idx, minlength=997), np.bincount(draws, minlength=997))
    np.testing.assert_array_equal(x, data[idx])
    # the batch mean, which is what a whole-batch loss sees, is unchanged
    np.testing.assert_allclose(x.mean(axis=0), data[draws].mean(axis=0), rtol=1e-12)
