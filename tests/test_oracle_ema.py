"""Pins of the exponential moving sum of the counts and of the Dirichlet
resample from its fp64 totals (Sec. 4 footnote: datasets whose per-minibatch
counts are not kept)."""
import numpy as np
from scipy import stats

import oracle
from tests import brute
from workloads import koller


def test_ema_closed_form_and_limits():
    c = np.array([0, 1, 7, 1000, 123456], dtype=np.int64)
    for rho in (0.0, 0.5, 0.875, 0.999, 1.0):
        t = np.zeros(len(c), dtype=np.float64)
        for k in range(1, 41):
            oracle.ema(t, rho, c)
            # k equal minibatches from zero: c * (1 - rho^k) / (1 - rho) (= k * c at rho = 1)
            expect = c * (k if rho == 1.0 else (1.0 - rho ** k) / (1.0 - rho))
            np.testing.assert_allclose(t, expect, rtol=1e-12, atol=0)
    # rho = 0 keeps only the newest minibatch; rho = 1 is the plain running sum, exact in integers
    t = np.full(5, 3.5)
    oracle.ema(t, 0.0, c)
    assert np.array_equal(t, c.astype(np.float64))
    t = np.zeros(5)
    rng = np.random.default_rng(1)
    s = np.zeros(5, dtype=np.int64)
    for _ in range(50):
        x = rng.integers(0, 1 << 20, 5)
        oracle.ema(t, 1.0, x)
        s += x
    assert np.array_equal(t, s.astype(np.float64))


def test_dirichlet_f64_reduces_to_integer_counts():
    # integral fp64 totals draw exactly what the integer path draws
    net = koller()
    off, _ = brute.layout(net.parents, net.card)
    tot = np.random.default_rng(2).integers(0, 500, off[-1])
    a, ga = oracle.dirichlet(net.parents, net.card, tot, 1.0, 9, 4, want_gamma=True)
    b, gb = oracle.dirichlet_f64(net.parents, net.card, tot.astype(np.float64), 1.0, 9, 4, want_gamma=True)
    assert np.array_equal(a, b) and np.array_equal(ga, gb)


def test_dirichlet_f64_fractional_beta_marginal():
    net = koller()
    off, _ = brute.layout(net.parents, net.card)
    rng = np.random.default_rng(3)
    totals = rng.random(off[-1]) * 20.0  # fractional moving sums
    alpha = 1.0
    draws = np.array([oracle.dirichlet_f64(net.parents, net.card, totals, alpha, 5, q) for q in range(3000)])
    e = 17  # Grade row 2, state 2: Beta(a_k, A - a_k)
    u = (e - off[3]) // 3
    row = np.arange(off[3] + u * 3, off[3] + u * 3 + 3)
    a = alpha + totals[e]
    A = alpha * 3 + totals[row].sum()
    assert stats.kstest(draws[:, e], stats.beta(a, A - a).cdf).pvalue > 1e-4
    np.testing.assert_allclose(draws[:, row].sum(-1), 1.0, atol=1e-6)  # rows are distributions
