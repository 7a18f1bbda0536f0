"""Pins for the oracle's counts, moving sum, Gamma and Dirichlet steps.

* Counts equal a numpy recount (np.add.at over (parent row, state)); every
  node's counts total n_cols * m.
* Moving sum (Sec. 4): after a full pass the running total equals the counts
  of all current states.
* Gamma(a): KS against scipy's Gamma(a) cdf, mean and variance; the
  Marsaglia-Tsang acceptance rate is above 0.95 for a >= 1.
* Dirichlet(alpha + T): rows sum to one; each entry is Beta(a_k, A - a_k)
  (KS); complete-data SAME: with every entry observed and alpha = 1 the
  resample is Dir(1 + m * n), i.e. P(Theta | X)^m normalised (Sec. 3).
"""
import numpy as np
import pytest
from scipy import stats

import oracle
from tests import brute, oracle_loop
from workloads import koller, make_workload


@pytest.mark.parametrize("dtype", [np.int8, np.int16])
def test_counts_equal_numpy_recount(dtype):
    rng = np.random.default_rng(3)
    parents, card = brute.random_net(rng, 15, 3, 2, 6)
    m, n_cols, ld = 3, 777, 800
    states = np.zeros((15, m, ld), dtype=dtype)
    for i in range(15):
        states[i, :, :n_cols] = rng.integers(0, card[i], (m, n_cols))
        states[i, :, n_cols:] = 99  # padding must be ignored
    got = oracle.counts(parents, card, states, m, n_cols)
    want = brute.recount(parents, card, states, m, n_cols)
    assert np.array_equal(got, want)
    off, _ = brute.layout(parents, card)
    for i in range(15):
        assert got[off[i]:off[i + 1]].sum() == n_cols * m


def test_moving_sum_equals_counts_of_current_states():
    w = make_workload(1, n_cols=3000, nb=1000, m=2)
    assert w.M == 3
    out = oracle_loop.run(w, sweeps=2)
    net = w.net
    direct = sum(oracle.counts(net.parents, net.card, s, w.m, w.mb_cols(b))
                 for b, s in enumerate(out["states"]))
    assert np.array_equal(out["totals"], direct)
    for b, s in enumerate(out["states"]):
        assert np.array_equal(out["mb_counts"][b],
                              brute.recount(net.parents, net.card, s, w.m, w.mb_cols(b)))


@pytest.mark.parametrize("shape", [0.3, 1.0, 2.5, 17.0, 1000.0])
def test_gamma_distribution(shape):
    n = 4000
    g = np.array([oracle.gamma(shape, 12345, e, 3)[0] for e in range(n)])
    ks = stats.kstest(g, stats.gamma(shape).cdf)
    assert ks.pvalue > 1e-4
    assert abs(g.mean() - shape) < 6 * np.sqrt(shape / n)
    if shape >= 1.0:
        att = np.array([oracle.gamma(shape, 12345, e, 3)[1] for e in range(n)])
        assert 1.0 / att.mean() > 0.95


def test_gamma_is_deterministic_per_counter():
    a = oracle.gamma(3.0, 1, 5, 7)
    assert a == oracle.gamma(3.0, 1, 5, 7)
    assert a != oracle.gamma(3.0, 1, 6, 7)
    assert a != oracle.gamma(3.0, 1, 5, 8)
    assert a != oracle.gamma(3.0, 2, 5, 7)


def test_dirichlet_rows_and_beta_marginals():
    net = koller()
    off, _ = brute.layout(net.parents, net.card)
    rng = np.random.default_rng(0)
    totals = rng.integers(0, 30, off[-1])
    alpha = 0.7
    draws = np.array([oracle.dirichlet(net.parents, net.card, totals, alpha, 77, q)
                      for q in range(3000)])
    for i in range(net.n):
        K = int(net.card[i])
        blk = draws[:, off[i]:off[i + 1]].reshape(draws.shape[0], -1, K)
        np.testing.assert_allclose(blk.sum(-1), 1.0, atol=1e-6)
    # entry 17 (Grade row 2, state 2) is Beta(a_k, A - a_k)
    e = 17
    i, u = 3, (17 - off[3]) // 3
    row = np.arange(off[3] + u * 3, off[3] + u * 3 + 3)
    a = alpha + totals[e]
    A = alpha * 3 + totals[row].sum()
    ks = stats.kstest(draws[:, e], stats.beta(a, A - a).cdf)
    assert ks.pvalue > 1e-4
    var = a * (A - a) / (A * A * (A + 1))
    assert abs(draws[:, e].mean() - a / A) < 6 * np.sqrt(var / draws.shape[0])


def test_complete_data_same_is_power_posterior():
    # every entry observed: replicas are identical, so the counts are m times the
    # data counts and Dir(1 + m n) is P(Theta | X)^m renormalised (alpha = 1)
    m = 4
    w = make_workload(1, n_cols=500, m=m, hidden=0.0, keep_data=True)
    net = w.net
    st = w.states[0].numpy()
    assert np.all(w.obs[0].numpy()[:, :500] == 1)
    data_counts = brute.recount(net.parents, net.card, st[:, :1, :], 1, 500)
    out = oracle_loop.run(w, sweeps=1)
    assert np.array_equal(out["totals"], m * data_counts)
    off, _ = brute.layout(net.parents, net.card)
    # many resamples from those totals: mean of Dir(1 + m n)
    draws = np.array([oracle.dirichlet(net.parents, net.card, out["totals"], 1.0, 5, q)
                      for q in range(2000)])
    for i in range(net.n):
        K = int(net.card[i])
        t = out["totals"][off[i]:off[i + 1]].reshape(-1, K) + 1.0
        mean = (t / t.sum(1, keepdims=True)).reshape(-1)
        got = draws[:, off[i]:off[i + 1]].mean(0)
        sd = np.sqrt(mean * (1 - mean) / (t.sum(1).repeat(K) + 1) / draws.shape[0])
        assert np.all(np.abs(got - mean) < 6 * sd + 1e-7)


def test_student_loop_learns_true_cpts():
    # sanity (untimed): KL_avg to the generating CPTs falls over the passes
    w = make_workload(1, n_cols=20000, m=2)
    kls = []
    oracle_loop.run(w, sweeps=8,
                    on_update=lambda s, b, th: kls.append(oracle_loop.kl_avg(w.net, w.true_theta, th)))
    init = oracle_loop.kl_avg(w.net, w.true_theta, w.init_theta)
    assert kls[-1] < 0.5 * init
    assert kls[-1] < 0.05
