"""Pins for the oracle's sweep.

* Brute force: a pure-Python sequential scan that visits the colour groups in
  order but the nodes INSIDE each colour in a random permutation, with every
  conditional computed from full joints, reproduces the oracle's states
  exactly (Sec. 4: colour-parallel sampling equals a sequential scan over a
  permutation; any order inside a colour is equivalent).
* Stationarity / posterior: with Theta fixed, many independent chains reach
  the exact posterior P(Z | x_obs, Theta) computed by enumeration (chi-square);
  chains started from the joint stay at the joint (prior invariance).
* Columns and replicas are independent chains: a sub-range of columns swept
  alone gives the same result as inside the full minibatch; the thread count
  does not change the result; observed entries never change.
"""
import numpy as np
import pytest
from scipy import stats

import oracle
from tests import brute
from workloads import koller


def _random_case(rng, parents, card, m, n_cols, ld, hidden=0.5):
    n = len(parents)
    states = np.zeros((n, m, ld), dtype=np.int8)
    obs = np.ones((n, ld), dtype=np.uint8)
    for i in range(n):
        obs[i, :n_cols] = (rng.random(n_cols) >= hidden).astype(np.uint8)
        data = rng.integers(0, card[i], n_cols)
        for r in range(m):
            lat = rng.integers(0, card[i], n_cols)
            states[i, r, :n_cols] = np.where(obs[i, :n_cols] == 1, data, lat)
    return states, obs


def _python_scan(parents, card, theta, color, states, obs, m, n_cols, col_offset, seed, sweep_id,
                 rng):
    n = len(parents)
    out = states.copy()
    for c in range(int(max(color)) + 1):
        members = [i for i in range(n) if color[i] == c]
        rng.shuffle(members)
        for i in members:
            for j in range(n_cols):
                if obs[i, j]:
                    continue
                for r in range(m):
                    x = [int(out[v, r, j]) for v in range(n)]
                    p = brute.conditional_by_joint(parents, card, theta, x, i)
                    u = oracle.gibbs_uniform(seed, i, r, col_offset + j, sweep_id)
                    out[i, r, j] = oracle.draw(p, u)[0]
    return out


@pytest.mark.parametrize("seed", range(4))
def test_sweep_equals_bruteforce_permuted_scan(seed):
    rng = np.random.default_rng(300 + seed)
    if seed == 0:
        net = koller()
        parents, card = net.parents, net.card
    else:
        parents, card = brute.random_net(rng, int(rng.integers(4, 8)), 3, 2, 4)
    theta = brute.random_theta(rng, parents, card, alpha=0.8)
    color = oracle.graph(parents, card)["color"]
    m, n_cols, ld = 3, 37, 40
    states, obs = _random_case(rng, parents, card, m, n_cols, ld)
    want = _python_scan(parents, card, theta, color, states, obs, m, n_cols, 8, 11, 2, rng)
    got = states.copy()
    res = oracle.sweep(parents, card, theta, color, got, obs, m, n_cols, 8, 11, 2, want_flags=True)
    diff = got != want
    assert not np.any(diff & (res["flags"] == 0))
    assert np.all(got[:, :, n_cols:] == states[:, :, n_cols:])  # padding untouched


def test_observed_entries_never_change_and_counts_of_draws():
    rng = np.random.default_rng(1)
    net = koller()
    theta = brute.random_theta(rng, net.parents, net.card)
    color = oracle.graph(net.parents, net.card)["color"]
    m, n_cols, ld = 4, 500, 512
    states, obs = _random_case(rng, net.parents, net.card, m, n_cols, ld)
    before = states.copy()
    res = oracle.sweep(net.parents, net.card, theta, color, states, obs, m, n_cols, 0, 3, 0)
    o = np.broadcast_to(obs[:, None, :], states.shape).astype(bool)
    assert np.all(states[o] == before[o])
    assert res["draws"] == int((obs[:, :n_cols] == 0).sum()) * m
    for i in range(5):
        assert states[i].max() < net.card[i] and states[i].min() >= 0


def test_columns_are_independent_chains_and_thread_invariance():
    rng = np.random.default_rng(2)
    parents, card = brute.random_net(rng, 12, 3, 2, 5)
    theta = brute.random_theta(rng, parents, card)
    color = oracle.graph(parents, card)["color"]
    m, n_cols, ld = 2, 1000, 1024
    states, obs = _random_case(rng, parents, card, m, n_cols, ld)
    full = states.copy()
    oracle.sweep(parents, card, theta, color, full, obs, m, n_cols, 4000, 5, 1, n_threads=4)
    one = states.copy()
    oracle.sweep(parents, card, theta, color, one, obs, m, n_cols, 4000, 5, 1, n_threads=1)
    assert np.array_equal(full, one)
    # columns 200..263 swept alone (global columns 4200..4263)
    sub = np.ascontiguousarray(states[:, :, 200:264])
    subo = np.ascontiguousarray(obs[:, 200:264])
    oracle.sweep(parents, card, theta, color, sub, subo, m, 64, 4200, 5, 1)
    assert np.array_equal(sub, full[:, :, 200:264])


def _chains_posterior_test(evidence, n_cols=20000, m=5, sweeps=15, seed=7):
    net = koller()
    rng = np.random.default_rng(seed)
    theta = brute.random_theta(rng, net.parents, net.card, alpha=1.5)
    color = oracle.graph(net.parents, net.card)["color"]
    n = net.n
    states = np.zeros((n, m, n_cols), dtype=np.int8)
    obs = np.zeros((n, n_cols), dtype=np.uint8)
    for i in range(n):
        if i in evidence:
            obs[i] = 1
            states[i] = evidence[i]
        else:
            states[i] = rng.integers(0, net.card[i], (m, n_cols))
    for s in range(sweeps):
        oracle.sweep(net.parents, net.card, theta, color, states, obs, m, n_cols, 0, 99, s)
    latent, post = brute.posterior_by_enumeration(net.parents, net.card, theta, evidence)
    keys = list(post)
    idx = {k: t for t, k in enumerate(keys)}
    cfgs = states[latent].reshape(len(latent), -1).T
    hist = np.zeros(len(keys))
    for row in map(tuple, cfgs):
        hist[idx[row]] += 1
    expected = np.array([post[k] for k in keys]) * cfgs.shape[0]
    return _chi2_p(hist, expected)


def _chi2_p(hist, expected):
    """Chi-square p-value, lumping cells with expected count <= 5 into one."""
    keep = expected > 5
    obs_k, exp_k = hist[keep], expected[keep]
    if expected[~keep].sum() > 0:
        obs_k = np.append(obs_k, hist[~keep].sum())
        exp_k = np.append(exp_k, expected[~keep].sum())
    exp_k = exp_k * obs_k.sum() / exp_k.sum()
    return stats.chisquare(obs_k, exp_k).pvalue


@pytest.mark.parametrize("evidence", [{2: 1, 4: 0}, {3: 2}, {0: 1, 4: 1}])
def test_chains_reach_exact_posterior(evidence):
    assert _chains_posterior_test(evidence) > 1e-4


def test_prior_invariance():
    # all latent; chains started exactly at the joint stay at the joint
    net = koller()
    rng = np.random.default_rng(11)
    theta = brute.random_theta(rng, net.parents, net.card, alpha=1.5)
    color = oracle.graph(net.parents, net.card)["color"]
    n, m, n_cols = 5, 4, 20000
    off, strides = brute.layout(net.parents, net.card)
    states = np.zeros((n, m, n_cols), dtype=np.int8)
    th = theta.astype(np.float64)
    for i in range(n):  # ids are topological for this network
        K = int(net.card[i])
        u = np.zeros((m, n_cols), dtype=np.int64)
        for p, s in zip(net.parents[i], strides[i]):
            u += states[p].astype(np.int64) * s
        cdf = np.cumsum(th[off[i]:off[i + 1]].reshape(-1, K), axis=1)
        cdf /= cdf[:, -1:]
        r = rng.random((m, n_cols))
        states[i] = (r[..., None] >= cdf[u][..., :K - 1]).sum(-1)
    obs = np.zeros((n, n_cols), dtype=np.uint8)
    for s in range(3):
        oracle.sweep(net.parents, net.card, theta, color, states, obs, m, n_cols, 0, 5, s)
    _, post = brute.posterior_by_enumeration(net.parents, net.card, theta, {})
    keys = list(post)
    idx = {k: t for t, k in enumerate(keys)}
    hist = np.zeros(len(keys))
    for row in map(tuple, states.reshape(n, -1).T):
        hist[idx[row]] += 1
    expected = np.array([post[k] for k in keys]) * m * n_cols
    assert _chi2_p(hist, expected) > 1e-4


def test_debug_window_conditionals_match_joint_ratio():
    rng = np.random.default_rng(4)
    net = koller()
    theta = brute.random_theta(rng, net.parents, net.card)
    color = oracle.graph(net.parents, net.card)["color"]
    m, n_cols, ld = 2, 30, 32
    states, obs = _random_case(rng, net.parents, net.card, m, n_cols, ld)
    work = states.copy()
    res = oracle.sweep(net.parents, net.card, theta, color, work, obs, m, n_cols, 0, 1, 0,
                       win=(5, 10))
    # recompute each window conditional from the chain as it stood at that node's visit:
    # nodes of later colours still hold their pre-sweep values, earlier ones their new ones
    for i in range(5):
        for r in range(m):
            for j in range(5, 15):
                if obs[i, j]:
                    assert np.all(np.isnan(res["probs"][i, r, j - 5]))
                    continue
                x = [int(work[v, r, j]) if color[v] < color[i] else int(states[v, r, j])
                     for v in range(5)]
                want = brute.conditional_by_joint(net.parents, net.card, theta, x, i)
                K = int(net.card[i])
                np.testing.assert_allclose(res["probs"][i, r, j - 5, :K], want, rtol=1e-12)
