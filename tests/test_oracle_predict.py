"""Pins of held-out prediction (Sec. 6): with the CPTs frozen, the frequency
with which the sampler visits a test entry's true state estimates that state's
probability given the known entries; ROC/AUC scores the estimates."""
import numpy as np
import pytest
from sklearn.metrics import roc_auc_score

import oracle
from paper_1511_06416_amd import evaluate
from tests import brute
from workloads import holdout, koller, make_workload


@pytest.mark.slow
@pytest.mark.parametrize("evidence,test_node", [({3: 1, 4: 0}, 2), ({0: 1}, 4), ({2: 0, 4: 1}, 1)])
def test_predictive_frequency_reaches_exact_predictive(evidence, test_node):
    # every column is the same evidence pattern with test_node held out: its
    # hit frequency over the chains converges to the exact posterior predictive
    # P(x_test = target | evidence), computed by enumerating the joint
    net = koller()
    rng = np.random.default_rng(21)
    theta = brute.random_theta(rng, net.parents, net.card, alpha=1.0)
    color = oracle.graph(net.parents, net.card)["color"]
    n, m, n_cols, burn, sweeps = 5, 2, 4000, 20, 40
    obs = np.zeros((n, n_cols), dtype=np.uint8)
    states = np.zeros((n, m, n_cols), dtype=np.int8)
    for i, v in evidence.items():
        obs[i] = 1
        states[i] = v
    oracle.init_latent(net.card, n_cols, m, 0, 3, states, obs)
    target = np.full((n, n_cols), -1, dtype=np.int8)
    target[test_node] = 1
    for s in range(burn):
        oracle.sweep(net.parents, net.card, theta, color, states, obs, m, n_cols, 0, 7, s)
    hits = oracle.predict(net.parents, net.card, theta, color, states, obs, target, m, n_cols, 0, 7,
                          burn, sweeps)
    latent, post = brute.posterior_by_enumeration(net.parents, net.card, theta, evidence)
    pos = latent.index(test_node)
    exact = sum(p for cfg, p in post.items() if cfg[pos] == 1)
    per_chain = hits[test_node].astype(np.float64) / (m * sweeps)
    est = per_chain.mean()
    se = per_chain.std(ddof=1) / np.sqrt(n_cols)
    assert abs(est - exact) < 5 * se + 1e-3, (est, exact, se)


def test_auc_matches_sklearn():
    rng = np.random.default_rng(5)
    y = rng.random(3000) < 0.6
    s = np.round(rng.random(3000) + 0.3 * y, 2)  # rounded: many ties
    assert abs(evaluate.auc(s, y) - roc_auc_score(y, s)) < 1e-12
    assert evaluate.auc([0.1, 0.4, 0.35, 0.8], [0, 0, 1, 1]) == 0.75  # the classic small example
    with pytest.raises(ValueError):
        evaluate.auc([0.2, 0.3], [1, 1])


def test_accumulate_hits_counts_only_test_entries():
    n, m, ld, n_cols = 3, 4, 12, 10
    rng = np.random.default_rng(1)
    st = rng.integers(0, 3, (n, m, ld)).astype(np.int16)
    target = np.full((n, ld), -1, dtype=np.int16)
    target[0, 2] = st[0, 1, 2]
    target[2, 9] = 1
    target[1, 11] = 0          # past n_cols: ignored
    hits = np.full((n, ld), 5, dtype=np.int32)
    oracle.accumulate_hits(st, target, m, n_cols, hits)
    expect = np.full((n, ld), 5, dtype=np.int32)
    expect[0, 2] += int((st[0, :, 2] == st[0, 1, 2]).sum())
    expect[2, 9] += int((st[2, :, 9] == 1).sum())
    assert np.array_equal(hits, expect) and expect[0, 2] >= 6


def test_holdout_split_and_binary_scores():
    w = make_workload(4)
    obs_train, target = holdout(w, 0, 0.2)
    obs = w.obs[0].numpy()
    q = target >= 0
    assert (obs[q] == 1).all() and (obs_train[q] == 0).all()
    assert np.array_equal(obs_train[~q], obs[~q])
    frac = q[:, :w.n_cols].sum() / float(obs[:, :w.n_cols].sum())
    assert 0.18 < frac < 0.22
    hits = np.where(q, 3, 0).astype(np.int32)
    sc, lab = evaluate.binary_scores(hits, target, 4)
    assert np.allclose(sc[lab], 0.75) and np.allclose(sc[~lab], 0.25)
