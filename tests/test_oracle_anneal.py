"""Pins of SAME annealing (Sec. 3: the replication factor raised during
sampling) and of the KL_avg evaluation metric (Sec. 5.1)."""
import numpy as np
from scipy import stats

import oracle
from paper_1511_06416_amd import evaluate
from tests import brute
from workloads import koller, make_workload


def test_grow_replicas_copies_chains():
    w = make_workload(3, n_cols=1_001, m=3)
    st = w.states[0].numpy()
    g = oracle.grow_replicas(st, 7)
    assert g.shape == (st.shape[0], 7, st.shape[2])
    for r in range(7):
        assert np.array_equal(g[:, r], st[:, r % 3])
    assert np.array_equal(oracle.grow_replicas(st, 3), st)


def test_grown_counts_scale_exactly():
    # copies of every chain: the histogram over m2 = k * m replicas is k times
    # the histogram over the m replicas (the SAME joint with more copies)
    w = make_workload(4)
    net = w.net
    st = w.states[0].numpy()
    c = oracle.counts(net.parents, net.card, st, w.m, w.n_cols)
    g = oracle.grow_replicas(st, 3 * w.m)
    c3 = oracle.counts(net.parents, net.card, g, 3 * w.m, w.n_cols)
    assert np.array_equal(c3, 3 * c)


def test_kl_avg_definition():
    net = koller()
    off, _ = brute.layout(net.parents, net.card)
    rng = np.random.default_rng(8)
    p = brute.random_theta(rng, net.parents, net.card, alpha=1.0)
    q = brute.random_theta(rng, net.parents, net.card, alpha=1.0)
    rows = []
    for i in range(net.n):
        K = int(net.card[i])
        for u in range((off[i + 1] - off[i]) // K):
            s = slice(off[i] + u * K, off[i] + (u + 1) * K)
            rows.append(stats.entropy(p[s], q[s]))  # sum p log(p / q)
    assert len(rows) == 11  # the student network's eleven distributions (Sec. 5.1)
    assert abs(evaluate.kl_avg(p, q, off, net.card) - np.mean(rows)) < 1e-12
    assert evaluate.kl_avg(p, p, off, net.card) == 0.0
    # terms with q(x) = 0 are left out of the sum (Sec. 5.1)
    q2 = q.copy()
    q2[0], q2[1] = 1.0, 0.0  # node 0's single row: all mass on state 0
    k = evaluate.kl_avg(p, q2, off, net.card)
    assert np.isfinite(k)
    assert abs(k - (np.mean(rows) + (p[0] * np.log(p[0] / 1.0) - stats.entropy(p[0:2], q[0:2])) / 11)) < 1e-12
