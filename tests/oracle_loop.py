"""The full SAME loop driven through the oracle's primitives (tests only).

Per pass s and minibatch b (Sec. 4, Fig. 1): one Gibbs sweep over the m
replicas of minibatch b, its new counts, the exact moving sum
totals += new - previous, then a Dirichlet resample of every CPT row from
alpha + totals with update id s*M + b.  Before the first pass a count-only
pre-pass over all minibatches initialises the per-minibatch counts.
"""
from __future__ import annotations

import numpy as np

import oracle


def run(w, sweeps=None, n_threads=0, theta=None, on_update=None):
    net = w.net
    color = oracle.graph(net.parents, net.card)["color"]
    theta = (w.init_theta if theta is None else theta).copy()
    states = [s.cpu().numpy().copy() for s in w.states]
    obs = [o.cpu().numpy() for o in w.obs]
    mb = [oracle.counts(net.parents, net.card, states[b], w.m, w.mb_cols(b), n_threads)
          for b in range(w.M)]
    totals = np.sum(mb, axis=0)
    S = w.sweeps if sweeps is None else sweeps
    for s in range(S):
        for b in range(w.M):
            oracle.sweep(net.parents, net.card, theta, color, states[b], obs[b], w.m,
                         w.mb_cols(b), b * w.nb, w.seed, s, n_threads=n_threads)
            new = oracle.counts(net.parents, net.card, states[b], w.m, w.mb_cols(b), n_threads)
            totals = oracle.moving_sum(totals, mb[b], new)
            mb[b] = new
            theta = oracle.dirichlet(net.parents, net.card, totals, w.alpha, w.seed, s * w.M + b)
            if on_update is not None:
                on_update(s, b, theta)
    return {"theta": theta, "totals": totals, "mb_counts": mb, "states": states,
            "color": color}


def kl_avg(net, p_theta, q_theta):
    """KL_avg of Sec. 5.1: mean over CPT rows of sum_x p log(p/q), over x with q(x) > 0."""
    from workloads import cpt_layout
    off, rows, _ = cpt_layout(net)
    tot, cnt = 0.0, 0
    for i in range(net.n):
        K = int(net.card[i])
        P = np.asarray(p_theta[off[i]:off[i + 1]], dtype=np.float64).reshape(-1, K)
        Q = np.asarray(q_theta[off[i]:off[i + 1]], dtype=np.float64).reshape(-1, K)
        for pr, qr in zip(P, Q):
            mask = (qr > 0) & (pr > 0)
            tot += float(np.sum(pr[mask] * np.log(pr[mask] / qr[mask])))
            cnt += 1
    return tot / cnt
