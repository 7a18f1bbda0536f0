"""Brute-force references used to pin the oracle (tests only).

Everything here works from the definition of a Bayesian network's joint
distribution, P(x) = prod_j theta_j(x_j | x_pa(j)) (Sec. 1), by plain
enumeration over all n factors or over all joint configurations, so that it
shares no formula with the oracle's Markov-blanket code.
"""
from __future__ import annotations

import itertools

import numpy as np

FLT_MIN = float(np.finfo(np.float32).tiny)


def layout(parents, card):
    """CPT offsets and per-node parent strides (listed order, last parent fastest)."""
    n = len(parents)
    off = [0]
    strides = []
    for i in range(n):
        st = []
        r = 1
        for p in reversed(parents[i]):
            st.insert(0, r)
            r *= int(card[p])
        strides.append(st)
        off.append(off[-1] + r * int(card[i]))
    return off, strides


def entry(parents, card, off, strides, i, x):
    u = sum(int(x[p]) * s for p, s in zip(parents[i], strides[i]))
    return off[i] + u * int(card[i]) + int(x[i])


def joint(parents, card, theta, x, clamp=True):
    """P(x) as the product over ALL n factors (no Markov-blanket shortcut)."""
    off, strides = layout(parents, card)
    p = 1.0
    for i in range(len(parents)):
        t = float(theta[entry(parents, card, off, strides, i, x)])
        if clamp:
            t = max(t, FLT_MIN)
        p *= t
    return p


def conditional_by_joint(parents, card, theta, x, node):
    """P(x_node = k | all other x) = P(x with x_node=k) / sum_k' P(...)."""
    K = int(card[node])
    w = np.zeros(K)
    y = list(x)
    for k in range(K):
        y[node] = k
        w[k] = joint(parents, card, theta, y)
    return w / w.sum()


def posterior_by_enumeration(parents, card, theta, evidence):
    """Exact P(latent configuration | evidence) by enumerating all joint states.

    evidence: dict node -> value.  Returns (latent_nodes, {config tuple: prob}).
    """
    n = len(parents)
    latent = [i for i in range(n) if i not in evidence]
    probs = {}
    for cfg in itertools.product(*[range(int(card[i])) for i in latent]):
        x = [0] * n
        for i, v in evidence.items():
            x[i] = v
        for i, v in zip(latent, cfg):
            x[i] = v
        probs[cfg] = joint(parents, card, theta, x, clamp=False)
    z = sum(probs.values())
    return latent, {k: v / z for k, v in probs.items()}


def recount(parents, card, states, m, n_cols):
    """Count histogram with numpy: for every node, replica and column, add one
    at (parent configuration, own state)."""
    off, strides = layout(parents, card)
    out = np.zeros(off[-1], dtype=np.int64)
    for i in range(len(parents)):
        u = np.zeros((m, n_cols), dtype=np.int64)
        for p, s in zip(parents[i], strides[i]):
            u += states[p, :, :n_cols].astype(np.int64) * s
        idx = off[i] + u * int(card[i]) + states[i, :, :n_cols].astype(np.int64)
        np.add.at(out, idx.reshape(-1), 1)
    return out


def moral_edges(parents):
    """Moral graph (Sec. 4): connect every parent pair of a node, drop directions."""
    e = set()
    for h, ps in enumerate(parents):
        for p in ps:
            e.add(frozenset((p, h)))
        for a, b in itertools.combinations(ps, 2):
            e.add(frozenset((a, b)))
    return e


def random_net(rng, n, max_par, kmin, kmax):
    parents, card = [], []
    for i in range(n):
        k = min(int(rng.integers(0, max_par + 1)), i)
        ps = list(rng.choice(i, size=k, replace=False)) if k else []
        rng.shuffle(ps)  # unsorted parent order exercises the listed-order radix
        parents.append([int(p) for p in ps])
        card.append(int(rng.integers(kmin, kmax + 1)))
    # relabel nodes by a random permutation so ids are not topological
    perm = rng.permutation(n)
    inv = np.argsort(perm)
    new_parents = [None] * n
    new_card = [0] * n
    for old in range(n):
        new = int(perm[old])
        new_parents[new] = [int(perm[p]) for p in parents[old]]
        new_card[new] = card[old]
    del inv
    return new_parents, np.array(new_card, dtype=np.int32)


def random_theta(rng, parents, card, alpha=1.0):
    off, _ = layout(parents, card)
    th = np.zeros(off[-1], dtype=np.float64)
    for i in range(len(parents)):
        K = int(card[i])
        R = (off[i + 1] - off[i]) // K
        th[off[i]:off[i + 1]] = rng.dirichlet(np.full(K, alpha), size=R).reshape(-1)
    return th.astype(np.float32)
