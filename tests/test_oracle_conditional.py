"""Pins for the oracle's full conditional and draw rule.

The conditional of a node given everything else must equal the ratio of full
joints P(x_i = k, x_-i) / sum_k' P(x_i = k', x_-i), computed here as the
product of ALL n CPT factors (Sec. 1's CPT factorisation), not from the
Markov blanket.  The draw is pinned on hand-built boundary cases.
"""
import numpy as np
import pytest

import oracle
from tests import brute
from workloads import koller


@pytest.mark.parametrize("seed", range(6))
def test_conditional_equals_joint_ratio_random_nets(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(3, 7))
    parents, card = brute.random_net(rng, n, 3, 2, 4)
    theta = brute.random_theta(rng, parents, card, alpha=0.7)
    for _ in range(20):
        x = [int(rng.integers(0, card[i])) for i in range(n)]
        for node in range(n):
            got = oracle.conditional(parents, card, theta, x, node)
            want = brute.conditional_by_joint(parents, card, theta, x, node)
            np.testing.assert_allclose(got, want, rtol=1e-12, atol=0)
            assert abs(got.sum() - 1.0) < 1e-12


def test_conditional_student_all_configs():
    net = koller()
    rng = np.random.default_rng(5)
    theta = brute.random_theta(rng, net.parents, net.card)
    import itertools
    for x in itertools.product(*[range(k) for k in net.card]):
        for node in range(5):
            got = oracle.conditional(net.parents, net.card, theta, list(x), node)
            want = brute.conditional_by_joint(net.parents, net.card, theta, list(x), node)
            np.testing.assert_allclose(got, want, rtol=1e-12)


def test_childless_node_is_its_cpt_row():
    net = koller()
    rng = np.random.default_rng(9)
    theta = brute.random_theta(rng, net.parents, net.card)
    off, _ = brute.layout(net.parents, net.card)
    for g in range(3):
        x = [0, 1, 1, g, 0]
        p = oracle.conditional(net.parents, net.card, theta, x, 4)  # Letter has no children
        row = theta[off[4] + g * 2: off[4] + g * 2 + 2].astype(np.float64)
        np.testing.assert_allclose(p, row / row.sum(), rtol=1e-12)


def test_zero_entries_are_clamped_to_flt_min():
    # a zero CPT entry behaves as FLT_MIN: the state keeps a tiny positive weight
    parents, card = [[], [0]], np.array([2, 2], np.int32)
    theta = np.array([0.5, 0.5, 1.0, 0.0, 0.25, 0.75], np.float32)
    p = oracle.conditional(parents, card, theta, [0, 1], 0)
    # P(x0=0, x1=1) = 0.5*FLT_MIN, P(x0=1, x1=1) = 0.5*0.75
    fm = brute.FLT_MIN
    np.testing.assert_allclose(p, [fm / (fm + 0.75), 0.75 / (fm + 0.75)], rtol=1e-12)


# ---------------------------------------------------------------- draw rule

def test_draw_boundaries():
    w = [0.25, 0.25, 0.5]
    eps = 2.0 ** -24
    assert oracle.draw(w, 0.0)[0] == 0
    assert oracle.draw(w, 0.25 - eps)[0] == 0
    assert oracle.draw(w, 0.25)[0] == 1          # strict: u*Z < S_k
    assert oracle.draw(w, 0.5 - eps)[0] == 1
    assert oracle.draw(w, 0.5)[0] == 2
    assert oracle.draw(w, 1.0 - eps)[0] == 2


def test_draw_skips_zero_weight_states():
    assert oracle.draw([0.5, 0.0, 0.5], 0.5)[0] == 2
    assert oracle.draw([0.0, 1.0], 0.0)[0] == 1
    assert oracle.draw([1.0, 0.0], 1.0 - 2.0 ** -24)[0] == 0
    # u*Z that rounds up to Z falls back to the largest positive-weight state
    assert oracle.draw([0.3, 0.7, 0.0], 1.0)[0] == 1


def test_draw_flags():
    w = [0.25, 0.75]
    assert oracle.draw(w, 0.25)[1] is True
    assert oracle.draw(w, 0.25 + 5e-7)[1] is True
    assert oracle.draw(w, 0.25 + 2e-6)[1] is False
    assert oracle.draw(w, 0.9)[1] is False


def test_draw_frequencies_match_weights():
    w = np.array([0.1, 0.2, 0.3, 0.4])
    us = (np.arange(2 ** 14) + 0.5) / 2 ** 14
    picks = np.array([oracle.draw(w, u)[0] for u in us])
    freq = np.bincount(picks, minlength=4) / len(us)
    np.testing.assert_allclose(freq, w, atol=1e-3)


@pytest.mark.parametrize("seed", range(3))
def test_batched_conditionals_equal_joint_ratio(seed):
    # the batched form (one graph build for many state vectors) against the
    # full-joint ratio, row by row
    rng = np.random.default_rng(300 + seed)
    n = int(rng.integers(4, 7))
    parents, card = brute.random_net(rng, n, 3, 2, 5)
    theta = brute.random_theta(rng, parents, card, alpha=0.6)
    X = np.stack([[int(rng.integers(0, card[i])) for i in range(n)] for _ in range(40)])
    for node in range(n):
        got = oracle.conditionals(parents, card, theta, X, node)
        for row, x in enumerate(X):
            want = brute.conditional_by_joint(parents, card, theta, list(x), node)
            np.testing.assert_allclose(got[row], want, rtol=1e-12, atol=0)
