"""Pins for the oracle's graph code: the student network's published shape
(Sec. 5.1), the moral graph definition (Sec. 4) and colouring validity."""
import os

import numpy as np
import pytest

import oracle
from tests import brute
from workloads import CONFIGS, koller, make_network


def _student(golden_dir):
    d = {"edge": [], "moral": []}
    with open(os.path.join(golden_dir, "student_network.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            vals = [int(v) for v in vals]
            if key in ("edge", "moral"):
                d[key].append(tuple(vals))
            elif key == "card":
                d[key] = vals
            else:
                d[key] = vals[0]
    return d


def test_student_network_shape(golden_dir):
    g = _student(golden_dir)
    net = koller()
    assert list(net.card) == g["card"]
    edges = {(p, h) for h, ps in enumerate(net.parents) for p in ps}
    assert edges == set(g["edge"])
    out = oracle.graph(net.parents, net.card)
    off = out["cpt_off"]
    assert off[-1] == g["entries"]
    rows = sum((off[i + 1] - off[i]) // net.card[i] for i in range(net.n))
    assert rows == g["rows"]
    adj = oracle.moral_adjacency(net.parents, net.card)
    got = {frozenset((a, b)) for a in range(5) for b in range(5) if a < b and adj[a, b]}
    assert got == {frozenset(e) for e in g["moral"]}
    assert out["n_colors"] == g["colors"]


def _neighbours(parents):
    nbrs = [set() for _ in parents]
    for e in brute.moral_edges(parents):
        a, b = tuple(e)
        nbrs[a].add(b)
        nbrs[b].add(a)
    return nbrs


def _check_colouring(parents, color, first_fit=False):
    for e in brute.moral_edges(parents):
        a, b = tuple(e)
        assert color[a] != color[b], (a, b)
    if first_fit:
        # greedy (Grundy) property: a node of colour c has a neighbour of every colour < c
        nbrs = _neighbours(parents)
        for v in range(len(parents)):
            have = {int(color[w]) for w in nbrs[v]}
            assert all(c in have for c in range(int(color[v])))


def _check_balanced(parents, card):
    """The balanced colouring: proper, as many colours as first-fit, a size
    spread no larger than first-fit's, and no move left that the balancing
    rule allows (a node moving to a group at least two smaller without a
    neighbour there)."""
    ff = oracle.graph(parents, card, balance=False)
    bal = oracle.graph(parents, card)
    _check_colouring(parents, ff["color"], first_fit=True)
    _check_colouring(parents, bal["color"])
    assert bal["n_colors"] == ff["n_colors"]
    C = bal["n_colors"]
    s_ff = np.bincount(ff["color"], minlength=C)
    s_b = np.bincount(bal["color"], minlength=C)
    assert s_b.min() >= 1 and s_b.sum() == len(parents)
    assert s_b.max() - s_b.min() <= s_ff.max() - s_ff.min()
    nbrs = _neighbours(parents)
    col = bal["color"]
    for v in range(len(parents)):
        for b in range(C):
            if s_b[b] + 1 < s_b[col[v]]:
                assert any(col[w] == b for w in nbrs[v]), ("movable", v, b)
    return s_ff, s_b


@pytest.mark.parametrize("seed", range(8))
def test_random_dag_colouring_valid(seed):
    rng = np.random.default_rng(seed)
    parents, card = brute.random_net(rng, 40, 4, 2, 5)
    out = oracle.graph(parents, card)
    _check_balanced(parents, card)
    # topological order respects every edge
    pos = {int(v): t for t, v in enumerate(out["topo"])}
    for h, ps in enumerate(parents):
        for p in ps:
            assert pos[p] < pos[h]
    # moral adjacency equals the definition
    adj = oracle.moral_adjacency(parents, card)
    want = brute.moral_edges(parents)
    got = {frozenset((a, b)) for a in range(40) for b in range(a + 1, 40) if adj[a, b]}
    assert got == want
    off, _ = brute.layout(parents, card)
    assert list(out["cpt_off"]) == off


@pytest.mark.parametrize("cfg", [1, 3, 4, 5])
def test_config_networks_colour(cfg):
    net = make_network(cfg)
    s_ff, s_b = _check_balanced(net.parents, net.card)
    print(cfg, "first-fit", s_ff.tolist(), "balanced", s_b.tolist())


def test_balancing_hand_example():
    # 1 <- 0 and two roots 2, 3: first-fit over the order 0, 1, 2, 3 gives
    # colours (0, 1, 0, 0); the largest group {0, 2, 3} gives its first
    # movable node to group 1: node 0 has neighbour 1 there, node 2 has none
    parents = [[], [0], [], []]
    card = [2, 2, 2, 2]
    assert list(oracle.graph(parents, card, balance=False)["color"]) == [0, 1, 0, 0]
    assert list(oracle.graph(parents, card)["color"]) == [0, 1, 1, 0]
    # a chain 0 - 1 - 2 - 3 - 4: first-fit alternates (3 / 2), already balanced
    chain = [[], [0], [1], [2], [3]]
    assert list(oracle.graph(chain, [2] * 5)["color"]) == [0, 1, 0, 1, 0]


def test_invalid_graphs_rejected():
    # self loop
    assert oracle.graph_rc([0, 1], [0], [2]) == -2
    # duplicate parent
    assert oracle.graph_rc([0, 0, 2], [0, 0], [2, 2]) == -2
    # parent out of range
    assert oracle.graph_rc([0, 1], [5], [2]) == -2
    # 2-cycle
    assert oracle.graph_rc([0, 1, 2], [1, 0], [2, 2]) == -2
    # bad cardinality
    assert oracle.graph_rc([0, 0], [], [1]) == -3
    # ok
    assert oracle.graph_rc([0, 0, 1], [0], [2, 3]) == 0


def test_configs_sizes_recorded():
    # c4 is two-layer: 30 parentless concepts, 300 items with 1-2 concept parents
    net = make_network(4)
    assert net.n == 330
    assert all(len(p) == 0 for p in net.parents[:30])
    assert all(1 <= len(p) <= 2 and max(p) < 30 for p in net.parents[30:])
    assert CONFIGS[5]["nb"] == 250_000
