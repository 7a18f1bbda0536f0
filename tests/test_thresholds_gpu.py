"""GPU parity of the precomputed threshold tables.

Nodes whose Markov blanket has few configurations draw from a table of
integer CDF thresholds T_k = ceil(2^24 S_k / Z), one row per blanket
configuration, built in fp64 once per CPT update; the draw with 24-bit uniform
u24 is #{k : T_k <= u24} (the inverse-CDF rule of the Gibbs draw, Sec. 4).
Here every row of every table is formed from the oracle's conditional
(the normalised product of the node's own CPT entry and its children's
entries) for that blanket configuration and compared with the library's
table word for word.  The only words excused are those where 2^24 S_k / Z lies
within 1e-6 of an integer, where rounding of the fp64 logs, exponentials and
sums may move the ceiling by one; they are counted and reported.  They are
not rare: when a conditional reduces to fp32 CPT entries (a node whose
children's factors are equal across its states), 2^24 S_k / Z is often an
exact integer, since an fp32 value in [0.5, 1) is a multiple of 2^-24.  A
draw can differ there only when u24 equals that integer, and the oracle flags
such a draw (u on a CDF boundary).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1511_06416_amd as same
from tests import brute, gpu_helpers as H
from workloads import Network, make_workload

pytestmark = pytest.mark.gpu

TWO24 = float(1 << 24)
EXCUSE = 1e-6


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


def blanket(parents, i):
    kids = [h for h, ps in enumerate(parents) if i in ps]
    b = set(parents[i]) | set(kids)
    for h in kids:
        b |= set(parents[h])
    b.discard(i)
    return sorted(b)


def kt_of(K):
    t = 1
    while t < K - 1:
        t <<= 1
    return t


def expected_rows(parents, card, theta, i):
    """[n_cfg][KT] thresholds from the oracle's conditional, and the mask of
    entries within rounding of an integer."""
    b = blanket(parents, i)
    K = int(card[i])
    KT = kt_of(K)
    cards = [int(card[v]) for v in b]
    n_cfg = int(np.prod(cards)) if b else 1
    X = np.zeros((n_cfg, len(parents)), dtype=np.int32)
    rem = np.arange(n_cfg)
    for t in range(len(b) - 1, -1, -1):       # last blanket node fastest
        X[:, b[t]] = rem % cards[t]
        rem //= cards[t]
    p = oracle.conditionals(parents, card, theta, X, i)
    S = np.cumsum(p, axis=1) / p.sum(axis=1, keepdims=True)
    T = np.full((n_cfg, KT), 1 << 24, dtype=np.int64)
    near = np.zeros((n_cfg, KT), dtype=bool)
    V = np.zeros((n_cfg, KT))
    for k in range(min(K - 1, KT)):
        v = S[:, k] * TWO24
        V[:, k] = v
        T[:, k] = np.minimum(np.ceil(v), TWO24).astype(np.int64)
        near[:, k] = np.abs(v - np.round(v)) < EXCUSE
    return T, near, V


def check_tables(parents, card, theta, ctx, table_limit=6144):
    th = torch.from_numpy(np.ascontiguousarray(theta, dtype=np.float32)).cuda()
    ws = ctx.new_workspace()
    off, kt, tab = same.same_debug_thresholds(ctx, th, ws)
    torch.cuda.synchronize()
    tab = tab.cpu().numpy().view(np.uint32).astype(np.int64)
    n = len(parents)
    checked = excused = nodes = 0
    samples = []
    for i in range(n):
        b = blanket(parents, i)
        K = int(card[i])
        n_cfg = int(np.prod([int(card[v]) for v in b])) if b else 1
        # the documented rule for which nodes get a table
        want_table = (table_limit > 0 and K <= 9 and n_cfg * kt_of(K) <= table_limit and n_cfg <= 65536
                      and len(b) <= 24)
        assert (off[i] >= 0) == want_table, (i, K, n_cfg, off[i])
        if off[i] < 0:
            continue
        assert kt[i] == kt_of(K)
        T, near, V = expected_rows(parents, card, theta, i)
        got = tab[off[i]:off[i] + T.size].reshape(T.shape)
        bad = (got != T) & ~near
        assert not bad.any(), ("node", i, "rows", np.argwhere(bad)[:5].tolist(),
                               got[bad][:5].tolist(), T[bad][:5].tolist())
        ex = (got != T) & near
        if ex.any() and len(samples) < 8:
            samples.append((i, got[ex][:3].tolist(), T[ex][:3].tolist(), V[ex][:3].tolist()))
        excused += int(ex.sum())
        checked += T.size
        nodes += 1
    if samples:
        print("excused (node, library, oracle, 2^24 S/Z):", samples)
    return {"nodes": nodes, "words": checked, "excused": excused}


def test_thresholds_random1000():
    """Every table node of the 1000-node network (about 450 of them), with the
    starting CPTs and with CPTs resampled from counts."""
    w = make_workload(5, n_cols=2_000, m=2)
    net = w.net
    ctx = H.context_for(net)
    out = check_tables(net.parents, net.card, w.init_theta, ctx)
    print("init theta", out)
    assert out["nodes"] == ctx.table_nodes and out["nodes"] > 300
    assert out["excused"] <= 0.01 * out["words"]
    tot = oracle.counts(net.parents, net.card, w.states[0].numpy(), w.m, w.mb_cols(0))
    theta = oracle.dirichlet(net.parents, net.card, tot, 1.0, 77, 3)
    out = check_tables(net.parents, net.card, theta, ctx)
    print("resampled theta", out)
    assert out["excused"] <= 0.01 * out["words"]


@pytest.mark.parametrize("cfg", [1, 3, 4])
def test_thresholds_other_workloads(cfg):
    w = make_workload(cfg, n_cols=1_000)
    net = w.net
    ctx = H.context_for(net)
    out = check_tables(net.parents, net.card, w.init_theta, ctx)
    print(w.name, out)
    assert out["nodes"] == ctx.table_nodes


@pytest.mark.parametrize("K", [2, 3, 4, 5, 6, 7, 8, 9])
def test_thresholds_cardinalities(K):
    """One table per threshold width (KT = 1, 2, 4, 8) and every K up to 9,
    with zero CPT entries (clamped to FLT_MIN) and sharp rows."""
    parents = [[], [0], [0, 1], [1], [2, 3]]
    card = [K, 3, K, 2, 4]
    rng = np.random.default_rng(40 + K)
    theta = brute.random_theta(rng, parents, card, alpha=0.3).astype(np.float32)
    theta[rng.random(theta.size) < 0.05] = 0.0
    out = check_tables(parents, card, theta, H.context_for(Network("custom", parents, card)))
    print("K", K, out)
    assert out["nodes"] >= 3


def test_thresholds_table_limit_zero():
    # with the tables disabled no node reports one
    w = make_workload(1, n_cols=100)
    ctx = H.context_for(w.net, table_limit=0)
    off, kt, _ = same.same_debug_thresholds(ctx)
    assert (off == -1).all() and (kt == 0).all()

