"""Pins of the oracle's data-ingest functions: the dense minibatch built from
the known entries of the (typically sparse) node x case matrix (Sec. 4), and
the random initial latent states (Sec. 5.2)."""
import numpy as np
import pytest
from scipy import stats

import oracle
from workloads import make_network, make_workload


def csr_of_observed(states, obs, n_cols):
    """Rows = variables (Sec. 4): the known entries of replica 0, by numpy."""
    n = obs.shape[0]
    row_ptr = np.zeros(n + 1, dtype=np.int64)
    cols, vals = [], []
    for i in range(n):
        j = np.nonzero(obs[i, :n_cols])[0]
        cols.append(j.astype(np.int32))
        vals.append(states[i, 0, j])
        row_ptr[i + 1] = row_ptr[i] + len(j)
    return row_ptr, np.concatenate(cols), np.concatenate(vals).astype(states.dtype)


@pytest.mark.parametrize("cfg,kw", [(4, {}), (1, {}), (3, dict(n_cols=3_001, m=2))])
def test_expand_round_trip(cfg, kw):
    # the generator's dense minibatch -> its known entries -> expand == the dense known part
    w = make_workload(cfg, **kw)
    st, ob = w.states[0].numpy(), w.obs[0].numpy()
    n, m, ld = st.shape
    row_ptr, col, val = csr_of_observed(st, ob, w.n_cols)
    out = np.full_like(st, 99)
    obs = np.full_like(ob, 7)
    oracle.expand(n, w.n_cols, m, ld, row_ptr, col, val, out, obs)
    assert np.array_equal(obs[:, :w.n_cols], ob[:, :w.n_cols])
    assert not obs[:, w.n_cols:].any()
    ob_valid = ob.copy()
    ob_valid[:, w.n_cols:] = 0  # padding columns are not data
    known = np.broadcast_to(ob_valid[:, None, :].astype(bool), st.shape)
    assert np.array_equal(out[known], st[known])
    assert (out[~known] == 99).all()  # latent and padding entries untouched


def test_expand_edge_cases():
    n, m, ld, n_cols = 3, 2, 8, 6
    st = np.full((n, m, ld), 5, dtype=np.int16)
    obs = np.ones((n, ld), dtype=np.uint8)
    # empty matrix: everything latent, states untouched
    oracle.expand(n, n_cols, m, ld, np.zeros(n + 1, np.int64), np.zeros(0, np.int32),
                  np.zeros(0, np.int16), st, obs)
    assert not obs.any() and (st == 5).all()
    # node 0: columns 1 and 6 (6 >= n_cols is skipped); node 2: column 3 twice, the later wins
    row_ptr = np.array([0, 2, 2, 4], dtype=np.int64)
    col = np.array([1, 6, 3, 3], dtype=np.int32)
    val = np.array([300, 1, 2, 7], dtype=np.int16)
    oracle.expand(n, n_cols, m, ld, row_ptr, col, val, st, obs)
    assert obs.sum() == 2 and obs[0, 1] == 1 and obs[2, 3] == 1
    assert (st[0, :, 1] == 300).all() and (st[2, :, 3] == 7).all()
    assert (st[0, :, 6] == 5).all()


def test_init_latent_uniform_and_observed_untouched():
    card = np.array([2, 3, 5, 7, 8], dtype=np.int32)
    n, m, n_cols = len(card), 3, 20_000
    ld = n_cols
    rng = np.random.default_rng(3)
    obs = (rng.random((n, ld)) < 0.3).astype(np.uint8)
    st = np.full((n, m, ld), -1, dtype=np.int8)
    oracle.init_latent(card, n_cols, m, 0, 12345, st, obs)
    known = np.broadcast_to(obs[:, None, :].astype(bool), st.shape)
    assert (st[known] == -1).all()
    for i, K in enumerate(card):
        x = st[i][~known[i]]
        assert x.min() >= 0 and x.max() < K
        f = np.bincount(x, minlength=K)
        # every state equally likely: chi-square against equal expected counts
        assert stats.chisquare(f).pvalue > 1e-4, (K, f)


def test_init_latent_counter_mapping():
    # the uniform of (node, replica, global column) depends on nothing else:
    # more replicas or a shifted column window reproduce the shared entries
    card = np.array([4, 6, 3], dtype=np.int32)
    n, ld = 3, 64
    obs = np.zeros((n, ld), dtype=np.uint8)
    a = np.zeros((n, 2, ld), dtype=np.int8)
    b = np.zeros((n, 3, ld), dtype=np.int8)
    oracle.init_latent(card, 64, 2, 100, 7, a, obs)
    oracle.init_latent(card, 64, 3, 100, 7, b, obs)
    assert np.array_equal(a, b[:, :2])
    c = np.zeros((n, 2, ld), dtype=np.int8)
    oracle.init_latent(card, 60, 2, 104, 7, c, obs)  # columns 104.. = columns 4.. of a
    assert np.array_equal(c[:, :, :60], a[:, :, 4:64])
    d = np.zeros((n, 2, ld), dtype=np.int8)
    oracle.init_latent(card, 64, 2, 100, 8, d, obs)  # another seed draws other states
    assert (d != a).mean() > 0.5
