"""GPU parity of the data-ingest entry points against the oracle, through the
C ABI: the dense minibatch expanded from the known entries of the (typically
sparse) node x case matrix (Sec. 4) and the random initial latent states
(Sec. 5.2).  Both are integer work: the bar is bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import paper_1511_06416_amd as same
from tests import gpu_helpers as H
from tests.test_oracle_ingest import csr_of_observed
from workloads import Network, make_network, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


def _expand_case(net, st, ob, n_cols, m, sentinel=99):
    n, _, ld = st.shape
    row_ptr, col, val = csr_of_observed(st, ob, n_cols)
    ref_st = np.full_like(st, sentinel)
    ref_ob = np.full_like(ob, 3)
    oracle.expand(n, n_cols, m, ld, row_ptr, col, val, ref_st, ref_ob)
    ctx = H.context_for(net)
    g_st = torch.full(same.state_shape(n, m, ld), sentinel, dtype=torch.from_numpy(st[:1, :1, :1]).dtype,
                      device="cuda")
    g_ob = torch.full(ob.shape, 3, dtype=torch.uint8, device="cuda")
    rp, ci, vv = (torch.from_numpy(a).cuda() for a in (row_ptr, col, val))
    same.same_expand_observed(ctx, rp, ci, vv, len(col), m, n_cols, ld, g_st, g_ob)
    torch.cuda.synchronize()
    assert np.array_equal(g_ob.cpu().numpy(), ref_ob)
    assert np.array_equal(same.unpack_states(g_st.cpu().numpy(), m), ref_st)
    ctx.close()
    return len(col)


@pytest.mark.parametrize("cfg,kw", [(4, {}), (1, {}), (5, dict(n_cols=3_001, m=3)), (3, dict(n_cols=5_000))])
def test_expand_matches_oracle(cfg, kw):
    w = make_workload(cfg, **kw)
    nnz = _expand_case(w.net, w.states[0].numpy(), w.obs[0].numpy(), w.n_cols, w.m)
    assert nnz > 0


def test_expand_int16_empty_rows_and_no_entries():
    parents = [[], [0], [0, 1], [2], [1]]
    card = np.array([130, 3, 200, 2, 5], dtype=np.int32)
    rng = np.random.default_rng(11)
    n, m, n_cols, ld = 5, 2, 301, 304
    st = np.zeros((n, m, ld), dtype=np.int16)
    ob = (rng.random((n, ld)) < 0.4).astype(np.uint8)
    ob[3] = 0  # a node with no known entry
    for i in range(n):
        st[i, :, :] = rng.integers(0, card[i], ld)[None, :]
    net = Network("custom", parents, card)
    _expand_case(net, st, ob, n_cols, m, sentinel=1000)
    _expand_case(net, st, np.zeros_like(ob), n_cols, m, sentinel=1000)  # nnz = 0


@pytest.mark.parametrize("cfg,kw,col_offset", [(5, dict(n_cols=2_003, m=3), 0), (4, {}, 4096),
                                                (1, {}, (1 << 33) + 8)])
def test_init_latent_matches_oracle(cfg, kw, col_offset):
    w = make_workload(cfg, **kw)
    st, ob = w.states[0].numpy().copy(), w.obs[0].numpy()
    ref = st.copy()
    oracle.init_latent(w.net.card, w.n_cols, w.m, col_offset, w.seed, ref, ob)
    ctx = H.context_for(w.net)
    g = torch.from_numpy(same.pack_states(st)).cuda()
    same.same_init_latent(ctx, g, torch.from_numpy(ob).cuda(), w.m, w.n_cols, w.ld, col_offset, w.seed)
    torch.cuda.synchronize()
    assert np.array_equal(same.unpack_states(g.cpu().numpy(), w.m), ref)
    ctx.close()


def test_init_latent_int16():
    parents = [[], [0], [0, 1]]
    card = np.array([300, 7, 2], dtype=np.int32)
    n, m, n_cols, ld = 3, 4, 1001, 1004
    rng = np.random.default_rng(2)
    ob = (rng.random((n, ld)) < 0.5).astype(np.uint8)
    st = np.full((n, m, ld), -5, dtype=np.int16)
    ref = st.copy()
    oracle.init_latent(card, n_cols, m, 12, 99, ref, ob)
    ctx = H.context_for(Network("custom", parents, card))
    g = torch.from_numpy(same.pack_states(st)).cuda()
    same.same_init_latent(ctx, g, torch.from_numpy(ob).cuda(), m, n_cols, ld, 12, 99)
    torch.cuda.synchronize()
    assert np.array_equal(same.unpack_states(g.cpu().numpy(), m), ref)
    ctx.close()


@pytest.mark.parametrize("cfg,kw", [(4, {}), (5, dict(n_cols=3_001, m=3))])
def test_expand_and_init_latent_4bit(cfg, kw):
    """4-bit states: the expanded known part and the random start equal the
    oracle's (latent entries of the expansion keep their value)."""
    w = make_workload(cfg, **kw)
    net = w.net
    st, ob = w.states[0].numpy(), w.obs[0].numpy()
    n, m, ld = st.shape
    row_ptr, col, val = csr_of_observed(st, ob, w.n_cols)
    ref_st = np.full_like(st, 9)
    ref_ob = np.full_like(ob, 3)
    oracle.expand(n, w.n_cols, m, ld, row_ptr, col, val, ref_st, ref_ob)
    ctx = H.context_for(net, state_bits=4)
    g_st = H.to_device(ctx, np.full_like(st, 9))
    g_ob = torch.full(ob.shape, 3, dtype=torch.uint8, device="cuda")
    rp, ci, vv = (torch.from_numpy(a).cuda() for a in (row_ptr, col, val))
    same.same_expand_observed(ctx, rp, ci, vv, len(col), m, w.n_cols, ld, g_st, g_ob)
    torch.cuda.synchronize()
    assert np.array_equal(g_ob.cpu().numpy(), ref_ob)
    assert np.array_equal(H.from_device(ctx, g_st, m), ref_st)
    ref = st.copy()
    oracle.init_latent(net.card, w.n_cols, m, 4096, w.seed, ref, ob)
    g = H.to_device(ctx, st)
    same.same_init_latent(ctx, g, torch.from_numpy(ob).cuda(), m, w.n_cols, ld, 4096, w.seed)
    torch.cuda.synchronize()
    assert np.array_equal(H.from_device(ctx, g, m), ref)
    ctx.close()
