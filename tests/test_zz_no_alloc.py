"""The allocation-free count entry point, same_counts_noalloc, against
same_counts (the entry point whose kernels it shares), through the C ABI.

Counts are integer work, so the bar is bit equality of the new per-minibatch
counts and of the moving-sum totals, on two calls in a row on the same
device (the second on a smaller minibatch, so that the scratch array still
holds the first call's larger histogram), plus the documented errors.
"""
import numpy as np
import pytest
import torch

import paper_1511_06416_amd as same
from tests import gpu_helpers as H
from workloads import Network, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


def _both(ctx, st, m, n_cols, ld, prev, tot0):
    """(mb, totals) from same_counts and from same_counts_noalloc on copies."""
    out = []
    for noalloc in (False, True):
        mb = torch.from_numpy(prev.copy()).cuda()
        tot = torch.from_numpy(tot0.copy()).cuda()
        if noalloc:
            same.same_counts_noalloc(ctx, st, m, n_cols, ld, mb, tot)
        else:
            same.same_counts(ctx, st, m, n_cols, ld, mb, tot, ctx.new_workspace())
        torch.cuda.synchronize()
        out.append((mb.cpu().numpy(), tot.cpu().numpy()))
    return out


@pytest.mark.parametrize("cfg,kw", [(5, dict(n_cols=9_000, m=10)), (3, dict(n_cols=20_001, m=5))])
def test_noalloc_counts_equal_same_counts(cfg, kw):
    w = make_workload(cfg, **kw)
    ctx = H.context_for(w.net)
    rng = np.random.default_rng(cfg)
    st = same.pack_states(w.states[0]).cuda()
    # first call: the whole minibatch; second: a smaller column range
    for n_cols in (w.mb_cols(0), w.mb_cols(0) // 3 + 1):
        prev = rng.integers(0, 500, ctx.cpt_total).astype(np.int32)
        tot0 = (prev + rng.integers(0, 500, ctx.cpt_total)).astype(np.int32)
        (mb_a, tot_a), (mb_b, tot_b) = _both(ctx, st, w.m, n_cols, w.ld, prev, tot0)
        assert np.array_equal(mb_a, mb_b)
        assert np.array_equal(tot_a, tot_b)
        off = ctx.cpt_off
        assert all(mb_b[off[i]:off[i + 1]].sum() == n_cols * w.m for i in range(w.net.n))


def test_noalloc_counts_without_totals_and_int16():
    parents = [[], [0], [0, 1], [2], [1, 2, 3]]
    card = [130, 3, 200, 2, 5]
    rng = np.random.default_rng(9)
    n_cols, ld, m = 4097, 4100, 3
    st = np.zeros((5, m, ld), dtype=np.int16)
    for i, k in enumerate(card):
        st[i, :, :n_cols] = rng.integers(0, k, (m, n_cols))
    st[:, :, n_cols:] = 120
    ctx = H.context_for(Network("custom", parents, card))
    d_st = torch.from_numpy(same.pack_states(st)).cuda()
    for cols in (n_cols, 1001):
        a = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        b = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        same.same_counts(ctx, d_st, m, cols, ld, a, None, ctx.new_workspace())
        same.same_counts_noalloc(ctx, d_st, m, cols, ld, b, None)
        torch.cuda.synchronize()
        assert np.array_equal(a.cpu().numpy(), b.cpu().numpy())


def test_noalloc_errors():
    # a context whose tables were never put on the device: rejected, not uploaded
    w = make_workload(1, n_cols=64)
    ctx = H.context_for(w.net)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    st = same.pack_states(w.states[0]).cuda()
    with pytest.raises(same.SameError) as e:
        same.same_counts_noalloc(ctx, st, w.m, 64, w.ld, mb, None)
    assert e.value.code == same.SAME_EINVAL
    # a CPT as large as the scratch array (6 parents of 8 states, 8 states of
    # its own: 8^7 = 2^21 entries) plus the parents' 48 entries
    parents = [[] for _ in range(6)] + [list(range(6))]
    big = H.context_for(Network("big", parents, [8] * 7))
    assert big.cpt_total > (1 << 21)
    with pytest.raises(same.SameError) as e:
        same.same_counts_noalloc(big, torch.zeros(same.state_shape(7, 1, 4), dtype=torch.int8, device="cuda"), 1, 4, 4,
                                 torch.zeros(8, dtype=torch.int32, device="cuda"), None)
    assert e.value.code == same.SAME_ESIZE


def test_noalloc_counts_4bit():
    """4-bit states: same_counts_noalloc equals same_counts on two calls in a
    row, the second over fewer columns."""
    w = make_workload(5, n_cols=9_000, m=10)
    ctx = H.context_for(w.net, state_bits=4)
    rng = np.random.default_rng(44)
    st = H.to_device(ctx, w.states[0])
    for n_cols in (w.mb_cols(0), w.mb_cols(0) // 3 + 1):
        prev = rng.integers(0, 500, ctx.cpt_total).astype(np.int32)
        tot0 = (prev + rng.integers(0, 500, ctx.cpt_total)).astype(np.int32)
        (mb_a, tot_a), (mb_b, tot_b) = _both(ctx, st, w.m, n_cols, w.ld, prev, tot0)
        assert np.array_equal(mb_a, mb_b)
        assert np.array_equal(tot_a, tot_b)
