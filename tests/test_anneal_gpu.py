"""GPU parity of SAME replica growth (Sec. 3 annealing) through the C ABI:
bit-exact against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_1511_06416_amd as same
from tests import gpu_helpers as H
from workloads import Network, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


@pytest.mark.parametrize("cfg,kw,m2", [(4, dict(m=2), 7), (5, dict(n_cols=3_001, m=3), 10), (1, {}, 1)])
def test_grow_replicas_matches_oracle(cfg, kw, m2):
    w = make_workload(cfg, **kw)
    st = w.states[0].numpy()
    ref = oracle.grow_replicas(st, m2)
    ctx = H.context_for(w.net)
    dst = torch.full(same.state_shape(w.net.n, m2, w.ld), 77, dtype=w.states[0].dtype, device="cuda")
    same.same_grow_replicas(ctx, same.pack_states(w.states[0]).cuda(), w.m, dst, m2, w.ld)
    torch.cuda.synchronize()
    assert np.array_equal(same.unpack_states(dst.cpu().numpy(), m2), ref)
    # padding slots of the last destination quad follow the same rule (a valid state)
    full = same.unpack_states(dst.cpu().numpy(), 4 * ((m2 + 3) // 4))
    for r in range(m2, full.shape[1]):
        assert np.array_equal(full[:, r], st[:, r % w.m])
    ctx.close()


def test_grow_replicas_int16_ragged_rows():
    card = np.array([300, 3], dtype=np.int32)
    ctx = H.context_for(Network("custom", [[], [0]], card))
    rng = np.random.default_rng(4)
    st = rng.integers(0, 3, (2, 3, 20)).astype(np.int16)  # 20 columns, m = 3 grown to 5
    ref = oracle.grow_replicas(st, 5)
    dst = torch.zeros(same.state_shape(2, 5, 20), dtype=torch.int16, device="cuda")
    same.same_grow_replicas(ctx, torch.from_numpy(same.pack_states(st)).cuda(), 3, dst, 5, 20)
    torch.cuda.synchronize()
    assert np.array_equal(same.unpack_states(dst.cpu().numpy(), 5), ref)
    ctx.close()


@pytest.mark.parametrize("m,m2", [(2, 7), (3, 10), (5, 5)])
def test_grow_replicas_4bit(m, m2):
    w = make_workload(5, n_cols=2_001, m=m)
    st = w.states[0].numpy()
    ref = oracle.grow_replicas(st, m2)
    ctx = H.context_for(w.net, state_bits=4)
    dst = torch.full(same.state_shape(w.net.n, m2, w.ld, 4), -1, dtype=torch.int16, device="cuda")
    same.same_grow_replicas(ctx, H.to_device(ctx, st), m, dst, m2, w.ld)
    torch.cuda.synchronize()
    assert np.array_equal(H.from_device(ctx, dst, m2), ref)
    ctx.close()
