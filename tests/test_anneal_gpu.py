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
    dst = torch.full(ref.shape, 77, dtype=w.states[0].dtype, device="cuda")
    same.same_grow_replicas(ctx, w.states[0].cuda(), w.m, dst, m2, w.ld)
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy(), ref)
    ctx.close()


def test_grow_replicas_int16_ragged_rows():
    card = np.array([300, 3], dtype=np.int32)
    ctx = H.context_for(Network("custom", [[], [0]], card))
    rng = np.random.default_rng(4)
    st = rng.integers(0, 3, (2, 3, 20)).astype(np.int16)  # rows of 40 bytes: 16-byte pieces and a tail
    ref = oracle.grow_replicas(st, 5)
    dst = torch.zeros(ref.shape, dtype=torch.int16, device="cuda")
    same.same_grow_replicas(ctx, torch.from_numpy(st).cuda(), 3, dst, 5, 20)
    torch.cuda.synchronize()
    assert np.array_equal(dst.cpu().numpy(), ref)
    ctx.close()
