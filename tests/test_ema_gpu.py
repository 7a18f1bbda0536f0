"""GPU parity of the exponential moving sum of the counts (Sec. 4 footnote)
through the C ABI: the fp64 totals bit-exact against the oracle, the Dirichlet
resample from them to the resample bar, and the out-of-core pass with the
moving sum equal, bit for bit, to the same calls on resident minibatches."""
import numpy as np
import pytest
import torch

import oracle
import paper_1511_06416_amd as same
from tests import gpu_helpers as H
from tests.test_stream_gpu import _host_arrays
from workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


@pytest.mark.parametrize("cfg,kw,decay", [(5, dict(n_cols=3_001, m=3), 0.875), (4, {}, 0.0), (2, dict(n_cols=9_000), 1.0)])
def test_counts_ema_bit_exact(cfg, kw, decay):
    w = make_workload(cfg, **kw)
    net = w.net
    ctx = H.context_for(net)
    ws = ctx.new_workspace()
    st = w.states[0].numpy()
    t0 = np.random.default_rng(cfg).random(ctx.cpt_total) * 1000.0
    ref = t0.copy()
    oracle.ema(ref, decay, oracle.counts(net.parents, net.card, st, w.m, w.mb_cols(0)))
    g = torch.from_numpy(t0).cuda()
    same.same_counts_ema(ctx, same.pack_states(w.states[0]).cuda(), w.m, w.mb_cols(0), w.ld, decay, g, ws)
    torch.cuda.synchronize()
    assert np.array_equal(g.cpu().numpy(), ref)
    ctx.close()


@pytest.mark.parametrize("cfg", [1, 3, 5])
def test_sample_cpts_ema_matches_oracle(cfg):
    net = make_workload(cfg, n_cols=8, minibatches=[]).net
    ctx = H.context_for(net)
    ws = ctx.new_workspace()
    tot = np.random.default_rng(7).random(ctx.cpt_total) * 50.0  # fractional moving sums
    want = oracle.dirichlet_f64(net.parents, net.card, tot, 1.0, 33, 9)
    got = torch.empty(ctx.cpt_total, dtype=torch.float32, device="cuda")
    same.same_sample_cpts_ema(ctx, torch.from_numpy(tot).cuda(), got, 33, 9, ws)
    torch.cuda.synchronize()
    got = got.cpu().numpy()
    assert np.mean(got == want) >= 1 - 1e-5
    np.testing.assert_allclose(got, want, rtol=1e-6, atol=0)
    ctx.close()


@pytest.mark.parametrize("bits", [0, 4], ids=["8bit", "4bit"])
def test_stream_pass_ema_equals_resident(bits):
    w = make_workload(3, n_cols=9_001, nb=3_000, m=3)
    ctx = H.context_for(w.net, state_bits=bits)
    M = w.M
    decay = 1.0 - 1.0 / M
    passes = 2
    # resident: the same calls in the same order on device minibatches
    dev = [H.to_device(ctx, s) for s in w.states]
    obs = [o.cuda() for o in w.obs]
    ws = ctx.new_workspace()
    cpts = torch.from_numpy(w.init_theta).cuda()
    tot = torch.zeros(ctx.cpt_total, dtype=torch.float64, device="cuda")
    for b in range(M):
        same.same_counts_ema(ctx, dev[b], w.m, w.mb_cols(b), w.ld, decay, tot, ws)
    for s in range(passes):
        for b in range(M):
            same.same_sweep(ctx, dev[b], obs[b], cpts, w.m, w.mb_cols(b), w.ld, b * w.nb, w.seed, s, ws)
            same.same_counts_ema(ctx, dev[b], w.m, w.mb_cols(b), w.ld, decay, tot, ws)
            same.same_sample_cpts_ema(ctx, tot, cpts, w.seed, s * M + b, ws)
    torch.cuda.synchronize()
    # streamed from pinned host memory
    hst, hob, host_ld = _host_arrays(w, H.bits_of(ctx))
    ws2 = ctx.new_workspace()
    slots = torch.empty(same.same_stream_slots_size(ctx, w.m, w.nb), dtype=torch.uint8, device="cuda")
    cp2 = torch.from_numpy(w.init_theta).cuda()
    tot2 = torch.zeros(ctx.cpt_total, dtype=torch.float64, device="cuda")
    same.same_stream_pass_ema(ctx, hst, hob, host_ld, w.n_cols, w.nb, w.m, cp2, tot2, decay, w.seed, 0,
                              same.SAME_STREAM_COUNTS_ONLY, slots, ws2)
    for s in range(passes):
        same.same_stream_pass_ema(ctx, hst, hob, host_ld, w.n_cols, w.nb, w.m, cp2, tot2, decay, w.seed, s, 0,
                                  slots, ws2)
    torch.cuda.synchronize()
    assert np.array_equal(tot2.cpu().numpy(), tot.cpu().numpy())
    assert np.array_equal(cp2.cpu().numpy(), cpts.cpu().numpy())
    hs = same.unpack_states(hst, w.m, H.bits_of(ctx))
    for b in range(M):
        c0, nc = b * w.nb, w.mb_cols(b)
        assert np.array_equal(hs[:, :, c0:c0 + nc].numpy(), H.from_device(ctx, dev[b], w.m)[:, :, :nc])
    ctx.close()
