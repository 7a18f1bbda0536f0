"""Parity at the benchmark's full size and launch configuration.

The 1000-node random network on one 250,000-column minibatch with m = 10
replicas, generated on the device and stepped exactly as bench.py times it
(same_step with the default options: every colour group's launches, the
count pass with its moving sum, the Dirichlet resample).  The oracle checks:

- sampled column windows of the sweep one by one (at the start, in the
  middle and at the minibatch's end, whose last block of columns is
  partial): columns are independent chains, and a window's draws depend
  only on its global columns, so the oracle sweeps just those columns;
- the counts of the whole minibatch and the moving sum, bit for bit, from
  the library's own post-sweep states;
- the resampled CPTs from those counts.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1511_06416_amd as same
from tests import gpu_helpers as H
from workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


@pytest.mark.parametrize("bits", [0, 4], ids=["8bit", "4bit"])
def test_full_minibatch_step_matches_oracle(bits):
    dev = torch.device("cuda:0")
    w = make_workload(5, device=dev, minibatches=[0])
    net = w.net
    nc, ld, m = w.mb_cols(0), w.ld, w.m
    assert (nc, m, net.n) == (250_000, 10, 1000)
    ctx = H.context_for(net, state_bits=bits)
    ws = ctx.new_workspace(dev)
    pre = w.states[0].clone()
    cpts = torch.from_numpy(w.init_theta).to(dev)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device=dev)
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device=dev)
    sweep_id = update_id = 3
    st = same.pack_states(w.states[0], H.bits_of(ctx))  # the library's replica-quad layout, on the device
    same.same_counts(ctx, st, m, nc, ld, mb, tot, ws)  # the pre-pass
    same.same_step(ctx, st, w.obs[0], cpts, m, nc, ld, 0, w.seed, sweep_id, mb, tot, update_id, ws)
    torch.cuda.synchronize()
    post = H.from_device(ctx, st, m)
    obs = w.obs[0].cpu().numpy()
    color = oracle.graph(net.parents, net.card)["color"]
    assert np.array_equal(ctx.color, color)

    for w0, wl in ((0, 1024), (125_000, 1024), (nc - 1_000, 1_000)):
        st_w = np.ascontiguousarray(pre[:, :, w0:w0 + wl].cpu().numpy())
        ob_w = np.ascontiguousarray(obs[:, w0:w0 + wl])
        res = oracle.sweep(net.parents, net.card, w.init_theta, color, st_w, ob_w, m, wl, w0, w.seed,
                           sweep_id, want_flags=True)
        out = H.compare_states(np.ascontiguousarray(post[:, :, w0:w0 + wl]), st_w, res["flags"], color, wl,
                               obs=ob_w)
        print("window", w0, wl, out)
    assert np.array_equal(post[:, :, nc:], pre[:, :, nc:].cpu().numpy())  # padding untouched

    want = oracle.counts(net.parents, net.card, post, m, nc)
    assert np.array_equal(mb.cpu().numpy(), want)
    assert np.array_equal(tot.cpu().numpy(), want)  # one minibatch: the moving sum is its counts
    theta = oracle.dirichlet(net.parents, net.card, want, w.alpha, w.seed, update_id)
    got = cpts.cpu().numpy()
    assert np.mean(got == theta) >= 1.0 - 1e-5
    assert np.max(np.abs(got.astype(np.float64) - theta) / np.maximum(theta, 1e-30)) <= 1e-6
