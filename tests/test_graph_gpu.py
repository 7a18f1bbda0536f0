"""Replayable step graphs (same_step_graph, same_graph_launch).

A replay runs the kernels of the same_step calls it stands for, with the sweep
and update ids read on the device from a two-word array that the graph
advances after every step.  So each replay must equal those eager calls bit
for bit: states, per-minibatch counts, totals and CPTs.  Every replay is
checked against the eager result, with the eager steps and host
synchronisations between replays, and the id array must end where the eager
ids did.  (The eager same_step is compared with the oracle elsewhere.)
"""
import numpy as np
import pytest
import torch

import paper_1511_06416_amd as same
from tests import gpu_helpers as H
from workloads import make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


class _Run:
    """Device copies of a workload's minibatches with counts initialised by a
    count-only pre-pass."""

    def __init__(self, w, ctx):
        self.states = [H.to_device(ctx, s) for s in w.states]
        self.obs = [o.cuda() for o in w.obs]
        self.ws = ctx.new_workspace()
        self.cpts = torch.from_numpy(w.init_theta).cuda()
        self.mb = torch.zeros((w.M, ctx.cpt_total), dtype=torch.int32, device="cuda")
        self.tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        for b in range(w.M):
            same.same_counts(ctx, self.states[b], w.m, w.mb_cols(b), w.ld, self.mb[b], self.tot, self.ws)


def _assert_equal(E, G, w, what):
    for b in range(w.M):
        assert torch.equal(E.states[b], G.states[b]), (what, "states", b)
    assert torch.equal(E.mb, G.mb), (what, "mb_counts")
    assert torch.equal(E.tot, G.tot), (what, "totals")
    assert torch.equal(E.cpts, G.cpts), (what, "cpts")


@pytest.mark.parametrize("cfg,kw,steps", [
    (1, dict(), 1),                                  # student-2k, m = 1
    (2, dict(n_cols=20_000), 1),                     # student network, m = 10
    (4, dict(), 1),                                  # concepts30-items300-4k, m = 20, full size
    (4, dict(), 3),                                  # three steps per replay
    (3, dict(n_cols=10_000, nb=2_048, m=3), 1),      # 5 minibatches, ragged last one, update stride 5
    (5, dict(n_cols=6_000, nb=1_500, m=2), 2),       # 1000 nodes (every launch class), 4 minibatches
    (5, dict(n_cols=6_000, nb=1_500, m=5, state_bits=4), 1),   # 4-bit states
])
def test_graph_replays_equal_eager(cfg, kw, steps):
    kw = dict(kw)
    bits = kw.pop("state_bits", 0)
    w = make_workload(cfg, **kw)
    ctx = H.context_for(w.net, state_bits=bits)
    E, G = _Run(w, ctx), _Run(w, ctx)
    _assert_equal(E, G, w, "start")
    # minibatch b's ids start at {0, b}; a step moves them by {1, M}
    ids = torch.tensor([[0, b] for b in range(w.M)], dtype=torch.int32, device="cuda")
    graphs = [same.same_step_graph(ctx, G.states[b], G.obs[b], G.cpts, w.m, w.mb_cols(b), w.ld, b * w.nb,
                                   w.seed, G.mb[b], G.tot, ids[b], w.M, steps, G.ws) for b in range(w.M)]
    # capturing runs nothing
    torch.cuda.synchronize()
    _assert_equal(E, G, w, "after capture")
    assert torch.equal(ids[:, 0].cpu(), torch.zeros(w.M, dtype=torch.int32))
    s = 0
    for rep in range(3):
        for b in range(w.M):
            for k in range(steps):
                same.same_step(ctx, E.states[b], E.obs[b], E.cpts, w.m, w.mb_cols(b), w.ld, b * w.nb, w.seed,
                               s + k, E.mb[b], E.tot, (s + k) * w.M + b, E.ws)
        torch.cuda.synchronize()
        for g in graphs:
            g.launch()
        torch.cuda.synchronize()
        _assert_equal(E, G, w, "replay %d" % rep)
        s += steps
        want = np.array([[s, s * w.M + b] for b in range(w.M)], dtype=np.int32)
        assert np.array_equal(ids.cpu().numpy(), want), rep
    for g in graphs:
        g.close()


def test_graph_then_eager_on_the_same_buffers():
    """Replays and eager steps mix on one set of buffers: eager steps with the
    ids the graph would have used continue its sequence exactly."""
    w = make_workload(4)
    ctx = H.context_for(w.net)
    E, G = _Run(w, ctx), _Run(w, ctx)
    ids = torch.tensor([5, 9], dtype=torch.int32, device="cuda")
    g = same.same_step_graph(ctx, G.states[0], G.obs[0], G.cpts, w.m, w.mb_cols(0), w.ld, 0, w.seed, G.mb[0],
                             G.tot, ids, 2, 1, G.ws)
    order = ["graph", "eager", "graph", "graph", "eager"]
    sweep, update = 5, 9
    for how in order:
        same.same_step(ctx, E.states[0], E.obs[0], E.cpts, w.m, w.mb_cols(0), w.ld, 0, w.seed, sweep, E.mb[0],
                       E.tot, update, E.ws)
        if how == "graph":
            g.launch()
        else:
            same.same_step(ctx, G.states[0], G.obs[0], G.cpts, w.m, w.mb_cols(0), w.ld, 0, w.seed, sweep,
                           G.mb[0], G.tot, update, G.ws)
            ids.copy_(torch.tensor([sweep + 1, update + 2], dtype=torch.int32))
        sweep, update = sweep + 1, update + 2
        torch.cuda.synchronize()
        _assert_equal(E, G, w, how)
    g.close()


def test_graph_with_kernel_timing_enabled():
    """Per-launch timing stays on the eager calls: a graph captured while it is
    enabled records no events and replays like any other."""
    w = make_workload(1)
    ctx = H.context_for(w.net)
    E, G = _Run(w, ctx), _Run(w, ctx)
    same.same_kernel_timing(ctx, True)
    ids = torch.tensor([0, 0], dtype=torch.int32, device="cuda")
    g = same.same_step_graph(ctx, G.states[0], G.obs[0], G.cpts, w.m, w.mb_cols(0), w.ld, 0, w.seed, G.mb[0],
                             G.tot, ids, 1, 2, G.ws)
    for s in range(2):
        same.same_step(ctx, E.states[0], E.obs[0], E.cpts, w.m, w.mb_cols(0), w.ld, 0, w.seed, s, E.mb[0],
                       E.tot, s, E.ws)
    g.launch()
    torch.cuda.synchronize()
    kt = same.same_kernel_times(ctx)
    same.same_kernel_timing(ctx, False)
    assert sum(kt["launches"]) > 0           # the eager sweeps were timed
    _assert_equal(E, G, w, "timed")
    g.close()
