"""Out-of-core passes (same_stream_pass): minibatches streamed from pinned
host memory through two device slots must reproduce, bit for bit, the same
call sequence on device-resident minibatches, and follow the oracle's loop."""
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


def _host_arrays(w, bits=None):
    """Pinned host states in the library's layout (replica quads, 4-bit with
    bits=4) and [n][host_ld] obs holding all columns."""
    n = w.net.n
    host_ld = (w.n_cols + 3) // 4 * 4
    full = torch.zeros((n, w.m, host_ld), dtype=w.states[0].dtype)
    ob = torch.ones((n, host_ld), dtype=torch.uint8, pin_memory=True)
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        full[:, :, c0:c0 + nc] = w.states[b][:, :, :nc]
        ob[:, c0:c0 + nc] = w.obs[b][:, :nc]
    return same.pack_states(full, bits).pin_memory(), ob, host_ld


def _resident(w, ctx, passes):
    """The device-resident call sequence; returns the states as [n][m][ld]."""
    dev = [H.to_device(ctx, s) for s in w.states]
    obs = [o.cuda() for o in w.obs]
    ws = ctx.new_workspace()
    cpts = torch.from_numpy(w.init_theta).cuda()
    mb = torch.zeros((w.M, ctx.cpt_total), dtype=torch.int32, device="cuda")
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    for b in range(w.M):
        same.same_counts(ctx, dev[b], w.m, w.mb_cols(b), w.ld, mb[b], tot, ws)
    for s in range(passes):
        for b in range(w.M):
            same.same_sweep(ctx, dev[b], obs[b], cpts, w.m, w.mb_cols(b), w.ld, b * w.nb, w.seed, s,
                            ws)
            same.same_counts(ctx, dev[b], w.m, w.mb_cols(b), w.ld, mb[b], tot, ws)
            same.same_sample_cpts(ctx, tot, cpts, w.seed, s * w.M + b, ws)
    torch.cuda.synchronize()
    return [torch.from_numpy(H.from_device(ctx, d, w.m)) for d in dev], mb.cpu(), tot.cpu(), cpts.cpu()


def _streamed(w, ctx, passes, on_pass=None):
    st, ob, host_ld = _host_arrays(w, H.bits_of(ctx))
    ws = ctx.new_workspace()
    slots = torch.empty(same.same_stream_slots_size(ctx, w.m, w.nb), dtype=torch.uint8, device="cuda")
    cpts = torch.from_numpy(w.init_theta).cuda()
    mb = torch.zeros((w.M, ctx.cpt_total), dtype=torch.int32, device="cuda")
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_stream_pass(ctx, st, ob, host_ld, w.n_cols, w.nb, w.m, cpts, mb, tot, w.seed, 0,
                          same.SAME_STREAM_COUNTS_ONLY, slots, ws)
    for s in range(passes):
        same.same_stream_pass(ctx, st, ob, host_ld, w.n_cols, w.nb, w.m, cpts, mb, tot, w.seed, s, 0,
                              slots, ws)
        if on_pass is not None:
            torch.cuda.synchronize()
            on_pass(s, same.unpack_states(st, w.m, H.bits_of(ctx)), mb, tot, cpts)
    torch.cuda.synchronize()
    return same.unpack_states(st, w.m, H.bits_of(ctx)), mb.cpu(), tot.cpu(), cpts.cpu()


@pytest.mark.parametrize("cfg,kw", [
    (3, dict(n_cols=10_000, nb=2_048, m=3)),     # 5 minibatches, ragged last one
    (5, dict(n_cols=6_000, nb=1_500, m=2)),      # 1000 nodes, 4 minibatches
    (1, dict(n_cols=1_000, nb=4_096, m=2)),      # one minibatch smaller than nb
])
@pytest.mark.parametrize("bits", [0, 4], ids=["8bit", "4bit"])
def test_stream_equals_resident(cfg, kw, bits):
    w = make_workload(cfg, **kw)
    ctx = H.context_for(w.net, state_bits=bits)
    res_states, res_mb, res_tot, res_cpts = _resident(w, ctx, passes=2)
    st, mb, tot, cpts = _streamed(w, ctx, passes=2)
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        assert torch.equal(st[:, :, c0:c0 + nc], res_states[b][:, :, :nc]), b
    assert torch.equal(mb, res_mb)
    assert torch.equal(tot, res_tot)
    assert torch.equal(cpts, res_cpts)


def test_stream_follows_oracle_loop():
    """Streamed passes and the oracle's loop run independently from the same
    inputs; they must agree pass by pass until a flagged boundary draw (if
    any) makes them diverge."""
    w = make_workload(1, n_cols=2_000, nb=500, m=2)
    net = w.net
    ctx = H.context_for(net)
    color = oracle.graph(net.parents, net.card)["color"]
    theta = w.init_theta.copy()
    states = [s.numpy().copy() for s in w.states]
    obs = [o.numpy() for o in w.obs]
    mbs = [oracle.counts(net.parents, net.card, states[b], w.m, w.mb_cols(b)) for b in range(w.M)]
    totals = np.sum(mbs, axis=0)
    state = {"diverged": False, "checked": 0}

    def on_pass(s, st, mb, tot, cpts):
        nonlocal theta, totals
        if state["diverged"]:
            return
        flags = []
        for b in range(w.M):
            res = oracle.sweep(net.parents, net.card, theta, color, states[b], obs[b], w.m,
                               w.mb_cols(b), b * w.nb, w.seed, s, want_flags=True)
            flags.append(res["flags"])
            new = oracle.counts(net.parents, net.card, states[b], w.m, w.mb_cols(b))
            totals = oracle.moving_sum(totals, mbs[b], new)
            mbs[b] = new
            theta = oracle.dirichlet(net.parents, net.card, totals, w.alpha, w.seed, s * w.M + b)
        host = st.numpy()
        for b in range(w.M):
            c0, nc = b * w.nb, w.mb_cols(b)
            got = np.ascontiguousarray(host[:, :, c0:c0 + nc])
            if not np.array_equal(got, states[b][:, :, :nc]):
                # the first divergence must be a flagged draw
                H.compare_states(np.ascontiguousarray(np.pad(got, ((0, 0), (0, 0), (0, w.ld - nc)))),
                                 np.ascontiguousarray(np.pad(states[b][:, :, :nc],
                                                             ((0, 0), (0, 0), (0, w.ld - nc)))),
                                 flags[b], color, nc)
                state["diverged"] = True
                return
        assert np.array_equal(tot.cpu().numpy(), totals)
        assert np.array_equal(mb.cpu().numpy(), np.array(mbs))
        g_th = cpts.cpu().numpy()
        assert np.mean(g_th == theta) >= 1.0 - 1e-5
        state["checked"] += 1
        if not np.array_equal(g_th, theta):
            # a last-bit difference of the fp64 Gamma variates: the runs part here
            state["diverged"] = True

    _streamed(w, ctx, passes=4, on_pass=on_pass)
    assert state["checked"] >= 1 or state["diverged"]


def _compact_case(w, ctx, passes):
    """Compact-state passes: the known data on the device, the latent replica
    states compacted on the host (built here with numpy from the dense
    minibatches); returns the dense states expanded back from the compact host
    array after the passes, and the counts, totals and CPTs."""
    n, m = w.net.n, w.m
    ld_dev = (w.n_cols + 3) // 4 * 4
    obs = np.ones((n, ld_dev), dtype=np.uint8)
    data = np.zeros((n, ld_dev), dtype=w.states[0].numpy().dtype)
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        obs[:, c0:c0 + nc] = w.obs[b].numpy()[:, :nc]
        data[:, c0:c0 + nc] = w.states[b].numpy()[:, 0, :nc]
    d_obs = torch.from_numpy(obs).cuda()
    d_data = torch.from_numpy(data).cuda()
    ws = ctx.new_workspace()
    off, slot_bytes = same.same_stream_compact_layout(ctx, d_obs, ld_dev, w.n_cols, w.nb, m, ws)
    # the compact host array: per (minibatch, node), replica-major latent states
    host = np.zeros(int(off[-1]), dtype=data.dtype)
    latcols = {}
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        st = w.states[b].numpy()
        for i in range(n):
            cols = np.nonzero(obs[i, c0:c0 + nc] == 0)[0]
            latcols[b, i] = cols
            L = len(cols)
            assert off[b * n + i + 1] - off[b * n + i] == m * L
            host[off[b * n + i]:off[b * n + i] + m * L] = st[i][:, cols].reshape(-1)
    lat = torch.from_numpy(host).pin_memory() if host.size else torch.zeros(1, dtype=torch.int8).pin_memory()
    slots = torch.empty(slot_bytes, dtype=torch.uint8, device="cuda")
    cpts = torch.from_numpy(w.init_theta).cuda()
    mb = torch.zeros((w.M, ctx.cpt_total), dtype=torch.int32, device="cuda")
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_stream_pass_compact(ctx, lat, off, d_obs, d_data, ld_dev, w.n_cols, w.nb, m, cpts, mb, tot, w.seed,
                                  0, same.SAME_STREAM_COUNTS_ONLY, slots, ws)
    for s in range(passes):
        same.same_stream_pass_compact(ctx, lat, off, d_obs, d_data, ld_dev, w.n_cols, w.nb, m, cpts, mb, tot,
                                      w.seed, s, 0, slots, ws)
    torch.cuda.synchronize()
    out = lat.numpy()
    dense = []
    for b in range(w.M):
        c0, nc = b * w.nb, w.mb_cols(b)
        d = np.repeat(data[:, None, c0:c0 + nc], m, axis=1).copy()
        for i in range(n):
            cols = latcols[b, i]
            d[i][:, cols] = out[off[b * n + i]:off[b * n + i] + m * len(cols)].reshape(m, len(cols))
        dense.append(d)
    return dense, mb.cpu(), tot.cpu(), cpts.cpu()


@pytest.mark.parametrize("cfg,kw", [
    (3, dict(n_cols=10_000, nb=2_048, m=3)),     # ragged last minibatch, m not a multiple of 4
    (5, dict(n_cols=6_000, nb=1_500, m=2)),
    (1, dict(n_cols=1_000, nb=4_096, m=2)),
    (4, dict(n_cols=3_000, nb=1_000, m=5)),      # concepts never observed
])
@pytest.mark.parametrize("bits", [0, 4], ids=["8bit", "4bit"])
def test_compact_stream_equals_resident(cfg, kw, bits):
    """Out-of-core passes that move only the compacted latent states over PCIe
    (known data resident on the device) equal the device-resident call
    sequence bit for bit: states, per-minibatch counts, totals and CPTs."""
    w = make_workload(cfg, **kw)
    ctx = H.context_for(w.net, state_bits=bits)
    res_states, res_mb, res_tot, res_cpts = _resident(w, ctx, passes=2)
    dense, mb, tot, cpts = _compact_case(w, ctx, passes=2)
    for b in range(w.M):
        nc = w.mb_cols(b)
        assert np.array_equal(dense[b], res_states[b].numpy()[:, :, :nc]), b
    assert torch.equal(mb, res_mb)
    assert torch.equal(tot, res_tot)
    assert torch.equal(cpts, res_cpts)
