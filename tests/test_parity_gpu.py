"""GPU parity: libsame (through the C ABI) against the oracle on the same
seeded inputs.

Bars: conditionals within 1e-5 relative (fp32 library vs fp64 oracle, where
the oracle's probability is >= 1e-30); sampled states identical except where
a chain's first differing draw is one whose uniform lies within 1e-6 of a CDF
boundary (the oracle flags those); counts bit-exact; Dirichlet resample equal
in fp32 (both sides draw the Gamma variates in fp64).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1511_06416_amd as same
from tests import brute, gpu_helpers as H
from tests import oracle_loop
from workloads import Network, make_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    same.load_library()


def _sweep_case(w, b=0, sweep_id=3, win=None, theta=None, n_threads=0, table_limit=None, **ctx_kw):
    net = w.net
    ctx = H.context_for(net, table_limit=table_limit, **ctx_kw)
    color = oracle.graph(net.parents, net.card)["color"]
    assert np.array_equal(ctx.color, color)
    theta = w.init_theta if theta is None else theta
    pre = w.states[b].cpu().numpy()
    obs = w.obs[b].cpu().numpy()
    ncols = w.mb_cols(b)
    gpu, dbg, gp = H.gpu_sweep_both(ctx, pre, obs, theta, w.m, ncols, b * w.nb, w.seed, sweep_id, win=win)
    ref = pre.copy()
    res = oracle.sweep(net.parents, net.card, theta, color, ref, obs, w.m, ncols, b * w.nb,
                       w.seed, sweep_id, want_flags=True, win=win, n_threads=n_threads)
    # the production kernels, then the debug build that wrote the conditionals
    st = H.compare_states(gpu, ref, res["flags"], color, ncols, obs=obs)
    out = {"states": st, "draws": res["draws"]}
    if win is not None:
        out["debug_states"] = H.compare_states(dbg, ref, res["flags"], color, ncols, obs=obs)
        div = H.diverged_chains(dbg, ref, ncols, win)
        out["probs"] = H.compare_probs(gp, res["probs"], obs, net.card, win, div)
    print(w.name, out)
    return out


# ------------------------------------------------------------ sweep parity

@pytest.mark.parametrize("cfg,kw,win", [
    (1, {}, (0, 2000)),                                  # student 2k, m=1, full window
    (2, dict(n_cols=20_000), (1000, 3000)),              # student, m=10
    (3, dict(n_cols=9_000), (8_000, 1000)),              # 100-node random DAG, ragged tail
    (4, {}, (0, 600)),                                   # two-layer concepts, m=20
    (5, dict(n_cols=5_000), (4_600, 400)),               # 1000-node random DAG, m=10
    (5, dict(n_cols=3_000, m=5), (0, 300)),              # odd m: a replica quad, then a partial one
    (5, dict(n_cols=2_001, m=7), (1_700, 301)),          # odd m and a ragged tail
])
@pytest.mark.parametrize("table_limit", [None, 0], ids=["tables", "products"])
def test_sweep_parity_configs(cfg, kw, win, table_limit):
    w = make_workload(cfg, **kw)
    out = _sweep_case(w, win=win, table_limit=table_limit)
    assert out["probs"]["checked"] > 0


@pytest.mark.parametrize("cfg,kw,win", [
    (2, dict(n_cols=6_000), (1000, 600)),
    (3, dict(n_cols=9_001), (8_000, 1001)),              # ragged tail
    (4, {}, (0, 600)),
    (5, dict(n_cols=3_000, m=4), (2_600, 400)),
])
@pytest.mark.parametrize("variant", [dict(lds_limit=0), dict(lds_limit=1024), dict(lds_limit=4096),
                                     dict(packed=False), dict(lds_limit=0, packed=False)],
                         ids=["global-tables", "mixed-tables", "partial-records", "wide-indices", "global-wide"])
def test_sweep_parity_kernel_classes(cfg, kw, win, variant):
    """The same conditionals and draws when every table is read from global
    memory, when a colour's nodes split between LDS-staged and global tables
    (two concurrent launches per colour), when records larger than the LDS
    budget stage only their smallest CPT groups and gather the rest from
    global memory, and/or every product-mode node takes the 32-bit index
    kernel."""
    w = make_workload(cfg, **kw)
    out = _sweep_case(w, win=win, **variant)
    assert out["probs"]["checked"] > 0


def test_sweep_parity_second_minibatch_offset():
    # minibatch 1 of a 3-minibatch split: global columns start at nb
    w = make_workload(3, n_cols=6_000, nb=2_000, m=3, minibatches=[1])
    _sweep_case(w, b=1, sweep_id=11, win=(500, 300))


def test_sweep_parity_after_resampled_cpts():
    # CPTs as the sampler produces them (Dirichlet draws from counts), not Dir(1)
    w = make_workload(5, n_cols=3_000, m=4)
    net = w.net
    tot = oracle.counts(net.parents, net.card, w.states[0].numpy(), w.m, w.mb_cols(0))
    theta = oracle.dirichlet(net.parents, net.card, tot, 1.0, 5, 0)
    _sweep_case(w, theta=theta, win=(0, 256))


def test_column_tiles_and_step_are_bit_identical():
    """A sweep split into column tiles equals the untiled sweep, same_step
    equals same_sweep + same_counts + same_sample_cpts, and the tiled sweep
    matches the oracle."""
    w = make_workload(5, n_cols=5_000, m=2)
    net = w.net
    pre, obs = w.states[0].numpy(), w.obs[0].numpy()
    tiled = H.context_for(net, tile_bytes=1)          # 1024-column tiles
    assert same.same_sweep_plan(tiled, w.m, 5_000)[0] == 1024
    whole = H.context_for(net)
    a, _ = H.gpu_sweep(tiled, pre, obs, w.init_theta, w.m, 5_000, 0, 9, 2)
    b, _ = H.gpu_sweep(whole, pre, obs, w.init_theta, w.m, 5_000, 0, 9, 2)
    assert np.array_equal(a, b)
    _sweep_case(w, win=(3_000, 600), sweep_id=2)
    outs = []
    for ctx, fused in ((tiled, True), (whole, False)):
        st = same.pack_states(w.states[0]).cuda()
        ob = w.obs[0].cuda()
        th = torch.from_numpy(w.init_theta).cuda()
        mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        ws = ctx.new_workspace()
        same.same_counts(ctx, st, w.m, 5_000, w.ld, mb, tot, ws)
        for s in range(2):
            if fused:
                same.same_step(ctx, st, ob, th, w.m, 5_000, w.ld, 0, w.seed, s, mb, tot, s, ws)
            else:
                same.same_sweep(ctx, st, ob, th, w.m, 5_000, w.ld, 0, w.seed, s, ws)
                same.same_counts(ctx, st, w.m, 5_000, w.ld, mb, tot, ws)
                same.same_sample_cpts(ctx, tot, th, w.seed, s, ws)
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy() for x in (st, mb, tot, th)])
    for x, y in zip(*outs):
        assert np.array_equal(x, y)


def test_sweep_deterministic_and_stream_independent():
    w = make_workload(3, n_cols=4_100, m=2)
    ctx = H.context_for(w.net)
    pre, obs = w.states[0].numpy(), w.obs[0].numpy()
    a, _ = H.gpu_sweep(ctx, pre, obs, w.init_theta, w.m, 4_100, 0, 9, 1)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b, _ = H.gpu_sweep(ctx, pre, obs, w.init_theta, w.m, 4_100, 0, 9, 1, stream=s)
    assert np.array_equal(a, b)


# ------------------------------------------------------------ edge cases

def _custom(parents, card, n_cols, m, hidden, seed, ld=None, theta=None, alpha=0.8):
    rng = np.random.default_rng(seed)
    card = np.asarray(card, dtype=np.int32)
    ld = ld or ((n_cols + 3) // 4 * 4)
    n = len(parents)
    dt = np.int8 if card.max() <= 127 else np.int16
    states = np.zeros((n, m, ld), dtype=dt)
    obs = np.ones((n, ld), dtype=np.uint8)
    for i in range(n):
        obs[i, :n_cols] = (rng.random(n_cols) >= hidden).astype(np.uint8)
        data = rng.integers(0, card[i], n_cols)
        for r in range(m):
            states[i, r, :n_cols] = np.where(obs[i, :n_cols] == 1, data,
                                             rng.integers(0, card[i], n_cols))
    if theta is None:
        theta = brute.random_theta(rng, parents, card, alpha=alpha)
    return Network("custom", parents, card), states, obs, theta


def _custom_case(net, states, obs, theta, m, n_cols, col_offset=0, win=None, sweep_id=1, seed=5,
                 table_limit=None, **ctx_kw):
    ctx = H.context_for(net, table_limit=table_limit, **ctx_kw)
    color = oracle.graph(net.parents, net.card)["color"]
    gpu, dbg, gp = H.gpu_sweep_both(ctx, states, obs, theta, m, n_cols, col_offset, seed, sweep_id, win=win)
    ref = states.copy()
    res = oracle.sweep(net.parents, net.card, theta, color, ref, obs, m, n_cols, col_offset, seed,
                       sweep_id, want_flags=True, win=win)
    # production kernels first, then the debug build and its conditionals
    st = H.compare_states(gpu, ref, res["flags"], color, n_cols, obs=obs)
    if win is not None:
        H.compare_states(dbg, ref, res["flags"], color, n_cols, obs=obs)
        H.compare_probs(gp, res["probs"], obs, net.card, win,
                        H.diverged_chains(dbg, ref, n_cols, win))
    return gpu, ref, st


@pytest.mark.parametrize("n_cols,ld", [(1, 4), (3, 4), (1021, 1024), (1025, 2048), (4097, 4100)])
def test_ragged_tails(n_cols, ld):
    net, st, ob, th = _custom([[], [0], [0, 1], [2]], [3, 2, 4, 2], n_cols, 3, 0.5, n_cols, ld=ld)
    # padding holds out-of-range states and "latent" obs: it must be neither read
    # into a table index, drawn, nor counted
    st[:, :, n_cols:] = 120
    ob[:, n_cols:] = 0
    _custom_case(net, st, ob, th, 3, n_cols, win=(0, min(n_cols, 64)))
    ctx = H.context_for(net)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, torch.from_numpy(same.pack_states(st)).cuda(), 3, n_cols, ld, mb, None, ctx.new_workspace())
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), oracle.counts(net.parents, net.card, st, 3, n_cols))


@pytest.mark.parametrize("bits", [0, 4, 16])
@pytest.mark.parametrize("lds", [None, 0, 256], ids=["staged", "global", "small-budget"])
def test_many_group_nodes(bits, lds):
    """Product nodes with four or more CPT groups walk their flat entry list
    (entries loaded across group boundaries): the roots 0 and 1 (empty own
    group, 7 groups each; K = 2 loads eight entries per batch, K = 5 four) and
    node 2 (a parent and 5 child groups).  Records staged in LDS, read from
    global memory, and a budget that stages only part of some records (those
    nodes keep the group walk).  bits = 16: an isolated 130-state node makes
    every state a 16-bit one."""
    parents = [[], [], [0], [0, 1], [0, 2], [0, 1, 2], [0, 2], [1, 2], [0, 1], [1], [2, 1]]
    card = [2, 5, 3, 2, 2, 2, 3, 2, 2, 2, 2]
    if bits == 16:
        parents, card, bits = parents + [[]], card + [130], 0
    net, st, ob, th = _custom(parents, card, 1000, 6, 0.5, 11)
    kw = dict(state_bits=bits) if bits else {}
    if lds is not None:
        kw["lds_limit"] = lds
    _custom_case(net, st, ob, th, 6, 1000, win=(0, 64), table_limit=0, **kw)


def test_zero_columns_is_noop():
    net, st, ob, th = _custom([[], [0]], [2, 2], 8, 2, 0.5, 1, ld=8)
    ctx = H.context_for(net)
    gpu, _ = H.gpu_sweep(ctx, st, ob, th, 2, 0, 0, 1, 0)
    assert np.array_equal(gpu, st)


def test_all_observed_and_all_latent():
    net, st, ob, th = _custom([[], [0], [1]], [2, 3, 2], 512, 2, 0.0, 2)
    gpu, _ = H.gpu_sweep(H.context_for(net), st, ob, th, 2, 512, 0, 1, 0)
    assert np.array_equal(gpu, st)
    net, st, ob, th = _custom([[], [0], [1]], [2, 3, 2], 512, 2, 1.0, 3)
    _custom_case(net, st, ob, th, 2, 512, win=(0, 512))


KERNEL_VARIANTS = [dict(), dict(lds_limit=0), dict(lds_limit=256), dict(packed=False)]
KERNEL_VARIANT_IDS = ["default", "global-tables", "partial-records", "wide-indices"]


@pytest.mark.parametrize("variant", KERNEL_VARIANTS, ids=KERNEL_VARIANT_IDS)
@pytest.mark.parametrize("table_limit", [None, 0], ids=["tables", "products"])
@pytest.mark.parametrize("K", [2, 3, 5, 6, 7, 8, 9, 16, 17, 40])
def test_cardinality_classes(K, table_limit, variant):
    # threshold tables for K <= 9, products with KP = 2/4/6/8/16, generic for K > 16
    parents = [[], [0], [0, 1], [1], [2, 3]]
    card = [K, 3, K, 2, 4]
    net, st, ob, th = _custom(parents, card, 700, 3, 0.6, K)
    _custom_case(net, st, ob, th, 3, 700, win=(0, 128), table_limit=table_limit, **variant)


@pytest.mark.parametrize("variant", KERNEL_VARIANTS, ids=KERNEL_VARIANT_IDS)
@pytest.mark.parametrize("table_limit", [None, 0], ids=["tables", "products"])
def test_int16_states(table_limit, variant):
    parents = [[], [0], [0, 1], [2], [1]]
    card = [130, 3, 200, 2, 5]
    net, st, ob, th = _custom(parents, card, 300, 2, 0.5, 17)
    assert st.dtype == np.int16
    _custom_case(net, st, ob, th, 2, 300, win=(0, 64), table_limit=table_limit, **variant)


def test_large_replica_count_and_column_offset():
    net, st, ob, th = _custom([[], [0], [0, 1], [2], [3, 1]], [2, 3, 2, 4, 2], 256, 37, 0.5, 4)
    _custom_case(net, st, ob, th, 37, 256, col_offset=(1 << 32) - 8192, win=(0, 32))


def test_underflow_rescale_path():
    # a binary root with 8 observed children whose CPTs alternately favour
    # each root state by a factor 1e20: every product term is tiny, so the
    # fp32 product must be renormalised to stay out of underflow
    parents = [[]] + [[0]] * 8
    card = [2] * 9
    theta = [0.5, 0.5]
    for c in range(8):
        tiny, big = 1e-20, 1.0 - 1e-20
        if c % 2 == 0:   # P(child=1 | root=0) tiny, P(child=1 | root=1) big
            theta += [big, tiny, tiny, big]
        else:
            theta += [tiny, big, big, tiny]
    theta = np.array(theta, dtype=np.float32)
    n_cols, m = 256, 2
    net, st, ob, _ = _custom(parents, card, n_cols, m, 0.0, 8, theta=theta)
    ob[0, :n_cols] = 0
    ob[1:, :n_cols] = 1
    st[1:, :, :n_cols] = 1
    # products from staged, global and partly staged records (budget 0 or 64 bytes)
    for tl, lds in ((None, None), (0, None), (0, 0), (0, 64)):
        gpu, ref, _ = _custom_case(net, st, ob, theta, m, n_cols, win=(0, 64), table_limit=tl, lds_limit=lds)
        # the conditional of the root is exactly (1/2, 1/2); both states must appear
        assert 0 < gpu[0, :, :n_cols].mean() < 1


def test_zero_cpt_entries_clamped():
    parents = [[], [0], [1]]
    card = [2, 3, 2]
    rng = np.random.default_rng(2)
    theta = brute.random_theta(rng, parents, card).astype(np.float32)
    theta[[1, 4, 9]] = 0.0
    net, st, ob, _ = _custom(parents, card, 512, 2, 0.5, 6, theta=theta)
    _custom_case(net, st, ob, theta, 2, 512, win=(0, 512))


# ------------------------------------------------------------ counts

@pytest.mark.parametrize("cfg,kw", [(1, {}), (3, dict(n_cols=7_001)), (4, {}),
                                    (5, dict(n_cols=3_000))])
def test_counts_bit_exact_and_moving_sum(cfg, kw):
    w = make_workload(cfg, **kw)
    net = w.net
    ctx = H.context_for(net)
    st = w.states[0]
    ncols = w.mb_cols(0)
    want = oracle.counts(net.parents, net.card, st.numpy(), w.m, ncols)
    rng = np.random.default_rng(cfg)
    prev = rng.integers(0, 1000, ctx.cpt_total).astype(np.int32)
    tot0 = prev.astype(np.int64) + rng.integers(0, 1000, ctx.cpt_total)
    mb = torch.from_numpy(prev.copy()).cuda()
    tot = torch.from_numpy(tot0.astype(np.int32)).cuda()
    ws = ctx.new_workspace()
    same.same_counts(ctx, same.pack_states(st).cuda(), w.m, ncols, w.ld, mb, tot, ws)
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), want)
    assert np.array_equal(tot.cpu().numpy(), tot0 - prev + want)
    off = ctx.cpt_off
    for i in range(net.n):
        assert want[off[i]:off[i + 1]].sum() == ncols * w.m
    # nullable totals; counting twice gives the same counts
    same.same_counts(ctx, same.pack_states(st).cuda(), w.m, ncols, w.ld, mb, None, ws)
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), want)


@pytest.mark.parametrize("n_par,K", [(4, 3), (4, 4), (4, 9), (5, 3)],
                         ids=["12288-bins-2-ranges", "16384-bins-2-ranges", "36864-bins-global",
                              "98304-bins-32bit-global"])
def test_counts_large_cpt(n_par, K):
    # one node whose CPT exceeds the count kernel's 8192-bin LDS histogram:
    # counted in LDS ranges up to 32768 bins, with global atomics beyond
    parents = [[] for _ in range(n_par)] + [list(range(n_par))]
    card = [8] * n_par + [K]
    net, st, _, _ = _custom(parents, card, 5000, 3, 0.0, 12)
    ctx = H.context_for(net)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, torch.from_numpy(same.pack_states(st)).cuda(), 3, 5000, st.shape[-1], mb, None,
                     ctx.new_workspace())
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), oracle.counts(parents, card, st, 3, 5000))


@pytest.mark.parametrize("n_cols,ld", [(3, 4), (4097, 4100), (2049, 2052), (6000, 6004)])
@pytest.mark.parametrize("big", [False, True], ids=["int8", "int16"])
def test_counts_ragged_rows(n_cols, ld, big):
    # rows whose length ld is not a multiple of 8 columns: the last column pair
    # of a row is read as one quad; padding holds out-of-range states
    card = [130 if big else 3, 3, 200 if big else 4, 2, 5]
    parents = [[], [0], [0, 1], [2], [1, 2, 3]]
    net, st, _, _ = _custom(parents, card, n_cols, 3, 0.0, 21, ld=ld)
    st[:, :, n_cols:] = 120
    ctx = H.context_for(net)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, torch.from_numpy(same.pack_states(st)).cuda(), 3, n_cols, ld, mb, None, ctx.new_workspace())
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), oracle.counts(parents, card, st, 3, n_cols))


# ------------------------------------------------------------ Dirichlet

@pytest.mark.parametrize("cfg,alpha", [(1, 1.0), (3, 1.0), (5, 1.0), (4, 0.3)])
def test_dirichlet_matches_oracle(cfg, alpha):
    w = make_workload(cfg, n_cols=8)
    net = w.net
    pptr, pidx, card = net.csr()
    ctx = same.same_create(pptr, pidx, card, alpha)
    rng = np.random.default_rng(cfg)
    totals = rng.integers(0, 5000, ctx.cpt_total).astype(np.int32)
    totals[rng.random(ctx.cpt_total) < 0.3] = 0
    out = torch.empty(ctx.cpt_total, dtype=torch.float32, device="cuda")
    same.same_sample_cpts(ctx, torch.from_numpy(totals).cuda(), out, 1234567, 42,
                          ctx.new_workspace())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    want = oracle.dirichlet(net.parents, net.card, totals, alpha, 1234567, 42)
    exact = np.mean(got == want)
    rel = np.max(np.abs(got.astype(np.float64) - want) / np.maximum(want, 1e-30))
    print("dirichlet exact fraction", exact, "max rel", rel)
    assert exact >= 1.0 - 1e-5
    assert rel <= 1e-6


# ------------------------------------------------------------ whole loop, lockstep

@pytest.mark.parametrize("cfg,kw,sweeps", [(1, {}, 20), (2, dict(n_cols=6_000, nb=2_000), 3),
                                           (4, dict(n_cols=1_000), 4)])
def test_lockstep_loop(cfg, kw, sweeps):
    """The oracle runs the loop; at every (pass, minibatch) step the library is
    fed the oracle's inputs for that step and must reproduce its outputs."""
    w = make_workload(cfg, **kw)
    net = w.net
    ctx = H.context_for(net)
    color = oracle.graph(net.parents, net.card)["color"]
    ws = ctx.new_workspace()
    theta = w.init_theta.copy()
    states = [s.numpy().copy() for s in w.states]
    obs = [o.numpy() for o in w.obs]
    mb = [oracle.counts(net.parents, net.card, states[b], w.m, w.mb_cols(b)) for b in range(w.M)]
    totals = np.sum(mb, axis=0)
    for s in range(sweeps):
        for b in range(w.M):
            nc = w.mb_cols(b)
            pre = states[b].copy()
            res = oracle.sweep(net.parents, net.card, theta, color, states[b], obs[b], w.m, nc,
                               b * w.nb, w.seed, s, want_flags=True)
            gpu, _ = H.gpu_sweep(ctx, pre, obs[b], theta, w.m, nc, b * w.nb, w.seed, s)
            H.compare_states(gpu, states[b], res["flags"], color, nc)
            new = oracle.counts(net.parents, net.card, states[b], w.m, nc)
            d_mb = torch.from_numpy(mb[b].astype(np.int32)).cuda()
            d_tot = torch.from_numpy(totals.astype(np.int32)).cuda()
            same.same_counts(ctx, torch.from_numpy(same.pack_states(states[b])).cuda(), w.m, nc, w.ld, d_mb, d_tot, ws)
            totals = oracle.moving_sum(totals, mb[b], new)
            mb[b] = new
            th_gpu = torch.empty(ctx.cpt_total, dtype=torch.float32, device="cuda")
            same.same_sample_cpts(ctx, d_tot, th_gpu, w.seed, s * w.M + b, ws)
            torch.cuda.synchronize()
            assert np.array_equal(d_mb.cpu().numpy(), new)
            assert np.array_equal(d_tot.cpu().numpy(), totals)
            theta = oracle.dirichlet(net.parents, net.card, totals, w.alpha, w.seed, s * w.M + b)
            assert np.mean(th_gpu.cpu().numpy() == theta) >= 1.0 - 1e-5


def test_independent_loops_agree_until_first_flagged_draw():
    """Library and oracle each run the whole student-2k loop on their own; the
    runs must be identical sweep by sweep until a flagged boundary draw (if
    any) makes them diverge."""
    w = make_workload(1)
    net = w.net
    ctx = H.context_for(net)
    color = oracle.graph(net.parents, net.card)["color"]
    ws = ctx.new_workspace()
    d_st = same.pack_states(w.states[0]).cuda()
    d_ob = w.obs[0].cuda()
    d_th = torch.from_numpy(w.init_theta).cuda()
    d_mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    d_tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, d_st, w.m, w.n_cols, w.ld, d_mb, d_tot, ws)
    st = w.states[0].numpy().copy()
    ob = w.obs[0].numpy()
    theta = w.init_theta.copy()
    mb = oracle.counts(net.parents, net.card, st, w.m, w.n_cols)
    tot = mb.copy()
    for s in range(w.sweeps):
        same.same_sweep(ctx, d_st, d_ob, d_th, w.m, w.n_cols, w.ld, 0, w.seed, s, ws)
        same.same_counts(ctx, d_st, w.m, w.n_cols, w.ld, d_mb, d_tot, ws)
        same.same_sample_cpts(ctx, d_tot, d_th, w.seed, s, ws)
        res = oracle.sweep(net.parents, net.card, theta, color, st, ob, w.m, w.n_cols, 0, w.seed,
                           s, want_flags=True)
        new = oracle.counts(net.parents, net.card, st, w.m, w.n_cols)
        tot = tot - mb + new
        mb = new
        theta = oracle.dirichlet(net.parents, net.card, tot, w.alpha, w.seed, s)
        torch.cuda.synchronize()
        g_st = same.unpack_states(d_st.cpu().numpy(), w.m)
        if not np.array_equal(g_st, st):
            H.compare_states(g_st, st, res["flags"], color, w.n_cols)
            print("diverged at sweep", s, "on a flagged draw")
            return
        assert np.array_equal(d_tot.cpu().numpy(), tot)
        g_th = d_th.cpu().numpy()
        if not np.array_equal(g_th, theta):
            assert np.mean(g_th == theta) >= 1.0 - 1e-5
            print("CPTs differ in the last bit at sweep", s)
            return
    print("identical over all", w.sweeps, "sweeps")


def test_kernel_timing_counts_launches_and_phases():
    """With timing on, every launch of a sweep is counted in its class and every
    colour group in one phase; the phase time covers the group's launches."""
    w = make_workload(5, n_cols=3_000, m=2)
    net = w.net
    ctx = H.context_for(net, lds_limit=1024)
    lay = same.same_layout(ctx)
    same.same_kernel_timing(ctx, True)
    H.gpu_sweep(ctx, w.states[0].numpy(), w.obs[0].numpy(), w.init_theta, w.m, 3_000, 0, w.seed, 3)
    kt = same.same_kernel_times(ctx)
    same.same_kernel_timing(ctx, False)
    assert sum(kt["launches"]) == lay["sweep_launches"]
    assert kt["launches"][0] > 0 and kt["launches"][1] > 0
    assert kt["phases"] == lay["n_colors"]
    assert kt["phase_ms"] > 0.0
    # every (node, column, replica) slot is covered by exactly one launch
    assert sum(kt["node_samples"]) == float(net.n * 3_000 * w.m)
    assert same.same_kernel_times(ctx) == {"ms": [0.0] * 4, "launches": [0] * 4, "phase_ms": 0.0, "phases": 0,
                                           "node_samples": [0.0] * 4}


@pytest.mark.parametrize("big", [False, True], ids=["int8", "int16"])
def test_tiled_step_counts_with_unaligned_rows(big):
    """same_step over 1024-column tiles with rows of ld = 5004 (not a multiple
    of 16): the count pass of the last tile reads its rows' ragged ends one
    quad at a time, and the tiled step equals the untiled one bit for bit
    (states, counts, moving sum, CPTs); the counts equal the oracle's."""
    card = [130 if big else 3, 3, 200 if big else 4, 2, 5]
    parents = [[], [0], [0, 1], [2], [1, 2, 3]]
    n_cols, ld, m = 5001, 5004, 3
    net, st, ob, th = _custom(parents, card, n_cols, m, 0.5, 23, ld=ld)
    outs = []
    for tb in (1, 0):
        ctx = H.context_for(net, tile_bytes=tb)
        d_st = torch.from_numpy(same.pack_states(st)).cuda()
        d_ob = torch.from_numpy(ob).cuda()
        d_th = torch.from_numpy(th.astype(np.float32)).cuda()
        mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        ws = ctx.new_workspace()
        same.same_step(ctx, d_st, d_ob, d_th, m, n_cols, ld, 0, 5, 0, mb, tot, 0, ws)
        torch.cuda.synchronize()
        outs.append([x.cpu().numpy() for x in (d_st, mb, tot, d_th)])
    for x, y in zip(*outs):
        assert np.array_equal(x, y)
    assert np.array_equal(outs[0][1], oracle.counts(parents, card, same.unpack_states(outs[0][0], m), m, n_cols))


@pytest.mark.parametrize("big", [False, True], ids=["int8", "int16"])
def test_padding_slots_may_hold_anything(big):
    """The padding slots of the last replica quad (m = 5: slots 5..7) may hold
    any value, out of range included: the sweep reads them as state 0 and the
    counts skip them, so a step (pre-pass counts, sweep, counts, resample)
    gives the same real replicas, counts and CPTs whatever they hold."""
    card = [130 if big else 3, 3, 200 if big else 4, 2, 5]
    parents = [[], [0], [0, 1], [2], [1, 2, 3]]
    n_cols, ld, m = 3001, 3004, 5
    net, st, ob, th = _custom(parents, card, n_cols, m, 0.5, 31, ld=ld)
    outs = []
    for fill in (0, 30000 if big else 120):
        q = same.pack_states(st)
        q[:, -1, :, m % 4:] = fill
        ctx = H.context_for(net)
        d_st = torch.from_numpy(q).cuda()
        d_ob = torch.from_numpy(ob).cuda()
        d_th = torch.from_numpy(th.astype(np.float32)).cuda()
        mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        ws = ctx.new_workspace()
        same.same_counts(ctx, d_st, m, n_cols, ld, mb, tot, ws)
        for s in range(2):
            same.same_step(ctx, d_st, d_ob, d_th, m, n_cols, ld, 0, 5, s, mb, tot, s, ws)
        torch.cuda.synchronize()
        outs.append([same.unpack_states(d_st.cpu().numpy(), m), mb.cpu().numpy(), tot.cpu().numpy(),
                     d_th.cpu().numpy()])
    for x, y in zip(*outs):
        assert np.array_equal(x, y)
    assert np.array_equal(outs[1][1], oracle.counts(parents, card, outs[1][0], m, n_cols))


# ------------------------------------------------------------ 4-bit states

@pytest.mark.parametrize("cfg,kw,win", [
    (1, {}, (0, 2000)),
    (2, dict(n_cols=20_000), (1000, 3000)),
    (3, dict(n_cols=9_000), (8_000, 1000)),
    (4, {}, (0, 600)),
    (5, dict(n_cols=3_000, m=5), (0, 300)),             # odd m: a replica quad, then a partial one
    (5, dict(n_cols=2_001, m=7), (1_700, 301)),         # odd m and a ragged tail
])
def test_sweep_parity_4bit(cfg, kw, win):
    """4-bit states (a replica quad in one 16-bit word): the production and
    debug sweeps against the oracle, as for 8-bit states."""
    w = make_workload(cfg, **kw)
    out = _sweep_case(w, win=win, state_bits=4)
    assert out["states"]["draws"] > 0


@pytest.mark.parametrize("cfg,kw", [(1, {}), (3, dict(n_cols=7_001)), (4, {}), (5, dict(n_cols=3_000))])
def test_counts_4bit(cfg, kw):
    w = make_workload(cfg, **kw)
    net = w.net
    ctx = H.context_for(net, state_bits=4)
    ncols = w.mb_cols(0)
    want = oracle.counts(net.parents, net.card, w.states[0].numpy(), w.m, ncols)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, H.to_device(ctx, w.states[0]), w.m, ncols, w.ld, mb, tot, ctx.new_workspace())
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), want)
    assert np.array_equal(tot.cpu().numpy(), want)


@pytest.mark.parametrize("n_par,K", [(4, 3), (5, 3)], ids=["12288-bins-2-ranges", "98304-bins-32bit-global"])
def test_counts_large_cpt_4bit(n_par, K):
    parents = [[] for _ in range(n_par)] + [list(range(n_par))]
    card = [8] * n_par + [K]
    net, st, _, _ = _custom(parents, card, 5000, 3, 0.0, 12)
    ctx = H.context_for(net, state_bits=4)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, H.to_device(ctx, st), 3, 5000, st.shape[-1], mb, None, ctx.new_workspace())
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), oracle.counts(parents, card, st, 3, 5000))


@pytest.mark.parametrize("n_cols,ld", [(3, 4), (4097, 4100), (6000, 6004)])
def test_counts_ragged_rows_4bit(n_cols, ld):
    card = [16, 3, 4, 2, 5]
    parents = [[], [0], [0, 1], [2], [1, 2, 3]]
    net, st, _, _ = _custom(parents, card, n_cols, 3, 0.0, 21, ld=ld)
    st[:, :, n_cols:] = 15
    ctx = H.context_for(net, state_bits=4)
    mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
    same.same_counts(ctx, H.to_device(ctx, st), 3, n_cols, ld, mb, None, ctx.new_workspace())
    torch.cuda.synchronize()
    assert np.array_equal(mb.cpu().numpy(), oracle.counts(parents, card, st, 3, n_cols))


def test_step_tiles_and_8bit_agree_4bit():
    """With 4-bit states a tiled step equals an untiled one and equals the
    same step on 8-bit states (the format does not change any result):
    states, counts, moving sum and CPTs, bit for bit."""
    w = make_workload(5, n_cols=5_000, m=3)
    net = w.net
    outs = []
    for kw in (dict(state_bits=4, tile_bytes=1), dict(state_bits=4), {}):
        ctx = H.context_for(net, **kw)
        st = H.to_device(ctx, w.states[0])
        ob = w.obs[0].cuda()
        th = torch.from_numpy(w.init_theta).cuda()
        mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        ws = ctx.new_workspace()
        same.same_counts(ctx, st, w.m, 5_000, w.ld, mb, tot, ws)
        for s in range(2):
            same.same_step(ctx, st, ob, th, w.m, 5_000, w.ld, 0, w.seed, s, mb, tot, s, ws)
        torch.cuda.synchronize()
        outs.append([H.from_device(ctx, st, w.m), mb.cpu().numpy(), tot.cpu().numpy(), th.cpu().numpy()])
    for o in outs[1:]:
        for x, y in zip(outs[0], o):
            assert np.array_equal(x, y)


def test_lockstep_loop_4bit():
    w = make_workload(4, n_cols=1_000)
    net = w.net
    ctx = H.context_for(net, state_bits=4)
    color = oracle.graph(net.parents, net.card)["color"]
    ws = ctx.new_workspace()
    theta = w.init_theta.copy()
    st = w.states[0].numpy().copy()
    obs = w.obs[0].numpy()
    mb = oracle.counts(net.parents, net.card, st, w.m, w.n_cols)
    totals = mb.copy()
    for s in range(4):
        pre = st.copy()
        res = oracle.sweep(net.parents, net.card, theta, color, st, obs, w.m, w.n_cols, 0, w.seed, s,
                           want_flags=True)
        gpu, _ = H.gpu_sweep(ctx, pre, obs, theta, w.m, w.n_cols, 0, w.seed, s)
        H.compare_states(gpu, st, res["flags"], color, w.n_cols)
        new = oracle.counts(net.parents, net.card, st, w.m, w.n_cols)
        d_mb = torch.from_numpy(mb.astype(np.int32)).cuda()
        d_tot = torch.from_numpy(totals.astype(np.int32)).cuda()
        same.same_counts(ctx, H.to_device(ctx, st), w.m, w.n_cols, w.ld, d_mb, d_tot, ws)
        totals = oracle.moving_sum(totals, mb, new)
        mb = new
        th_gpu = torch.empty(ctx.cpt_total, dtype=torch.float32, device="cuda")
        same.same_sample_cpts(ctx, d_tot, th_gpu, w.seed, s, ws)
        torch.cuda.synchronize()
        assert np.array_equal(d_mb.cpu().numpy(), new)
        assert np.array_equal(d_tot.cpu().numpy(), totals)
        theta = oracle.dirichlet(net.parents, net.card, totals, w.alpha, w.seed, s)
        assert np.mean(th_gpu.cpu().numpy() == theta) >= 1.0 - 1e-5


def test_padding_slots_may_hold_anything_4bit():
    card = [3, 3, 4, 2, 5]
    parents = [[], [0], [0, 1], [2], [1, 2, 3]]
    n_cols, ld, m = 3001, 3004, 5
    net, st, ob, th = _custom(parents, card, n_cols, m, 0.5, 31, ld=ld)
    outs = []
    for fill in (False, True):
        q = same.pack_states(st, 4)
        if fill:  # slots 1..3 of the last quad (replicas 5..7) hold 15, out of range for every node
            q[:, -1, :] = (q[:, -1, :].view(np.uint16) | np.uint16(0xFFF0)).view(np.int16)
        ctx = H.context_for(net, state_bits=4)
        d_st = torch.from_numpy(q).cuda()
        d_ob = torch.from_numpy(ob).cuda()
        d_th = torch.from_numpy(th.astype(np.float32)).cuda()
        mb = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        tot = torch.zeros(ctx.cpt_total, dtype=torch.int32, device="cuda")
        ws = ctx.new_workspace()
        same.same_counts(ctx, d_st, m, n_cols, ld, mb, tot, ws)
        for s in range(2):
            same.same_step(ctx, d_st, d_ob, d_th, m, n_cols, ld, 0, 5, s, mb, tot, s, ws)
        torch.cuda.synchronize()
        outs.append([H.from_device(ctx, d_st, m), mb.cpu().numpy(), tot.cpu().numpy(), d_th.cpu().numpy()])
    for x, y in zip(*outs):
        assert np.array_equal(x, y)
    assert np.array_equal(outs[1][1], oracle.counts(parents, card, outs[1][0], m, n_cols))
