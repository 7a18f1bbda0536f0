"""Host-side checks of libsame (no GPU needed): the library loads and exports
every entry point include/same.h declares; the host graph compiler's layout
and colouring agree with the oracle's independent graph code; invalid graphs
and invalid arguments return their error codes before any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

import oracle
import paper_1511_06416_amd as same
from tests import brute
from workloads import CONFIGS, koller, make_network

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_symbols():
    names = set()
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            txt = open(os.path.join(ROOT, "include", fn)).read()
            txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
            names |= set(re.findall(r"\b(same_[a-z_0-9]+)\s*\(", txt))
    return names


def test_library_exports_every_declared_symbol():
    L = same.load_library()
    names = _declared_symbols()
    assert {"same_create", "same_sweep", "same_counts", "same_sample_cpts"} <= names
    for name in sorted(names):
        assert hasattr(L, name), name


def _ctx(net, prior=1.0):
    pptr, pidx, card = net.csr()
    return same.same_create(pptr, pidx, card, prior)


@pytest.mark.parametrize("cfg", sorted(CONFIGS))
def test_layout_and_colouring_match_oracle(cfg):
    net = make_network(cfg)
    ctx = _ctx(net)
    ref = oracle.graph(net.parents, net.card)
    assert np.array_equal(ctx.cpt_off, ref["cpt_off"])
    assert np.array_equal(ctx.color, ref["color"])
    assert ctx.n_colors == ref["n_colors"]
    assert ctx.cpt_total == ref["cpt_off"][-1]
    assert ctx.state_bytes == 1
    assert ctx.workspace_bytes > 4 * ctx.cpt_total
    ctx.close()


@pytest.mark.parametrize("cfg", sorted(CONFIGS))
def test_first_fit_colouring_option_matches_oracle(cfg):
    # the option that skips the balancing moves gives the oracle's first-fit
    # colouring; the default gives its balanced one
    net = make_network(cfg)
    pptr, pidx, card = net.csr()
    ff = same.same_create_ex(pptr, pidx, card, 1.0, first_fit_colours=True)
    assert np.array_equal(ff.color, oracle.graph(net.parents, net.card, balance=False)["color"])
    assert np.array_equal(_ctx(net).color, oracle.graph(net.parents, net.card)["color"])
    ff.close()


@pytest.mark.parametrize("seed", range(5))
def test_random_graphs_balanced_colours_match_oracle(seed):
    rng = np.random.default_rng(1000 + seed)
    parents, card = brute.random_net(rng, 200, 4, 2, 6)
    pptr = np.cumsum([0] + [len(p) for p in parents]).astype(np.int32)
    pidx = np.array([p for ps in parents for p in ps], dtype=np.int32)
    for ffc in (False, True):
        ctx = same.same_create_ex(pptr, pidx, card, 1.0, first_fit_colours=ffc)
        assert np.array_equal(ctx.color, oracle.graph(parents, card, balance=not ffc)["color"])
        ctx.close()


def test_student_layout():
    ctx = _ctx(koller())
    assert ctx.cpt_total == 26 and ctx.n_rows == 11 and ctx.n_colors == 3
    assert ctx.max_card == 3


@pytest.mark.parametrize("seed", range(5))
def test_random_graphs_match_oracle(seed):
    rng = np.random.default_rng(seed)
    parents, card = brute.random_net(rng, 60, 5, 2, 9)
    pptr = np.cumsum([0] + [len(p) for p in parents]).astype(np.int32)
    pidx = np.array([p for ps in parents for p in ps], dtype=np.int32)
    ctx = same.same_create(pptr, pidx, card)
    ref = oracle.graph(parents, card)
    assert np.array_equal(ctx.color, ref["color"])
    assert np.array_equal(ctx.cpt_off, ref["cpt_off"])


def test_int16_states_for_large_cardinality():
    ctx = same.same_create([0, 0, 1], [0], [200, 3])
    assert ctx.state_bytes == 2 and ctx.max_card == 200


@pytest.mark.parametrize("pptr,pidx,card,code", [
    ([0, 1], [0], [2], same.SAME_EGRAPH),               # self loop
    ([0, 0, 2], [0, 0], [2, 2], same.SAME_EGRAPH),      # duplicate parent
    ([0, 1], [5], [2], same.SAME_EGRAPH),               # parent out of range
    ([0, 1, 2], [1, 0], [2, 2], same.SAME_EGRAPH),      # cycle
    ([0, 2, 3, 4], [1, 2, 2, 0], [2, 2, 2], same.SAME_EGRAPH),  # 3-cycle
    ([0, 0], [], [1], same.SAME_ECARD),
    ([0, 0], [], [40000], same.SAME_ECARD),
    ([1, 1], [0], [2], same.SAME_EGRAPH),               # parent_ptr[0] != 0
])
def test_invalid_graphs(pptr, pidx, card, code):
    with pytest.raises(same.SameError) as ei:
        same.same_create(pptr, pidx, card)
    assert ei.value.code == code
    assert same.same_last_error() != ""


def test_row_overflow_is_esize():
    # 12 parents of cardinality 8 -> 8^12 rows
    n = 13
    pptr = np.array([0] * 13 + [12], dtype=np.int32)
    pidx = np.arange(12, dtype=np.int32)
    card = np.full(n, 8, dtype=np.int32)
    with pytest.raises(same.SameError) as ei:
        same.same_create(pptr, pidx, card)
    assert ei.value.code == same.SAME_ESIZE


def test_bad_prior():
    with pytest.raises(same.SameError) as ei:
        same.same_create([0, 0], [], [2], 0.0)
    assert ei.value.code == same.SAME_EINVAL


# Argument validation happens before any HIP call, so these run without a GPU.
# The fake addresses are never dereferenced.
FAKE = 1 << 20


@pytest.mark.parametrize("kw,code", [
    (dict(m=0), same.SAME_EINVAL),
    (dict(n_cols=100, ld=96), same.SAME_EINVAL),
    (dict(ld=98, n_cols=90), same.SAME_EALIGN),
    (dict(col_offset=2), same.SAME_EALIGN),
    (dict(col_offset=-4), same.SAME_EALIGN),
    (dict(states=0), same.SAME_EINVAL),
    (dict(obs=0), same.SAME_EINVAL),
    (dict(workspace=FAKE + 8), same.SAME_EALIGN),
    (dict(obs=FAKE + 1), same.SAME_EALIGN),
    (dict(states=FAKE + 2), same.SAME_EALIGN),
])
def test_sweep_argument_errors(kw, code):
    ctx = _ctx(koller())
    L = same.load_library()
    a = dict(states=FAKE, obs=FAKE, cpts=FAKE, m=2, n_cols=64, ld=64, col_offset=0, workspace=FAKE)
    a.update(kw)
    rc = L.same_sweep(ctx.handle, C.c_void_p(a["states"]), C.c_void_p(a["obs"]),
                      C.c_void_p(a["cpts"]), a["m"], a["n_cols"], a["ld"], a["col_offset"], 1, 0,
                      C.c_void_p(a["workspace"]), None)
    assert rc == code


def test_counts_and_sample_argument_errors():
    ctx = _ctx(koller())
    L = same.load_library()
    assert L.same_counts(ctx.handle, C.c_void_p(FAKE), 0, 4, 4, C.c_void_p(FAKE), None,
                         C.c_void_p(FAKE), None) == same.SAME_EINVAL
    assert L.same_counts(ctx.handle, C.c_void_p(FAKE), 1, 4, 4, None, None,
                         C.c_void_p(FAKE), None) == same.SAME_EINVAL
    assert L.same_sample_cpts(ctx.handle, None, C.c_void_p(FAKE), 1, 0, C.c_void_p(FAKE),
                              None) == same.SAME_EINVAL
    assert L.same_sample_cpts(ctx.handle, C.c_void_p(FAKE), C.c_void_p(FAKE), 1, 0,
                              C.c_void_p(FAKE + 16), None) == same.SAME_EALIGN
    assert L.same_sweep_debug(ctx.handle, C.c_void_p(FAKE), C.c_void_p(FAKE), C.c_void_p(FAKE),
                              1, 8, 8, 0, 1, 0, 0, 0, None, C.c_void_p(FAKE),
                              None) == same.SAME_EINVAL


def test_null_context():
    L = same.load_library()
    assert L.same_layout(None, None, None, None) == same.SAME_EINVAL
    assert L.same_workspace_size(None, None) == same.SAME_EINVAL
    L.same_destroy(None)


def test_stream_argument_errors():
    ctx = _ctx(koller())
    L = same.load_library()
    P = C.c_void_p
    good = dict(hs=FAKE, ho=FAKE, host_ld=1000, n_cols=1000, nb=256, m=2, flags=0, slots=FAKE)

    def call(**kw):
        a = dict(good)
        a.update(kw)
        return L.same_stream_pass(ctx.handle, P(a["hs"]), P(a["ho"]), a["host_ld"], a["n_cols"],
                                  a["nb"], a["m"], P(FAKE), P(FAKE), P(FAKE), 1, 0, a["flags"],
                                  P(a["slots"]), P(FAKE), None)

    assert call(nb=250) == same.SAME_EALIGN
    assert call(nb=0) == same.SAME_EALIGN
    assert call(host_ld=999) == same.SAME_EINVAL
    assert call(m=0) == same.SAME_EINVAL
    assert call(hs=0) == same.SAME_EINVAL
    assert call(flags=4) == same.SAME_EINVAL
    assert call(slots=FAKE + 64) == same.SAME_EALIGN
    assert call(n_cols=0) == same.SAME_OK
    size = C.c_size_t()
    assert L.same_stream_slots_size(ctx.handle, 2, 256, C.byref(size)) == same.SAME_OK
    # two slots of 5 nodes x 2 replicas x 256 columns plus 5 x 256 obs bytes
    assert size.value >= 2 * (5 * 2 * 256 + 5 * 256)


@pytest.mark.parametrize("field,value", [("lds_limit", -2), ("lds_limit", 40000),
                                         ("packed_indices", 2), ("tile_bytes", -1),
                                         ("table_limit", -5)])
def test_bad_options(field, value):
    net = koller()
    pptr, pidx, card = net.csr()
    L = same.load_library()
    opts = same._Options(-1, 0, -1, 1)
    setattr(opts, field, value)
    h = C.c_void_p()
    pptr = np.ascontiguousarray(pptr, dtype=np.int32)
    pidx = np.ascontiguousarray(pidx, dtype=np.int32)
    card = np.ascontiguousarray(card, dtype=np.int32)
    rc = L.same_create_ex(len(card), pptr.ctypes.data, pidx.ctypes.data, card.ctypes.data, 1.0,
                          C.byref(opts), C.byref(h))
    assert rc == same.SAME_EINVAL


@pytest.mark.parametrize("cfg", [3, 5])
@pytest.mark.parametrize("kw", [dict(lds_limit=0), dict(lds_limit=1024), dict(lds_limit=32768),
                                dict(packed_indices=False), dict(lds_limit=0, packed_indices=False)])
def test_kernel_class_options_keep_layout(cfg, kw):
    # the LDS budget (whole or partly staged records) and the index width
    # change only how the sweep reads its tables: CPT layout, colouring and
    # workspace stay the same
    net = make_network(cfg)
    pptr, pidx, card = net.csr()
    a = same.same_create(pptr, pidx, card)
    b = same.same_create_ex(pptr, pidx, card, **kw)
    assert np.array_equal(a.cpt_off, b.cpt_off) and np.array_equal(a.color, b.color)
    assert a.workspace_bytes == b.workspace_bytes
    # a smaller budget or wider indices never merge launches (lds_limit=0
    # moves every node to one global-table class; a larger budget may merge)
    if kw.get("lds_limit", 1) not in (0, 32768):
        assert b.sweep_launches >= a.sweep_launches


def test_kernel_timing_host_calls():
    ctx = _ctx(koller())
    assert same.same_kernel_times(ctx) == {"ms": [0.0] * 4, "launches": [0] * 4, "phase_ms": 0.0, "phases": 0,
                                           "node_samples": [0.0] * 4}
    same.same_kernel_timing(ctx, True)
    same.same_kernel_timing(ctx, False)
    L = same.load_library()
    assert L.same_kernel_timing(None, 1) == same.SAME_EINVAL
    assert L.same_kernel_times(ctx.handle, None) == same.SAME_EINVAL


def test_ingest_argument_errors():
    # argument checks return before any device work (no GPU needed)
    L = same.load_library()
    ctx = _ctx(koller())
    h = ctx.handle
    P = C.c_void_p
    fake = P(1 << 20)  # never dereferenced: every call below fails its checks first
    rp = P(1 << 21)
    # null states / obs / row_ptr
    assert L.same_expand_observed(h, rp, fake, fake, 4, 2, 8, 8, None, fake, None) == same.SAME_EINVAL
    assert L.same_expand_observed(h, None, fake, fake, 4, 2, 8, 8, fake, fake, None) == same.SAME_EINVAL
    assert L.same_expand_observed(h, rp, None, fake, 4, 2, 8, 8, fake, fake, None) == same.SAME_EINVAL
    assert L.same_expand_observed(h, rp, fake, fake, -1, 2, 8, 8, fake, fake, None) == same.SAME_EINVAL
    # m, n_cols > ld, ld not a multiple of 4, misaligned obs
    assert L.same_expand_observed(h, rp, fake, fake, 4, 0, 8, 8, fake, fake, None) == same.SAME_EINVAL
    assert L.same_expand_observed(h, rp, fake, fake, 4, 2, 9, 8, fake, fake, None) == same.SAME_EINVAL
    assert L.same_expand_observed(h, rp, fake, fake, 4, 2, 6, 6, fake, fake, None) == same.SAME_EALIGN
    assert L.same_expand_observed(h, rp, fake, fake, 4, 2, 8, 8, fake, P((1 << 20) + 1), None) == \
        same.SAME_EALIGN
    assert L.same_init_latent(h, None, fake, 2, 8, 8, 0, 1, None) == same.SAME_EINVAL
    assert L.same_init_latent(h, fake, None, 2, 8, 8, 0, 1, None) == same.SAME_EINVAL
    assert L.same_init_latent(h, fake, fake, 2, 8, 8, 2, 1, None) == same.SAME_EALIGN
    assert L.same_init_latent(None, fake, fake, 2, 8, 8, 0, 1, None) == same.SAME_EINVAL
    ctx.close()


def test_grow_replicas_argument_errors():
    L = same.load_library()
    ctx = _ctx(koller())
    h = ctx.handle
    P = C.c_void_p
    a, b = P(1 << 20), P(1 << 30)
    assert L.same_grow_replicas(h, a, 3, b, 2, 8, None) == same.SAME_EINVAL          # m2 < m
    assert L.same_grow_replicas(h, None, 3, b, 4, 8, None) == same.SAME_EINVAL
    assert L.same_grow_replicas(h, a, 3, P((1 << 20) + 16), 4, 8, None) == same.SAME_EINVAL  # overlap
    assert L.same_grow_replicas(h, a, 3, b, 4, 6, None) == same.SAME_EALIGN          # ld % 4
    ctx.close()


def test_step_graph_argument_errors():
    """same_step_graph validates before any device call; launch and destroy
    reject or ignore a null graph."""
    ctx = _ctx(koller())
    L = same.load_library()
    P = C.c_void_p
    good = dict(st=FAKE, ob=FAKE, cp=FAKE, m=2, n_cols=1000, ld=1024, col_offset=0, mb=FAKE, tot=FAKE,
                ids=FAKE, stride=1, steps=1, ws=FAKE)

    def call(**kw):
        a = dict(good)
        a.update(kw)
        out = P()
        rc = L.same_step_graph(ctx.handle, P(a["st"]), P(a["ob"]), P(a["cp"]), a["m"], a["n_cols"], a["ld"],
                               a["col_offset"], 1, P(a["mb"]), P(a["tot"]), P(a["ids"]), a["stride"],
                               a["steps"], P(a["ws"]), C.byref(out))
        assert out.value is None
        return rc

    assert call(ids=None) == same.SAME_EINVAL
    assert call(mb=None) == same.SAME_EINVAL
    assert call(st=None) == same.SAME_EINVAL
    assert call(steps=0) == same.SAME_EINVAL
    assert call(steps=65) == same.SAME_EINVAL
    assert call(n_cols=0) == same.SAME_EINVAL
    assert call(ids=FAKE + 2) == same.SAME_EALIGN
    assert call(ld=1022) == same.SAME_EALIGN
    assert call(col_offset=(1 << 32) - 512) == same.SAME_ESIZE
    assert L.same_step_graph(ctx.handle, P(FAKE), P(FAKE), P(FAKE), 2, 1000, 1024, 0, 1, P(FAKE), P(FAKE),
                             P(FAKE), 1, 1, P(FAKE), None) == same.SAME_EINVAL
    assert L.same_graph_launch(None, None) == same.SAME_EINVAL
    L.same_graph_destroy(None)


@pytest.mark.parametrize("m", [1, 3, 4, 10, 37])
def test_state_quad_layout_helpers(m):
    """pack_states places replica r of node i at column j at element
    ((i * mq + r // 4) * ld + j) * 4 + r % 4 of the flat array (the layout
    include/same.h documents), padding slots 0; unpack_states inverts it, for
    numpy arrays and torch tensors alike."""
    import torch
    rng = np.random.default_rng(m)
    n, ld = 3, 12
    rows = rng.integers(0, 100, (n, m, ld)).astype(np.int8)
    q = same.pack_states(rows)
    mq = (m + 3) // 4
    assert q.shape == same.state_shape(n, m, ld) == (n, mq, ld, 4)
    flat = q.reshape(-1)
    for i in range(n):
        for r in range(m):
            for j in range(ld):
                assert flat[((i * mq + r // 4) * ld + j) * 4 + r % 4] == rows[i, r, j]
    pad = same.unpack_states(q, 4 * mq)[:, m:]
    assert (pad == 0).all()
    assert np.array_equal(same.unpack_states(q, m), rows)
    t = same.pack_states(torch.from_numpy(rows.astype(np.int16)))
    assert t.is_contiguous() and tuple(t.shape) == q.shape
    assert np.array_equal(t.numpy(), q.astype(np.int16))
    assert np.array_equal(same.unpack_states(t, m).numpy(), rows.astype(np.int16))


def test_binding_refuses_states_in_another_layout():
    """A states tensor that is not [n][ceil(m/4)][ld][4] is refused by the
    binding before any device call."""
    import torch
    ctx = _ctx(koller())
    with pytest.raises(same.SameError) as e:
        same.same_counts(ctx, torch.zeros((ctx.n_nodes, 2, 8), dtype=torch.int8), 2, 8, 8, None, None, None)
    assert e.value.code == same.SAME_EINVAL and "replica quads" in str(e.value)


def test_state_bits_option():
    """state_bits = 4 stores 4-bit states when every K <= 16; otherwise the
    context is refused (SAME_ECARD); other values are SAME_EINVAL.  The
    colouring and CPT layout do not depend on it."""
    net = koller()
    pptr, pidx, card = net.csr()
    a = same.same_create(pptr, pidx, card)
    b = same.same_create_ex(pptr, pidx, card, state_bits=4)
    assert (a.state_bits, b.state_bits) == (8, 4)
    assert np.array_equal(a.color, b.color) and np.array_equal(a.cpt_off, b.cpt_off)
    assert same.same_layout(b)["state_bits"] == 4 and b.state_bytes == 1
    big = np.array(card, dtype=np.int32)
    big[0] = 17
    with pytest.raises(same.SameError) as e:
        same.same_create_ex(pptr, pidx, big, state_bits=4)
    assert e.value.code == same.SAME_ECARD
    with pytest.raises(same.SameError) as e:
        same.same_create_ex(pptr, pidx, card, state_bits=5)
    assert e.value.code == same.SAME_EINVAL
    big[0] = 200
    assert same.same_create(pptr, pidx, big).state_bits == 16
