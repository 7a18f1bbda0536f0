"""Reference oracle for SAME Gibbs sampling (arXiv 1511.06416) -- TEST INFRASTRUCTURE.

A ctypes wrapper around ``same_oracle.c``, a plain fp64 CPU implementation of
the SAME Gibbs sweep, the count histogram, the moving sum and the Dirichlet
resample.  Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import this package.  It shares no code with the HIP
library and never imports it; the two meet only on arrays produced by the
seeded input generators in ``workloads``.

Every wrapper takes numpy arrays and returns numpy arrays.  See the C file's
header for the paper passages each routine follows and for the readings taken
where the paper is silent.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "same_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

FLAG_BAND = 1e-6
FLT_MIN = float(np.finfo(np.float32).tiny)


def build(force: bool = False) -> str:
    """Compile ``same_oracle.c`` with gcc into ``liboracle.so`` (in place)."""
    if force or not os.path.exists(_LIB_PATH) or (
        os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)
    ):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
        )
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _i32p(a):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build()
            L = C.CDLL(_LIB_PATH)
            P = C.c_void_p
            L.oracle_philox4x32_10.argtypes = [P, P, P]
            L.oracle_philox4x32_10.restype = None
            L.oracle_gibbs_uniform.argtypes = [C.c_uint64, C.c_int32, C.c_int32, C.c_int64, C.c_uint32]
            L.oracle_gibbs_uniform.restype = C.c_double
            L.oracle_graph.argtypes = [C.c_int32, P, P, P, P, P, P, P]
            L.oracle_graph.restype = C.c_int
            L.oracle_graph_ex.argtypes = [C.c_int32, P, P, P, C.c_int32, P, P, P, P]
            L.oracle_graph_ex.restype = C.c_int
            L.oracle_moral.argtypes = [C.c_int32, P, P, P, P]
            L.oracle_moral.restype = C.c_int
            L.oracle_conditional.argtypes = [C.c_int32, P, P, P, P, P, C.c_int32, P]
            L.oracle_conditional.restype = C.c_int
            L.oracle_conditionals.argtypes = [C.c_int32, P, P, P, P, P, C.c_int64, C.c_int32, P]
            L.oracle_conditionals.restype = C.c_int
            L.oracle_draw.argtypes = [P, C.c_int32, C.c_double, P]
            L.oracle_draw.restype = C.c_int32
            L.oracle_sweep.argtypes = [
                C.c_int32, P, P, P, P, P, C.c_int32, P, P, C.c_int32, C.c_int64, C.c_int64,
                C.c_int64, C.c_uint64, C.c_uint32, P, C.c_int64, C.c_int64, P, C.c_int32,
                C.c_int32,
            ]
            L.oracle_sweep.restype = C.c_int64
            L.oracle_counts.argtypes = [
                C.c_int32, P, P, P, C.c_int32, P, C.c_int32, C.c_int64, C.c_int64, P, C.c_int32,
            ]
            L.oracle_counts.restype = C.c_int
            L.oracle_gamma.argtypes = [C.c_double, C.c_uint64, C.c_uint32, C.c_uint32, P]
            L.oracle_gamma.restype = C.c_double
            L.oracle_dirichlet.argtypes = [
                C.c_int32, P, P, P, P, C.c_double, C.c_uint64, C.c_uint32, P, P,
            ]
            L.oracle_dirichlet.restype = C.c_int
            L.oracle_expand.argtypes = [C.c_int32, C.c_int64, C.c_int32, C.c_int64, P, P, P, C.c_int32,
                                        P, P]
            L.oracle_expand.restype = C.c_int
            L.oracle_init_latent.argtypes = [C.c_int32, P, C.c_int64, C.c_int32, C.c_int64, C.c_int64,
                                             C.c_uint64, C.c_int32, P, P]
            L.oracle_init_latent.restype = C.c_int
            L.oracle_accumulate_hits.argtypes = [C.c_int32, C.c_int64, C.c_int32, C.c_int64, C.c_int32,
                                                 P, P, P]
            L.oracle_accumulate_hits.restype = C.c_int
            L.oracle_dirichlet_f64.argtypes = [C.c_int32, P, P, P, P, C.c_double, C.c_uint64, C.c_uint32, P, P]
            L.oracle_dirichlet_f64.restype = C.c_int
            L.oracle_ema.argtypes = [C.c_int64, C.c_double, P, P]
            L.oracle_ema.restype = None
            L.oracle_grow_replicas.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int64, C.c_int32, P, P]
            L.oracle_grow_replicas.restype = C.c_int
            _lib = L
        return _lib


class OracleError(RuntimeError):
    pass


def _check(rc):
    if rc < 0:
        raise OracleError("oracle returned error %d" % rc)
    return rc


def _dag(parents, card):
    """(parent_ptr, parent_idx, card) int32 arrays from a list of parent lists."""
    pptr = np.zeros(len(parents) + 1, dtype=np.int32)
    for i, ps in enumerate(parents):
        pptr[i + 1] = pptr[i] + len(ps)
    pidx = np.array([p for ps in parents for p in ps] or [0], dtype=np.int32)
    return pptr, pidx, np.ascontiguousarray(card, dtype=np.int32)


def _ptr(a):
    return C.c_void_p(a.ctypes.data) if a is not None else None


# ----------------------------------------------------------------------------
# Philox


def philox4x32_10(ctr, key):
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def gibbs_uniform(seed, node, replica, gcol, sweep_id):
    return lib().oracle_gibbs_uniform(int(seed), int(node), int(replica), int(gcol), int(sweep_id))


# ----------------------------------------------------------------------------
# Graph


def graph(parents, card, balance=True):
    """Returns dict(cpt_off[n+1], topo[n], color[n], n_colors); balance=False
    gives the first-fit colouring before the balancing moves."""
    pptr, pidx, card = _dag(parents, card)
    n = len(card)
    off = np.zeros(n + 1, dtype=np.int64)
    topo = np.zeros(n, dtype=np.int32)
    color = np.zeros(n, dtype=np.int32)
    nc = C.c_int32(0)
    _check(lib().oracle_graph_ex(n, _ptr(pptr), _ptr(pidx), _ptr(card), 1 if balance else 0, _ptr(off),
                                 _ptr(topo), _ptr(color), C.byref(nc)))
    return {"cpt_off": off, "topo": topo, "color": color, "n_colors": nc.value}


def graph_rc(parents_ptr, parents_idx, card):
    """Raw return code of the oracle's graph validation (for error tests)."""
    pptr = np.ascontiguousarray(parents_ptr, dtype=np.int32)
    pidx = np.ascontiguousarray(parents_idx if len(parents_idx) else [0], dtype=np.int32)
    card = np.ascontiguousarray(card, dtype=np.int32)
    return lib().oracle_graph(len(card), _ptr(pptr), _ptr(pidx), _ptr(card), None, None, None, None)


def moral_adjacency(parents, card):
    pptr, pidx, card = _dag(parents, card)
    n = len(card)
    adj = np.zeros((n, n), dtype=np.uint8)
    _check(lib().oracle_moral(n, _ptr(pptr), _ptr(pidx), _ptr(card), _ptr(adj)))
    return adj.astype(bool)


# ----------------------------------------------------------------------------
# Conditional and draw


def conditional(parents, card, theta, x, node):
    pptr, pidx, card = _dag(parents, card)
    th = np.ascontiguousarray(theta, dtype=np.float32)
    xv = np.ascontiguousarray(x, dtype=np.int32)
    p = np.zeros(int(card[node]), dtype=np.float64)
    _check(lib().oracle_conditional(len(card), _ptr(pptr), _ptr(pidx), _ptr(card), _ptr(th),
                                    _ptr(xv), int(node), _ptr(p)))
    return p


def conditionals(parents, card, theta, X, node):
    """conditional() for every row of X ([count][n] states), as [count][K]."""
    pptr, pidx, card = _dag(parents, card)
    th = np.ascontiguousarray(theta, dtype=np.float32)
    xv = np.ascontiguousarray(X, dtype=np.int32)
    assert xv.ndim == 2 and xv.shape[1] == len(card)
    p = np.zeros((xv.shape[0], int(card[node])), dtype=np.float64)
    _check(lib().oracle_conditionals(len(card), _ptr(pptr), _ptr(pidx), _ptr(card), _ptr(th), _ptr(xv),
                                     int(xv.shape[0]), int(node), _ptr(p)))
    return p


def draw(weights, u):
    w = np.ascontiguousarray(weights, dtype=np.float64)
    f = C.c_int32(0)
    k = lib().oracle_draw(_ptr(w), len(w), float(u), C.byref(f))
    return int(k), bool(f.value)


# ----------------------------------------------------------------------------
# Sweep, counts, Dirichlet


def sweep(parents, card, theta, color, states, obs, m, n_cols, col_offset, seed, sweep_id,
          want_flags=False, win=None, n_threads=0):
    """One sweep over one minibatch; ``states`` ([n][m][ld] int8/int16) is updated in place.

    Returns dict(draws, flags (or None), probs (or None)).
    ``win`` = (win_begin, win_len) asks for the conditionals of those columns.
    """
    pptr, pidx, card = _dag(parents, card)
    th = np.ascontiguousarray(theta, dtype=np.float32)
    col = np.ascontiguousarray(color, dtype=np.int32)
    assert states.flags.c_contiguous and obs.flags.c_contiguous
    n = len(card)
    ld = states.shape[-1]
    assert states.shape == (n, m, ld) and obs.shape == (n, ld)
    sb = states.dtype.itemsize
    flags = np.zeros(states.shape, dtype=np.uint8) if want_flags else None
    probs = None
    wb, wl, kmax = 0, 0, 1
    if win is not None:
        wb, wl = int(win[0]), int(win[1])
        kmax = int(card.max())
        probs = np.full((n, m, wl, kmax), np.nan, dtype=np.float64)
    draws = lib().oracle_sweep(
        n, _ptr(pptr), _ptr(pidx), _ptr(card), _ptr(th), _ptr(col), sb, _ptr(states), _ptr(obs),
        int(m), int(n_cols), int(ld), int(col_offset), int(seed), int(sweep_id), _ptr(flags),
        wb, wl, _ptr(probs), kmax, int(n_threads))
    _check(draws)
    return {"draws": int(draws), "flags": flags, "probs": probs}


def counts(parents, card, states, m, n_cols, n_threads=0):
    pptr, pidx, card = _dag(parents, card)
    n = len(card)
    ld = states.shape[-1]
    assert states.shape == (n, m, ld) and states.flags.c_contiguous
    total = graph(parents, card)["cpt_off"][-1]
    out = np.zeros(int(total), dtype=np.int64)
    _check(lib().oracle_counts(n, _ptr(pptr), _ptr(pidx), _ptr(card), states.dtype.itemsize,
                               _ptr(states), int(m), int(n_cols), int(ld), _ptr(out),
                               int(n_threads)))
    return out


def gamma(shape, seed, entry, update_id):
    att = C.c_int32(0)
    g = lib().oracle_gamma(float(shape), int(seed), int(entry), int(update_id), C.byref(att))
    return g, att.value


def dirichlet(parents, card, totals, alpha, seed, update_id, want_gamma=False):
    pptr, pidx, card = _dag(parents, card)
    tot = np.ascontiguousarray(totals, dtype=np.int64)
    theta = np.zeros(len(tot), dtype=np.float32)
    gv = np.zeros(len(tot), dtype=np.float64) if want_gamma else None
    _check(lib().oracle_dirichlet(len(card), _ptr(pptr), _ptr(pidx), _ptr(card), _ptr(tot),
                                  float(alpha), int(seed), int(update_id), _ptr(theta), _ptr(gv)))
    return (theta, gv) if want_gamma else theta


def moving_sum(totals, mb_prev, new):
    """Exact moving sum of the per-minibatch counts (Sec. 4): subtract this
    minibatch's previous counts from the total, add its new counts."""
    return totals - mb_prev + new


def expand(n, n_cols, m, ld, row_ptr, col_idx, values, states, obs):
    """Dense minibatch from its known entries in CSR form (rows = variables,
    Sec. 4): obs is cleared, then every stored entry is marked observed and
    written into all m replicas of states (in place); latent entries of states
    are left as they are."""
    row_ptr = np.ascontiguousarray(row_ptr, dtype=np.int64)
    col_idx = np.ascontiguousarray(col_idx, dtype=np.int32)
    values = np.ascontiguousarray(values, dtype=states.dtype)
    assert states.shape == (n, m, ld) and states.flags.c_contiguous
    assert obs.shape == (n, ld) and obs.dtype == np.uint8 and obs.flags.c_contiguous
    _check(lib().oracle_expand(int(n), int(n_cols), int(m), int(ld), _ptr(row_ptr), _ptr(col_idx),
                               _ptr(values), states.dtype.itemsize, _ptr(states), _ptr(obs)))


def init_latent(card, n_cols, m, col_offset, seed, states, obs):
    """Random initial latent states (Sec. 5.2), in place: every latent entry
    of every replica becomes floor(U * K_i) from its Philox uniform (tag 2)."""
    card = np.ascontiguousarray(card, dtype=np.int32)
    n = len(card)
    ld = states.shape[-1]
    assert states.shape == (n, m, ld) and states.flags.c_contiguous and obs.shape == (n, ld)
    _check(lib().oracle_init_latent(n, _ptr(card), int(n_cols), int(m), int(ld), int(col_offset),
                                    int(seed), states.dtype.itemsize, _ptr(states),
                                    _ptr(np.ascontiguousarray(obs, dtype=np.uint8))))


def accumulate_hits(states, target, m, n_cols, hits):
    """Held-out prediction (Sec. 6), in place: hits[i][j] += number of replicas
    whose state equals target[i][j] at every test entry (target >= 0)."""
    n, _, ld = states.shape
    assert target.shape == (n, ld) and target.dtype == states.dtype and target.flags.c_contiguous
    assert hits.shape == (n, ld) and hits.dtype == np.int32 and hits.flags.c_contiguous
    _check(lib().oracle_accumulate_hits(int(n), int(n_cols), int(m), int(ld), states.dtype.itemsize,
                                        _ptr(np.ascontiguousarray(states)), _ptr(target), _ptr(hits)))


def predict(parents, card, theta, color, states, obs, target, m, n_cols, col_offset, seed,
            sweep_id0, n_sweeps):
    """Testing phase of Sec. 6: n_sweeps sequential-scan sweeps with the CPTs
    frozen (test entries latent in obs), the hits accumulated after each.
    states is updated in place; returns hits (int32 [n][ld])."""
    n, _, ld = states.shape
    hits = np.zeros((n, ld), dtype=np.int32)
    for s in range(n_sweeps):
        sweep(parents, card, theta, color, states, obs, m, n_cols, col_offset, seed, sweep_id0 + s)
        accumulate_hits(states, target, m, n_cols, hits)
    return hits


def ema(totals, decay, new):
    """Exponential moving sum (Sec. 4 footnote), in place on fp64 totals:
    totals = decay * totals + new."""
    assert totals.dtype == np.float64 and totals.flags.c_contiguous
    nc = np.ascontiguousarray(new, dtype=np.int64)
    assert nc.shape == totals.shape
    lib().oracle_ema(int(totals.size), float(decay), _ptr(nc), _ptr(totals))


def dirichlet_f64(parents, card, totals, alpha, seed, update_id, want_gamma=False):
    """Dirichlet resample from fp64 (moving-sum) totals."""
    pptr, pidx, card = _dag(parents, card)
    tot = np.ascontiguousarray(totals, dtype=np.float64)
    theta = np.zeros(len(tot), dtype=np.float32)
    gv = np.zeros(len(tot), dtype=np.float64) if want_gamma else None
    _check(lib().oracle_dirichlet_f64(len(card), _ptr(pptr), _ptr(pidx), _ptr(card), _ptr(tot), float(alpha),
                                      int(seed), int(update_id), _ptr(theta), _ptr(gv)))
    return (theta, gv) if want_gamma else theta


def grow_replicas(states, m2):
    """SAME annealing (Sec. 3): states [n][m][ld] -> [n][m2][ld]; replica r >= m
    starts as a copy of replica r mod m."""
    n, m, ld = states.shape
    src = np.ascontiguousarray(states)
    out = np.zeros((n, m2, ld), dtype=states.dtype)
    _check(lib().oracle_grow_replicas(int(n), int(m), int(m2), int(ld), states.dtype.itemsize, _ptr(src),
                                      _ptr(out)))
    return out
