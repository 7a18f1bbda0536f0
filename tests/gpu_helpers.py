"""Helpers for the GPU parity tests: run the library on workload arrays and
compare with the oracle on the same arrays."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_1511_06416_amd as same

REL_TOL = 1e-5       # conditionals, fp32 vs fp64
TINY = 1e-30         # below this the oracle's probability is not compared relatively


def context_for(net, prior=1.0, table_limit=None, tile_bytes=0, lds_limit=None, packed=True, state_bits=0):
    """Library context; table_limit=0 forces every node onto the product path,
    a small tile_bytes forces sweeps over several column tiles, lds_limit=0
    reads every table from global memory, packed=False sends every
    product-mode node through the 32-bit index kernel, state_bits=4 stores
    4-bit states."""
    pptr, pidx, card = net.csr()
    if table_limit is None and not tile_bytes and lds_limit is None and packed and not state_bits:
        return same.same_create(pptr, pidx, card, prior)
    return same.same_create_ex(pptr, pidx, card, prior,
                               -1 if table_limit is None else table_limit, tile_bytes,
                               -1 if lds_limit is None else lds_limit, packed, state_bits=state_bits)


def bits_of(ctx):
    """pack_states/unpack_states argument for a context's state format."""
    return 4 if ctx.state_bits == 4 else None


def to_device(ctx, states):
    """[n][m][ld] numpy array or tensor -> the context's state layout on the GPU."""
    q = same.pack_states(states, bits_of(ctx))
    return (torch.from_numpy(q) if isinstance(q, np.ndarray) else q).cuda()


def from_device(ctx, quads, m):
    """The context's state layout (device tensor) -> [n][m][ld] numpy array."""
    return same.unpack_states(quads.cpu().numpy(), m, bits_of(ctx))


def gpu_sweep(ctx, states_np, obs_np, theta_np, m, n_cols, col_offset, seed, sweep_id, win=None,
              stream=None):
    """Runs one library sweep on copies of the given host arrays (states
    [n][m][ld], packed into the library's replica quads); returns (states
    after, as [n][m][ld], probs or None)."""
    st = to_device(ctx, np.ascontiguousarray(states_np))
    ob = torch.from_numpy(np.ascontiguousarray(obs_np)).cuda()
    th = torch.from_numpy(np.ascontiguousarray(theta_np, dtype=np.float32)).cuda()
    ws = ctx.new_workspace()
    ld = st.shape[2]
    probs = None
    if win is not None:
        probs = torch.full((ctx.n_nodes, m, win[1], ctx.max_card), float("nan"), device="cuda")
        same.same_sweep_debug(ctx, st, ob, th, m, n_cols, ld, col_offset, seed, sweep_id, win[0],
                              win[1], probs, ws, stream)
    else:
        same.same_sweep(ctx, st, ob, th, m, n_cols, ld, col_offset, seed, sweep_id, ws, stream)
    torch.cuda.synchronize()
    return from_device(ctx, st, m), (probs.cpu().numpy() if probs is not None else None)


def gpu_sweep_both(ctx, states_np, obs_np, theta_np, m, n_cols, col_offset, seed, sweep_id, win=None):
    """The production sweep (same_sweep) on one copy of the inputs and, when a
    window is asked for, the debug sweep (same_sweep_debug, which also writes
    the conditionals) on another.  The two are separate kernel builds (the
    production one is compiled for a higher occupancy bound and writes no
    conditionals), so each is compared with the oracle on its own.  Returns (production states,
    debug states or None, probs or None)."""
    prod, _ = gpu_sweep(ctx, states_np, obs_np, theta_np, m, n_cols, col_offset, seed, sweep_id)
    if win is None:
        return prod, None, None
    dbg, probs = gpu_sweep(ctx, states_np, obs_np, theta_np, m, n_cols, col_offset, seed, sweep_id, win=win)
    return prod, dbg, probs


def visit_order(color):
    return sorted(range(len(color)), key=lambda i: (int(color[i]), i))


MISMATCH_RATE = 1e-5  # excused boundary mismatches per latent draw


def compare_states(gpu, ref, flags, color, n_cols, obs=None):
    """States must agree chain by chain (column, replica) up to the first
    differing draw in visit order, and that draw must be a flagged boundary
    draw.  With obs, the excused mismatches must also stay under 1e-5 of all
    latent draws (checked where the case has at least 1e6 draws, so that the
    rate is meaningful).  Returns dict with counts; raises AssertionError
    otherwise."""
    assert gpu.shape == ref.shape
    diff = gpu[:, :, :n_cols] != ref[:, :, :n_cols]
    # untouched padding
    assert np.array_equal(gpu[:, :, n_cols:], ref[:, :, n_cols:])
    chains = np.argwhere(diff.any(axis=0))  # (r, j) pairs with any difference
    order = visit_order(color)
    excused = 0
    for r, j in chains:
        first = next(i for i in order if diff[i, r, j])
        assert flags[first, r, j] == 1, (
            "unflagged mismatch at node %d replica %d column %d: gpu %d oracle %d"
            % (first, r, j, gpu[first, r, j], ref[first, r, j]))
        excused += 1
    out = {"mismatched_chains": excused, "flagged": int(flags[:, :, :n_cols].sum()),
           "diff_entries": int(diff.sum())}
    if obs is not None:
        draws = int((obs[:, :n_cols] == 0).sum()) * gpu.shape[1]
        out["draws"] = draws
        out["mismatch_rate"] = excused / max(draws, 1)
        if draws >= 1_000_000:
            assert excused < MISMATCH_RATE * draws, out
    return out


def compare_probs(gpu_p, ref_p, obs, card, win, diverged=None):
    """Window conditionals: relative 1e-5 where the oracle's p >= 1e-30, else
    the library's p below 1e-29.  Chains marked in diverged [m][win] (whose
    states differed earlier in the sweep) are skipped."""
    n, m, W, kmax = ref_p.shape
    worst, checked = 0.0, 0
    for i in range(n):
        K = int(card[i])
        lat = (obs[i, win[0]:win[0] + W] == 0)[None, :].repeat(m, axis=0)
        if diverged is not None:
            lat &= ~diverged
        p = ref_p[i, :, :, :K][lat]
        q = gpu_p[i, :, :, :K][lat].astype(np.float64)
        if p.size == 0:
            continue
        big = p >= TINY
        rel = np.abs(q[big] - p[big]) / p[big]
        if rel.size:
            worst = max(worst, float(rel.max()))
        bad = np.argwhere(rel > REL_TOL)
        assert bad.size == 0, ("node", i, "worst rel", float(rel.max()))
        assert np.all(q[~big] < 1e-29), ("node", i)
        checked += p.shape[0]
    return {"checked": checked, "worst_rel": worst}


def diverged_chains(gpu, ref, n_cols, win):
    """[m][win] mask of chains whose states differ anywhere in the sweep."""
    d = (gpu[:, :, :n_cols] != ref[:, :, :n_cols]).any(axis=0)
    return d[:, win[0]:win[0] + win[1]]
