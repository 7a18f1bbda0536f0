"""MI355X (gfx950) SAME Gibbs sampling for discrete Bayesian networks.

A thin ctypes binding over ``libsame.so`` (C ABI declared in
``include/same.h``).  The functions carry the C names and only marshal
arguments: tensors become device pointers, the stream defaults to torch's
current stream.  Every step of the sampler runs in the library's HIP
kernels; there is no Python or CPU fallback, and calling anything here
without the built library raises ``SameError``.
"""
from __future__ import annotations

import ctypes as C
import os
import threading

import numpy as np

__all__ = [
    "SameError", "Context", "same_create", "same_create_ex", "same_destroy", "same_layout", "same_workspace_size",
    "same_sweep", "same_sweep_debug", "same_counts", "same_sample_cpts", "same_last_error",
    "same_step", "same_sweep_plan", "same_stream_slots_size", "same_stream_pass", "SAME_STREAM_COUNTS_ONLY",
    "same_kernel_timing", "same_kernel_times", "same_expand_observed", "same_init_latent",
    "same_accumulate_hits", "same_predict", "same_counts_ema", "same_sample_cpts_ema", "same_stream_pass_ema",
    "same_grow_replicas", "same_debug_thresholds", "same_counts_noalloc", "same_stream_compact_layout",
    "same_stream_pass_compact", "same_step_graph", "same_graph_launch", "same_graph_destroy", "StepGraph",
    "pack_states", "unpack_states", "state_shape",
    "library_path", "load_library",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsame.so")
_lock = threading.Lock()
_lib = None

SAME_OK, SAME_EINVAL, SAME_EGRAPH, SAME_ECARD, SAME_ESIZE, SAME_ENOMEM, SAME_EHIP, SAME_EALIGN = (
    0, -1, -2, -3, -4, -5, -6, -7)
SAME_STREAM_COUNTS_ONLY = 1
_NAMES = {0: "SAME_OK", -1: "SAME_EINVAL", -2: "SAME_EGRAPH", -3: "SAME_ECARD",
          -4: "SAME_ESIZE", -5: "SAME_ENOMEM", -6: "SAME_EHIP", -7: "SAME_EALIGN"}


class SameError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s (%d): %s" % (_NAMES.get(code, "?"), code, msg))
        self.code = code


class _Options(C.Structure):
    _fields_ = [("table_limit", C.c_int64), ("tile_bytes", C.c_int64), ("lds_limit", C.c_int64),
                ("packed_indices", C.c_int32), ("first_fit_colours", C.c_int32), ("state_bits", C.c_int32)]


class _KernelTimes(C.Structure):
    _fields_ = [("ms", C.c_double * 4), ("launches", C.c_int64 * 4), ("phase_ms", C.c_double),
                ("phases", C.c_int64), ("node_samples", C.c_double * 4)]


class _Layout(C.Structure):
    _fields_ = [("n_nodes", C.c_int32), ("n_colors", C.c_int32), ("cpt_total", C.c_int64),
                ("n_rows", C.c_int64), ("state_bytes", C.c_int32), ("max_card", C.c_int32),
                ("sweep_launches", C.c_int32), ("table_nodes", C.c_int32), ("state_bits", C.c_int32)]


def library_path() -> str:
    return _LIB_PATH


def load_library():
    """Loads libsame.so; raises SameError if it has not been built."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(_LIB_PATH):
            raise SameError(SAME_EINVAL, "libsame.so is not built (run __graft_entry__.build())")
        L = C.CDLL(_LIB_PATH)
        P, I32, I64, U64, U32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_uint32
        L.same_create.argtypes = [I32, P, P, P, C.c_double, C.POINTER(P)]
        L.same_create_ex.argtypes = [I32, P, P, P, C.c_double, C.POINTER(_Options), C.POINTER(P)]
        L.same_destroy.argtypes = [P]
        L.same_destroy.restype = None
        L.same_layout.argtypes = [P, C.POINTER(_Layout), P, P]
        L.same_workspace_size.argtypes = [P, C.POINTER(C.c_size_t)]
        L.same_sweep.argtypes = [P, P, P, P, I32, I64, I64, I64, U64, U32, P, P]
        L.same_sweep_debug.argtypes = [P, P, P, P, I32, I64, I64, I64, U64, U32, I64, I64, P, P, P]
        L.same_counts.argtypes = [P, P, I32, I64, I64, P, P, P, P]
        L.same_sample_cpts.argtypes = [P, P, P, U64, U32, P, P]
        L.same_step.argtypes = [P, P, P, P, I32, I64, I64, I64, U64, U32, P, P, U32, P, P]
        L.same_sweep_plan.argtypes = [P, I32, I64, C.POINTER(C.c_int64), C.POINTER(C.c_int32)]
        L.same_stream_slots_size.argtypes = [P, I32, I64, C.POINTER(C.c_size_t)]
        L.same_stream_pass.argtypes = [P, P, P, I64, I64, I64, I32, P, P, P, U64, U32, I32, P, P, P]
        L.same_kernel_timing.argtypes = [P, I32]
        L.same_kernel_times.argtypes = [P, C.POINTER(_KernelTimes)]
        L.same_expand_observed.argtypes = [P, P, P, P, I64, I32, I64, I64, P, P, P]
        L.same_init_latent.argtypes = [P, P, P, I32, I64, I64, I64, U64, P]
        L.same_accumulate_hits.argtypes = [P, P, P, I32, I64, I64, P, P]
        L.same_counts_ema.argtypes = [P, P, I32, I64, I64, C.c_double, P, P, P]
        L.same_grow_replicas.argtypes = [P, P, I32, P, I32, I64, P]
        L.same_sample_cpts_ema.argtypes = [P, P, P, U64, U32, P, P]
        L.same_stream_pass_ema.argtypes = [P, P, P, I64, I64, I64, I32, P, P, C.c_double, U64, U32, I32, P, P,
                                           P]
        L.same_predict.argtypes = [P, P, P, P, P, I32, I64, I64, I64, U64, U32, I32, P, P, P]
        L.same_counts_noalloc.argtypes = [P, P, I32, I64, I64, P, P, P]
        L.same_stream_compact_layout.argtypes = [P, P, I64, I64, I64, I32, P, C.POINTER(C.c_size_t), P, P]
        L.same_stream_pass_compact.argtypes = [P, P, P, P, P, I64, I64, I64, I32, P, P, P, U64, U32, I32, P, P, P]
        L.same_debug_thresholds.argtypes = [P, P, P, P, C.POINTER(C.c_int64), P, P, P]
        L.same_step_graph.argtypes = [P, P, P, P, I32, I64, I64, I64, U64, P, P, P, U32, I32, P, C.POINTER(P)]
        L.same_graph_launch.argtypes = [P, P]
        L.same_graph_destroy.argtypes = [P]
        L.same_graph_destroy.restype = None
        L.same_last_error.argtypes = []
        L.same_last_error.restype = C.c_char_p
        for f in ("same_create", "same_create_ex", "same_layout", "same_workspace_size", "same_sweep",
                  "same_sweep_debug", "same_counts", "same_sample_cpts", "same_step", "same_sweep_plan",
                  "same_stream_slots_size", "same_stream_pass", "same_kernel_timing",
                  "same_kernel_times", "same_expand_observed", "same_init_latent",
                  "same_accumulate_hits", "same_predict", "same_counts_ema", "same_sample_cpts_ema",
                  "same_stream_pass_ema", "same_grow_replicas", "same_debug_thresholds",
                  "same_counts_noalloc", "same_stream_compact_layout", "same_stream_pass_compact",
                  "same_step_graph", "same_graph_launch"):
            getattr(L, f).restype = C.c_int
        _lib = L
        return L


def same_last_error() -> str:
    return load_library().same_last_error().decode()


def _check(rc):
    if rc != SAME_OK:
        raise SameError(rc, same_last_error())


def _ptr(t):
    """Device pointer of a tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return C.c_void_p(t)
    return C.c_void_p(t.data_ptr())


def state_shape(n, m, ld, bits=8):
    """Shape of a states array of n nodes, m replicas and leading dimension
    ld: replica quads [n][ceil(m / 4)][ld][4] of 8- or 16-bit states, or
    [n][ceil(m / 4)][ld] 16-bit words of four 4-bit states (see
    include/same.h)."""
    mq = (int(m) + 3) // 4
    return (int(n), mq, int(ld)) if bits == 4 else (int(n), mq, int(ld), 4)


def pack_states(states, bits=None):
    """[n][m][ld] (replica rows) -> the library's replica quads (padding slots
    0): [n][ceil(m/4)][ld][4] in the same dtype, or with bits=4 (values below
    16) [n][ceil(m/4)][ld] int16 words, replica 4q + s in bits 4s .. 4s + 3.
    torch tensor (same device) or numpy array; a layout permutation for
    callers, not part of any entry point."""
    n, m, ld = states.shape
    mq = (m + 3) // 4
    pad = 4 * mq - m
    if isinstance(states, np.ndarray):
        if pad:
            states = np.concatenate([states, np.zeros((n, pad, ld), dtype=states.dtype)], axis=1)
        q = np.ascontiguousarray(states.reshape(n, mq, 4, ld).transpose(0, 1, 3, 2))
        if bits == 4:
            w = q.astype(np.int32) & 0xF
            q = (w[..., 0] | (w[..., 1] << 4) | (w[..., 2] << 8) | (w[..., 3] << 12)).astype(np.uint16).view(np.int16)
            q = np.ascontiguousarray(q)
        return q
    if pad:
        states = torch_cat([states, states.new_zeros((n, pad, ld))], 1)
    q = states.reshape(n, mq, 4, ld).permute(0, 1, 3, 2).contiguous()
    if bits == 4:
        import torch
        w = q.to(torch.int32) & 0xF
        q = (w[..., 0] | (w[..., 1] << 4) | (w[..., 2] << 8) | (w[..., 3] << 12))
        q = torch.where(q >= 0x8000, q - 0x10000, q).to(torch.int16).contiguous()
    return q


def unpack_states(quads, m, bits=None):
    """The library's replica quads -> [n][m][ld] (padding slots dropped); with
    bits=4 the int16 words of four 4-bit states, returned as int8."""
    if bits == 4:
        n, mq, ld = quads.shape
        if isinstance(quads, np.ndarray):
            w = quads.view(np.uint16).astype(np.int32)
            q = np.stack([(w >> (4 * s)) & 0xF for s in range(4)], axis=-1).astype(np.int8)
        else:
            import torch
            w = quads.to(torch.int32) & 0xFFFF
            q = torch.stack([(w >> (4 * s)) & 0xF for s in range(4)], dim=-1).to(torch.int8)
        quads = q
    n, mq, ld, four = quads.shape
    assert four == 4 and 4 * mq >= m
    if isinstance(quads, np.ndarray):
        return np.ascontiguousarray(quads.transpose(0, 1, 3, 2).reshape(n, 4 * mq, ld)[:, :m])
    return quads.permute(0, 1, 3, 2).reshape(n, 4 * mq, ld)[:, :m].contiguous()


def torch_cat(ts, dim):
    import torch
    return torch.cat(ts, dim)


def _st(ctx, t, m, ld, what="states"):
    """A states tensor must have the library's layout and be contiguous: a
    tensor in another layout is refused here, before any device call."""
    if t is None or isinstance(t, int):
        return t
    want = state_shape(ctx.n_nodes, m, ld, ctx.state_bits)
    if tuple(t.shape) != want:
        raise SameError(SAME_EINVAL, "%s must have shape %s (replica quads, see pack_states), got %s"
                        % (what, want, tuple(t.shape)))
    if hasattr(t, "is_contiguous") and not t.is_contiguous():
        raise SameError(SAME_EINVAL, "%s must be contiguous" % what)
    return t


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


class Context:
    """Owns one same_ctx (one network)."""

    def __init__(self, parent_ptr, parent_idx, card, dirichlet_prior=1.0, table_limit=None,
                 tile_bytes=0, lds_limit=None, packed_indices=True, first_fit_colours=False, state_bits=0):
        L = load_library()
        self._pptr = np.ascontiguousarray(parent_ptr, dtype=np.int32)
        self._pidx = np.ascontiguousarray(parent_idx if len(parent_idx) else [0], dtype=np.int32)
        self._card = np.ascontiguousarray(card, dtype=np.int32)
        h = C.c_void_p()
        if (table_limit is None and not tile_bytes and lds_limit is None and packed_indices and not first_fit_colours
                and not state_bits):
            _check(L.same_create(len(self._card), self._pptr.ctypes.data, self._pidx.ctypes.data,
                                 self._card.ctypes.data, float(dirichlet_prior), C.byref(h)))
        else:
            opts = _Options(-1 if table_limit is None else int(table_limit), int(tile_bytes),
                            -1 if lds_limit is None else int(lds_limit), 1 if packed_indices else 0,
                            1 if first_fit_colours else 0, int(state_bits))
            _check(L.same_create_ex(len(self._card), self._pptr.ctypes.data,
                                    self._pidx.ctypes.data, self._card.ctypes.data,
                                    float(dirichlet_prior), C.byref(opts), C.byref(h)))
        self._h = h
        lay = _Layout()
        off = np.zeros(len(self._card) + 1, dtype=np.int64)
        col = np.zeros(len(self._card), dtype=np.int32)
        _check(L.same_layout(self._h, C.byref(lay), off.ctypes.data, col.ctypes.data))
        self.n_nodes, self.n_colors = lay.n_nodes, lay.n_colors
        self.cpt_total, self.n_rows = lay.cpt_total, lay.n_rows
        self.state_bytes, self.max_card = lay.state_bytes, lay.max_card
        self.sweep_launches, self.table_nodes = lay.sweep_launches, lay.table_nodes
        self.state_bits = lay.state_bits
        self.cpt_off, self.color = off, col
        ws = C.c_size_t()
        _check(L.same_workspace_size(self._h, C.byref(ws)))
        self.workspace_bytes = int(ws.value)

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load_library().same_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def new_workspace(self, device="cuda"):
        import torch
        # torch's caching allocator returns >= 512-byte aligned blocks
        return torch.empty(max(self.workspace_bytes, 1), dtype=torch.uint8, device=device)


def same_create(parent_ptr, parent_idx, card, dirichlet_prior=1.0) -> Context:
    return Context(parent_ptr, parent_idx, card, dirichlet_prior)


def same_create_ex(parent_ptr, parent_idx, card, dirichlet_prior=1.0, table_limit=-1,
                   tile_bytes=0, lds_limit=-1, packed_indices=True, first_fit_colours=False,
                   state_bits=0) -> Context:
    return Context(parent_ptr, parent_idx, card, dirichlet_prior, table_limit=table_limit,
                   tile_bytes=tile_bytes, lds_limit=lds_limit, packed_indices=packed_indices,
                   first_fit_colours=first_fit_colours, state_bits=state_bits)


def same_destroy(ctx: Context) -> None:
    ctx.close()


def same_layout(ctx: Context) -> dict:
    return {"n_nodes": ctx.n_nodes, "n_colors": ctx.n_colors, "cpt_total": ctx.cpt_total,
            "n_rows": ctx.n_rows, "state_bytes": ctx.state_bytes, "max_card": ctx.max_card,
            "sweep_launches": ctx.sweep_launches, "table_nodes": ctx.table_nodes, "state_bits": ctx.state_bits,
            "cpt_off": ctx.cpt_off.copy(), "color": ctx.color.copy()}


def same_workspace_size(ctx: Context) -> int:
    return ctx.workspace_bytes


def same_sweep(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, workspace,
               stream=None):
    _check(load_library().same_sweep(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(obs), _ptr(cpts), int(m),
                                     int(n_cols), int(ld), int(col_offset), int(seed),
                                     int(sweep_id), _ptr(workspace), _stream(stream)))


def same_sweep_debug(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id,
                     win_begin, win, probs, workspace, stream=None):
    _check(load_library().same_sweep_debug(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(obs), _ptr(cpts), int(m),
                                           int(n_cols), int(ld), int(col_offset), int(seed),
                                           int(sweep_id), int(win_begin), int(win), _ptr(probs),
                                           _ptr(workspace), _stream(stream)))


def same_counts(ctx, states, m, n_cols, ld, mb_counts, totals, workspace, stream=None):
    _check(load_library().same_counts(ctx.handle, _ptr(_st(ctx, states, m, ld)), int(m), int(n_cols), int(ld),
                                      _ptr(mb_counts), _ptr(totals), _ptr(workspace),
                                      _stream(stream)))


def same_counts_noalloc(ctx, states, m, n_cols, ld, mb_counts, totals, stream=None):
    """same_counts without a workspace: the histogram lives in the library's
    per-device scratch array (see include/same.h)."""
    _check(load_library().same_counts_noalloc(ctx.handle, _ptr(_st(ctx, states, m, ld)), int(m), int(n_cols), int(ld),
                                              _ptr(mb_counts), _ptr(totals), _stream(stream)))


def same_sample_cpts(ctx, totals, cpts_out, seed, update_id, workspace, stream=None):
    _check(load_library().same_sample_cpts(ctx.handle, _ptr(totals), _ptr(cpts_out), int(seed),
                                           int(update_id), _ptr(workspace), _stream(stream)))


def same_step(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, mb_counts, totals,
              update_id, workspace, stream=None):
    _check(load_library().same_step(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(obs), _ptr(cpts), int(m),
                                    int(n_cols), int(ld), int(col_offset), int(seed), int(sweep_id),
                                    _ptr(mb_counts), _ptr(totals), int(update_id), _ptr(workspace),
                                    _stream(stream)))


class StepGraph:
    """Handle of a captured step graph (same_step_graph); close() or garbage
    collection frees it.  The tensors it was captured with are kept alive."""

    def __init__(self, handle, keep):
        self.handle = handle
        self._keep = keep

    def launch(self, stream=None):
        same_graph_launch(self, stream)

    def close(self):
        if self.handle:
            same_graph_destroy(self)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def same_step_graph(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, mb_counts, totals, ids,
                    update_stride, steps, workspace):
    """Captures `steps` same_step calls whose sweep and update ids are read
    from the two-word device tensor `ids` (advanced by 1 and update_stride
    after each step); returns a StepGraph."""
    h = C.c_void_p()
    _check(load_library().same_step_graph(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(obs), _ptr(cpts), int(m), int(n_cols),
                                          int(ld), int(col_offset), int(seed), _ptr(mb_counts), _ptr(totals),
                                          _ptr(ids), int(update_stride), int(steps), _ptr(workspace),
                                          C.byref(h)))
    return StepGraph(h.value, (ctx, states, obs, cpts, mb_counts, totals, ids, workspace))


def same_graph_launch(graph, stream=None):
    _check(load_library().same_graph_launch(graph.handle, _stream(stream)))


def same_graph_destroy(graph):
    load_library().same_graph_destroy(graph.handle)
    graph.handle = None


def same_sweep_plan(ctx, m, n_cols):
    """(tile width in columns, sweep-kernel launches per same_sweep call)."""
    t, n = C.c_int64(), C.c_int32()
    _check(load_library().same_sweep_plan(ctx.handle, int(m), int(n_cols), C.byref(t), C.byref(n)))
    return int(t.value), int(n.value)


def same_stream_slots_size(ctx, m, nb) -> int:
    out = C.c_size_t()
    _check(load_library().same_stream_slots_size(ctx.handle, int(m), int(nb), C.byref(out)))
    return int(out.value)


def same_stream_pass(ctx, host_states, host_obs, host_ld, n_cols, nb, m, cpts, mb_counts, totals,
                     seed, pass_id, flags, slots, workspace, stream=None):
    """host_states / host_obs: pinned host tensors (or addresses); the rest device."""
    _check(load_library().same_stream_pass(ctx.handle, _ptr(_st(ctx, host_states, m, host_ld, "host_states")), _ptr(host_obs),
                                           int(host_ld), int(n_cols), int(nb), int(m), _ptr(cpts),
                                           _ptr(mb_counts), _ptr(totals), int(seed), int(pass_id),
                                           int(flags), _ptr(slots), _ptr(workspace),
                                           _stream(stream)))


def same_kernel_timing(ctx, enable=True):
    """Starts (or stops) per-launch event timing of ctx's sweep kernels; clears the totals."""
    _check(load_library().same_kernel_timing(ctx.handle, 1 if enable else 0))


def same_kernel_times(ctx):
    """{'ms': [4 floats], 'launches': [4 ints], 'node_samples': [4 floats]} per
    launch class since timing was enabled, and the summed colour-phase time
    'phase_ms' over 'phases' phases."""
    t = _KernelTimes()
    _check(load_library().same_kernel_times(ctx.handle, C.byref(t)))
    return {"ms": list(t.ms), "launches": list(t.launches), "phase_ms": t.phase_ms, "phases": t.phases,
            "node_samples": list(t.node_samples)}


def same_expand_observed(ctx, row_ptr, col_idx, values, nnz, m, n_cols, ld, states, obs, stream=None):
    _check(load_library().same_expand_observed(ctx.handle, _ptr(row_ptr), _ptr(col_idx), _ptr(values),
                                               int(nnz), int(m), int(n_cols), int(ld), _ptr(_st(ctx, states, m, ld)),
                                               _ptr(obs), _stream(stream)))


def same_init_latent(ctx, states, obs, m, n_cols, ld, col_offset, seed, stream=None):
    _check(load_library().same_init_latent(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(obs), int(m), int(n_cols),
                                           int(ld), int(col_offset), int(seed), _stream(stream)))


def same_accumulate_hits(ctx, states, target, m, n_cols, ld, hits, stream=None):
    _check(load_library().same_accumulate_hits(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(target), int(m), int(n_cols),
                                               int(ld), _ptr(hits), _stream(stream)))


def same_predict(ctx, states, obs, cpts, target, m, n_cols, ld, col_offset, seed, sweep_id0, n_sweeps, hits,
                 workspace, stream=None):
    _check(load_library().same_predict(ctx.handle, _ptr(_st(ctx, states, m, ld)), _ptr(obs), _ptr(cpts), _ptr(target), int(m),
                                       int(n_cols), int(ld), int(col_offset), int(seed), int(sweep_id0),
                                       int(n_sweeps), _ptr(hits), _ptr(workspace), _stream(stream)))


def same_counts_ema(ctx, states, m, n_cols, ld, decay, totals, workspace, stream=None):
    _check(load_library().same_counts_ema(ctx.handle, _ptr(_st(ctx, states, m, ld)), int(m), int(n_cols), int(ld), float(decay),
                                          _ptr(totals), _ptr(workspace), _stream(stream)))


def same_sample_cpts_ema(ctx, totals, cpts_out, seed, update_id, workspace, stream=None):
    _check(load_library().same_sample_cpts_ema(ctx.handle, _ptr(totals), _ptr(cpts_out), int(seed),
                                               int(update_id), _ptr(workspace), _stream(stream)))


def same_stream_pass_ema(ctx, host_states, host_obs, host_ld, n_cols, nb, m, cpts, totals, decay, seed, pass_id,
                         flags, slots, workspace, stream=None):
    """host_states / host_obs: pinned host tensors (or addresses); the rest device (totals fp64)."""
    _check(load_library().same_stream_pass_ema(ctx.handle, _ptr(_st(ctx, host_states, m, host_ld, "host_states")), _ptr(host_obs), int(host_ld),
                                               int(n_cols), int(nb), int(m), _ptr(cpts), _ptr(totals),
                                               float(decay), int(seed), int(pass_id), int(flags), _ptr(slots),
                                               _ptr(workspace), _stream(stream)))


def same_grow_replicas(ctx, states, m, dst, m2, ld, stream=None):
    _check(load_library().same_grow_replicas(ctx.handle, _ptr(_st(ctx, states, m, ld)), int(m), _ptr(_st(ctx, dst, m2, ld, "dst")), int(m2), int(ld),
                                             _stream(stream)))


def same_debug_thresholds(ctx, cpts=None, workspace=None, stream=None):
    """(node_off [n] int64, node_kt [n] int32, tables) -- the threshold tables
    the sweep reads for cpts, as a uint32 tensor on cpts' device (None when
    cpts is None: layout only)."""
    n = ctx.n_nodes
    off = np.zeros(n, dtype=np.int64)
    kt = np.zeros(n, dtype=np.int32)
    words = C.c_int64()
    L = load_library()
    _check(L.same_debug_thresholds(ctx.handle, None, off.ctypes.data, kt.ctypes.data, C.byref(words), None,
                                   None, None))
    if cpts is None:
        return off, kt, None
    import torch
    out = torch.zeros(max(int(words.value), 1), dtype=torch.int32, device=cpts.device)
    if int(words.value) > 0:
        _check(L.same_debug_thresholds(ctx.handle, _ptr(cpts), off.ctypes.data, kt.ctypes.data, C.byref(words),
                                       _ptr(out), _ptr(workspace), _stream(stream)))
    return off, kt, out


def same_stream_compact_layout(ctx, obs_dev, ld_dev, n_cols, nb, m, workspace, stream=None):
    """(lat_off int64 numpy [M*n + 1], slot bytes) of the compact host layout."""
    M = (int(n_cols) + int(nb) - 1) // int(nb)
    off = np.zeros(M * ctx.n_nodes + 1, dtype=np.int64)
    sz = C.c_size_t()
    _check(load_library().same_stream_compact_layout(ctx.handle, _ptr(obs_dev), int(ld_dev), int(n_cols), int(nb),
                                                     int(m), off.ctypes.data, C.byref(sz), _ptr(workspace),
                                                     _stream(stream)))
    return off, int(sz.value)


def same_stream_pass_compact(ctx, lat_host, lat_off, obs_dev, data_dev, ld_dev, n_cols, nb, m, cpts, mb_counts, totals,
                             seed, pass_id, flags, slots, workspace, stream=None):
    """lat_host: pinned host tensor of the compact latent states; lat_off: the
    layout's host offsets (numpy int64); obs_dev, data_dev and the rest on the
    device."""
    off = np.ascontiguousarray(lat_off, dtype=np.int64)
    _check(load_library().same_stream_pass_compact(ctx.handle, _ptr(lat_host), off.ctypes.data, _ptr(obs_dev),
                                                   _ptr(data_dev), int(ld_dev), int(n_cols), int(nb), int(m),
                                                   _ptr(cpts), _ptr(mb_counts), _ptr(totals), int(seed), int(pass_id),
                                                   int(flags), _ptr(slots), _ptr(workspace), _stream(stream)))
