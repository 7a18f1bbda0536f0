// C ABI of libsame (declared in include/same.h): argument validation, the
// per-device structure tables, the workspace layout and the launch sequence of
// each entry point.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/same.h"
#include "graph.hpp"
#include "launch.hpp"

namespace {

thread_local std::string g_last_error;

int set_error(int code, const std::string &msg) {
    g_last_error = msg;
    return code;
}

constexpr size_t kAlign = 256;
constexpr int64_t kCompactChunkCols = 1024;  // columns per block of the compact-state kernels

inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// States are stored as replica quads, [n][mq][ld][4] with mq = ceil(m / 4):
// one node's block holds mq * ld * 4 states.
inline int64_t replica_quads(int32_t m) { return ((int64_t)m + 3) / 4; }
// quad_bytes: 2, 4 or 8 (4-, 8- or 16-bit states)
inline double node_state_bytes(int32_t m, int64_t ld, int32_t quad_bytes) {
    return (double)replica_quads(m) * (double)ld * (double)quad_bytes;
}

}  // namespace

// Copy streams and events of the out-of-core passes, per device.
struct StreamRes {
    int device = -1;
    hipStream_t up = nullptr, down = nullptr;
    hipEvent_t ev_up[2] = {nullptr, nullptr}, ev_comp[2] = {nullptr, nullptr},
               ev_down[2] = {nullptr, nullptr};
    bool slot_used[2] = {false, false};
    // sweeps: a colour's global-table launch runs on `side`, beside the
    // colour's other launches on the caller's stream (fork / join events)
    hipStream_t side = nullptr;
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
};

// Optional per-launch timing of the sweep kernels (same_kernel_timing).
struct KernelTiming {
    bool on = false;
    struct Rec {
        int32_t klass, launches;
        hipEvent_t start, end;
        double node_samples;  // (node, column, replica) slots the launch covers
    };
    std::vector<Rec> pending;
    double ms[same::kLaunchClasses] = {};
    int64_t launches[same::kLaunchClasses] = {};
    double node_samples[same::kLaunchClasses] = {};
    // colour phases: from before a colour's first launch to after its last
    // (joined) launch, on the caller's stream; records with klass < 0
    double phase_ms = 0.0;
    int64_t phases = 0;
};

struct same_ctx {
    same::Compiled g;
    KernelTiming timing;
    double alpha = 1.0;
    std::vector<same::DeviceTables> dev;  // indexed by device ordinal
    std::vector<StreamRes> sres;          // indexed by device ordinal
    std::mutex mu;
    // workspace layout
    size_t ws_table = 0, ws_cond = 0, ws_counts = 0, ws_gamma = 0, ws_total = 0;
    double tile_bytes = 0.0;  // 0: one tile (the whole minibatch)
};

namespace {

template <typename T>
hipError_t upload(T **dst, const std::vector<T> &src) {
    if (src.empty()) {
        *dst = nullptr;
        return hipSuccess;
    }
    hipError_t e = hipMalloc((void **)dst, src.size() * sizeof(T));
    if (e != hipSuccess) return e;
    return hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
}

void free_tables(same::DeviceTables &t) {
    if (t.device < 0) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(t.device);
    void *ptrs[] = {t.desc, t.desc_off, t.order, t.cdesc, t.cdesc_off, t.cwork, t.segs, t.blk_seg,
                    t.blk_first, t.row_off, t.row_k, t.cprog, t.cprog_off, t.cblk_prog, t.cblk_first};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);
    if (cur >= 0) (void)hipSetDevice(cur);
    t = same::DeviceTables();
}

// Device tables of the current device, uploaded on first use (synchronous).
int tables_for_current_device(same_ctx *ctx, same::DeviceTables **out) {
    int device = -1;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return set_error(SAME_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    std::lock_guard<std::mutex> lock(ctx->mu);
    if ((int)ctx->dev.size() <= device) ctx->dev.resize(device + 1);
    same::DeviceTables &t = ctx->dev[device];
    if (t.device == device) {
        *out = &t;
        return SAME_OK;
    }
    const same::Compiled &g = ctx->g;
    // table-build block map: each segment gets ceil(n_groups / 256) blocks
    std::vector<int32_t> blk_seg, blk_first;
    for (size_t s = 0; s < g.segments.size(); ++s)
        for (int32_t f = 0; f < g.segments[s].n_groups; f += 256) {
            blk_seg.push_back((int32_t)s);
            blk_first.push_back(f);
        }
    std::vector<int32_t> cblk_prog, cblk_first;
    for (size_t t2 = 0; t2 < g.cprog_off.size(); ++t2) {
        const int32_t ncfg = g.cprog[g.cprog_off[t2] + 3];
        for (int32_t f = 0; f < ncfg; f += 256) {
            cblk_prog.push_back((int32_t)t2);
            cblk_first.push_back(f);
        }
    }
    same::DeviceTables nt;
    nt.device = device;
    nt.n_build_blocks = (int32_t)blk_seg.size();
    nt.n_cond_blocks = (int32_t)cblk_prog.size();
    hipError_t r = hipSuccess;
    if (r == hipSuccess) r = upload(&nt.desc, g.desc);
    if (r == hipSuccess) r = upload(&nt.desc_off, g.desc_off);
    if (r == hipSuccess) r = upload(&nt.order, g.order);
    if (r == hipSuccess) r = upload(&nt.cdesc, g.cdesc);
    if (r == hipSuccess) r = upload(&nt.cdesc_off, g.cdesc_off);
    if (r == hipSuccess) r = upload(&nt.cwork, g.cwork);
    nt.n_cwork = (int32_t)(g.cwork.size() / 2);
    if (r == hipSuccess) r = upload(&nt.segs, g.segments);
    if (r == hipSuccess) r = upload(&nt.blk_seg, blk_seg);
    if (r == hipSuccess) r = upload(&nt.blk_first, blk_first);
    if (r == hipSuccess) r = upload(&nt.row_off, g.row_off);
    if (r == hipSuccess) r = upload(&nt.row_k, g.row_k);
    if (r == hipSuccess) r = upload(&nt.cprog, g.cprog);
    if (r == hipSuccess) r = upload(&nt.cprog_off, g.cprog_off);
    if (r == hipSuccess) r = upload(&nt.cblk_prog, cblk_prog);
    if (r == hipSuccess) r = upload(&nt.cblk_first, cblk_first);
    if (r != hipSuccess) {
        free_tables(nt);
        return set_error(r == hipErrorOutOfMemory ? SAME_ENOMEM : SAME_EHIP,
                         std::string("uploading structure tables: ") + hipGetErrorString(r));
    }
    t = nt;
    *out = &t;
    return SAME_OK;
}

void free_stream_res(StreamRes &r) {
    if (r.device < 0) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(r.device);
    if (r.up) (void)hipStreamSynchronize(r.up);
    if (r.down) (void)hipStreamSynchronize(r.down);
    if (r.side) (void)hipStreamSynchronize(r.side);
    if (r.ev_fork) (void)hipEventDestroy(r.ev_fork);
    if (r.ev_join) (void)hipEventDestroy(r.ev_join);
    if (r.side) (void)hipStreamDestroy(r.side);
    for (int i = 0; i < 2; ++i) {
        if (r.ev_up[i]) (void)hipEventDestroy(r.ev_up[i]);
        if (r.ev_comp[i]) (void)hipEventDestroy(r.ev_comp[i]);
        if (r.ev_down[i]) (void)hipEventDestroy(r.ev_down[i]);
    }
    if (r.up) (void)hipStreamDestroy(r.up);
    if (r.down) (void)hipStreamDestroy(r.down);
    if (cur >= 0) (void)hipSetDevice(cur);
    r = StreamRes();
}

int stream_res_for_current_device(same_ctx *ctx, StreamRes **out) {
    int device = -1;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return set_error(SAME_EHIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
    std::lock_guard<std::mutex> lock(ctx->mu);
    if ((int)ctx->sres.size() <= device) ctx->sres.resize(device + 1);
    StreamRes &r = ctx->sres[device];
    if (r.device == device) {
        *out = &r;
        return SAME_OK;
    }
    StreamRes nr;
    nr.device = device;
    hipError_t h = hipStreamCreateWithFlags(&nr.up, hipStreamNonBlocking);
    if (h == hipSuccess) h = hipStreamCreateWithFlags(&nr.down, hipStreamNonBlocking);
    if (h == hipSuccess) h = hipStreamCreateWithFlags(&nr.side, hipStreamNonBlocking);
    if (h == hipSuccess) h = hipEventCreateWithFlags(&nr.ev_fork, hipEventDisableTiming);
    if (h == hipSuccess) h = hipEventCreateWithFlags(&nr.ev_join, hipEventDisableTiming);
    for (int i = 0; i < 2 && h == hipSuccess; ++i) {
        h = hipEventCreateWithFlags(&nr.ev_up[i], hipEventDisableTiming);
        if (h == hipSuccess) h = hipEventCreateWithFlags(&nr.ev_comp[i], hipEventDisableTiming);
        if (h == hipSuccess) h = hipEventCreateWithFlags(&nr.ev_down[i], hipEventDisableTiming);
    }
    if (h != hipSuccess) {
        free_stream_res(nr);
        return set_error(SAME_EHIP, std::string("creating copy streams: ") + hipGetErrorString(h));
    }
    r = nr;
    *out = &r;
    return SAME_OK;
}

int check_hip(hipError_t e, const char *what) {
    if (e == hipSuccess) return SAME_OK;
    return set_error(SAME_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

int check_minibatch(const same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld) {
    if (!ctx) return set_error(SAME_EINVAL, "ctx is null");
    if (!states) return set_error(SAME_EINVAL, "states is null");
    if (m < 1 || m > 65535) return set_error(SAME_EINVAL, "m must be in [1, 65535]");
    if (n_cols < 0 || ld < n_cols) return set_error(SAME_EINVAL, "need 0 <= n_cols <= ld");
    if (ld % 4 != 0) return set_error(SAME_EALIGN, "ld must be a multiple of 4");
    if (!aligned(states, (size_t)ctx->g.quad_bytes))
        return set_error(SAME_EALIGN, "states must be aligned to a state quad");
    if (node_state_bytes(m, ld, ctx->g.quad_bytes) >= 2147483648.0)
        return set_error(SAME_ESIZE, "one node's state quads (4 * ceil(m / 4) * ld states) must stay below 2^31 bytes");
    if ((double)ctx->g.n * node_state_bytes(m, ld, ctx->g.quad_bytes) > 9.0e18)
        return set_error(SAME_ESIZE, "states array too large");
    return SAME_OK;
}

// Column tiles (optional, same_options_t.tile_bytes): a sweep visits its
// colour groups tile by tile, so that one tile's states can stay in the
// last-level cache while every colour group re-reads them; counts of the tile
// follow while it is still there.  Measured on MI355X the smaller launches
// cost more than the cache saves, so the default is one tile.
int64_t tile_cols(const same_ctx *ctx, int32_t m, int64_t n_cols) {
    if (ctx->tile_bytes <= 0.0) return n_cols;
    const double per_col = (double)ctx->g.n * ((double)replica_quads(m) * ctx->g.quad_bytes + 1.0);
    int64_t t = (int64_t)(ctx->tile_bytes / per_col) / 1024 * 1024;
    if (t < 1024) t = 1024;
    return t >= n_cols ? n_cols : t;
}

int check_sweep_args(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts, int32_t m,
                     int64_t n_cols, int64_t ld, int64_t col_offset, int64_t win_begin, int64_t win,
                     float *probs, void *workspace) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!obs || !cpts || !workspace) return set_error(SAME_EINVAL, "obs, cpts and workspace must be non-null");
    if (col_offset < 0 || col_offset % 4 != 0)
        return set_error(SAME_EALIGN, "col_offset must be a non-negative multiple of 4");
    if (col_offset + n_cols > ((int64_t)1 << 32))
        return set_error(SAME_ESIZE, "global column index exceeds the Philox counter range (2^32 columns)");
    if (!aligned(obs, 4)) return set_error(SAME_EALIGN, "obs must be 4-byte aligned");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    if (win > 0) {
        if (!probs) return set_error(SAME_EINVAL, "probs is null");
        if (win_begin < 0) return set_error(SAME_EINVAL, "win_begin must be >= 0");
    }
    return SAME_OK;
}

// Builds this call's tables from cpts (and clears zero[0 .. zero_count) in
// the same launch) and fills the sweep parameters.
int prepare_sweep(same_ctx *ctx, same::DeviceTables *t, void *states, const uint8_t *obs,
                  const float *cpts, int32_t m, int64_t n_cols, int64_t ld, int64_t col_offset,
                  uint64_t seed, uint32_t sweep_id, int64_t win_begin, int64_t win, float *probs,
                  void *workspace, hipStream_t s, same::SweepParams &P, int32_t *zero = nullptr,
                  int64_t zero_count = 0) {
    float *table = (float *)((char *)workspace + ctx->ws_table);
    uint32_t *cond = (uint32_t *)((char *)workspace + ctx->ws_cond);
    int rc = check_hip(same::launch_prepare(*t, cpts, table, cond, zero, zero_count, s), "table build launch");
    if (rc) return rc;
    P = same::SweepParams{};
    P.desc = t->desc;
    P.desc_off = t->desc_off;
    P.order = t->order;
    P.table = table;
    P.cond = cond;
    P.states = states;
    P.obs = obs;
    P.m = m;
    P.n_cols = n_cols;
    P.ld = ld;
    P.col_offset = col_offset;
    P.key0 = (uint32_t)seed;
    P.key1 = (uint32_t)(seed >> 32);
    P.sweep_id = sweep_id;
    P.win_begin = win_begin;
    P.win = win > 0 ? win : 0;
    P.probs = probs;
    P.max_card = ctx->g.max_card;
    return SAME_OK;
}

// All colour groups over columns [t0, t0 + nt) of the minibatch described by P.
int sweep_tile(same_ctx *ctx, const same::SweepParams &P0, int64_t t0, int64_t nt, hipStream_t s) {
    const same::Compiled &g = ctx->g;
    same::SweepParams P = P0;
    P.states = (char *)P0.states + t0 * g.quad_bytes;  // column t0 of every quad row
    P.obs = P0.obs + t0;
    P.n_cols = nt;
    P.col_offset = P0.col_offset + t0;
    P.win_begin = P0.win_begin - t0;
    StreamRes *sr = nullptr;
    int rc = stream_res_for_current_device(ctx, &sr);
    if (rc) return rc;
    const int32_t L = same::kLaunchClasses;
    for (int32_t c = 0; c < g.n_colors; ++c) {
        P.reverse = c & 1;
        // the nodes of one colour are independent: the global-table launch
        // (bound by the texture addresser) runs beside the LDS-bound one
        const int32_t b1 = g.launch[c * (L + 1) + 1], e1 = g.launch[c * (L + 1) + 2];
        const bool fork = e1 > b1 && nt > 0;
        KernelTiming::Rec phase{-1, 1, nullptr, nullptr, 0.0};
        const bool phase_timed = ctx->timing.on && nt > 0 && g.launch[c * (L + 1) + L] > g.launch[c * (L + 1)];
        if (phase_timed) {
            rc = check_hip(hipEventCreate(&phase.start), "hipEventCreate");
            if (!rc) rc = check_hip(hipEventCreate(&phase.end), "hipEventCreate");
            if (!rc) rc = check_hip(hipEventRecord(phase.start, s), "hipEventRecord");
            if (rc) return rc;
        }
        if (fork) {
            rc = check_hip(hipEventRecord(sr->ev_fork, s), "hipEventRecord");
            if (!rc) rc = check_hip(hipStreamWaitEvent(sr->side, sr->ev_fork, 0), "hipStreamWaitEvent");
            if (rc) return rc;
        }
        for (int32_t k = 0; k < L; ++k) {
            const int32_t b = g.launch[c * (L + 1) + k], e = g.launch[c * (L + 1) + k + 1];
            hipStream_t ls = (fork && k == 1) ? sr->side : s;
            KernelTiming::Rec rec{k, 1, nullptr, nullptr, (double)(e - b) * (double)nt * (double)P.m};
            const bool timed = ctx->timing.on && e > b && nt > 0;
            if (timed) {
                rc = check_hip(hipEventCreate(&rec.start), "hipEventCreate");
                if (!rc) rc = check_hip(hipEventCreate(&rec.end), "hipEventCreate");
                if (!rc) rc = check_hip(hipEventRecord(rec.start, ls), "hipEventRecord");
                if (rc) return rc;
            }
            rc = check_hip(same::launch_sweep(P, b, e - b, k, g.launch_lds[c * L + k], g.state_bits, ls),
                           "sweep launch");
            if (rc) return rc;
            if (timed) {
                rc = check_hip(hipEventRecord(rec.end, ls), "hipEventRecord");
                if (rc) return rc;
                ctx->timing.pending.push_back(rec);
            }
        }
        if (fork) {
            rc = check_hip(hipEventRecord(sr->ev_join, sr->side), "hipEventRecord");
            if (!rc) rc = check_hip(hipStreamWaitEvent(s, sr->ev_join, 0), "hipStreamWaitEvent");
            if (rc) return rc;
        }
        if (phase_timed) {
            rc = check_hip(hipEventRecord(phase.end, s), "hipEventRecord");
            if (rc) return rc;
            ctx->timing.pending.push_back(phase);
        }
    }
    return SAME_OK;
}

// Folds the finished timing records into the totals (waits for each).
int collect_timing(same_ctx *ctx) {
    KernelTiming &t = ctx->timing;
    int rc = SAME_OK;
    for (const KernelTiming::Rec &r : t.pending) {
        float ms = 0.f;
        if (!rc) rc = check_hip(hipEventSynchronize(r.end), "hipEventSynchronize");
        if (!rc) rc = check_hip(hipEventElapsedTime(&ms, r.start, r.end), "hipEventElapsedTime");
        if (!rc && r.klass < 0) {
            t.phase_ms += ms;
            t.phases += r.launches;
        } else if (!rc) {
            t.ms[r.klass] += ms;
            t.launches[r.klass] += r.launches;
            t.node_samples[r.klass] += r.node_samples;
        }
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.end);
    }
    t.pending.clear();
    return rc;
}

int do_sweep(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts, int32_t m,
             int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed, uint32_t sweep_id,
             int64_t win_begin, int64_t win, float *probs, void *workspace, void *stream) {
    int rc = check_sweep_args(ctx, states, obs, cpts, m, n_cols, ld, col_offset, win_begin, win, probs,
                              workspace);
    if (rc) return rc;
    if (n_cols == 0) return SAME_OK;
    same::DeviceTables *t = nullptr;
    rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    same::SweepParams P;
    rc = prepare_sweep(ctx, t, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, win_begin, win,
                       probs, workspace, s, P);
    if (rc) return rc;
    const int64_t T = tile_cols(ctx, m, n_cols);
    for (int64_t t0 = 0; t0 < n_cols; t0 += T) {
        rc = sweep_tile(ctx, P, t0, n_cols - t0 < T ? n_cols - t0 : T, s);
        if (rc) return rc;
    }
    return SAME_OK;
}

// Sweep, counts with the moving sum, and the Dirichlet resample of one
// minibatch, tile by tile for the sweep and counts.
// ids (nullable, device): the sweep and update ids are read there at launch
// time instead of sweep_id and update_id.
int do_step(same_ctx *ctx, void *states, const uint8_t *obs, float *cpts, int32_t m, int64_t n_cols,
            int64_t ld, int64_t col_offset, uint64_t seed, uint32_t sweep_id, int32_t *mb_counts,
            int32_t *totals, uint32_t update_id, void *workspace, void *stream,
            const uint32_t *ids = nullptr) {
    int rc = check_sweep_args(ctx, states, obs, cpts, m, n_cols, ld, col_offset, 0, 0, nullptr, workspace);
    if (rc) return rc;
    if (!mb_counts || !totals) return set_error(SAME_EINVAL, "mb_counts and totals must be non-null");
    if ((double)n_cols * (double)m >= 2147483648.0)
        return set_error(SAME_ESIZE, "n_cols * m must stay below 2^31");
    same::DeviceTables *t = nullptr;
    rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    const int64_t total = ctx->g.off[ctx->g.n];
    int32_t *newc = (int32_t *)((char *)workspace + ctx->ws_counts);
    same::SweepParams P;
    rc = prepare_sweep(ctx, t, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, 0, 0, nullptr,
                       workspace, s, P, newc, total);
    if (rc) return rc;
    P.ids = ids;
    const int64_t T = tile_cols(ctx, m, n_cols);
    for (int64_t t0 = 0; t0 < n_cols; t0 += T) {
        const int64_t nt = n_cols - t0 < T ? n_cols - t0 : T;
        rc = sweep_tile(ctx, P, t0, nt, s);
        if (rc) return rc;
        rc = check_hip(same::launch_counts(*t, states, ctx->g.state_bits, m, t0, nt, ld, newc, s),
                       "count launch");
        if (rc) return rc;
    }
    // the moving sum and the Dirichlet resample (same_sample_cpts), with the
    // moving sum fused into the Gamma launch
    double *gv = (double *)((char *)workspace + ctx->ws_gamma);
    rc = check_hip(same::launch_moving_sum_gamma(newc, mb_counts, totals, ctx->alpha, (uint32_t)seed,
                                                 (uint32_t)(seed >> 32), update_id, ids, gv, total, s),
                   "moving-sum and gamma launch");
    if (rc) return rc;
    return check_hip(same::launch_normalize(*t, gv, cpts, ctx->g.n_rows, s), "normalize launch");
}

// Device slot geometry of the out-of-core passes.
struct SlotGeom {
    int64_t ld = 0;          // leading dimension of a slot (columns)
    size_t states = 0;       // bytes of the states part
    size_t bytes = 0;        // bytes of one slot (states + obs)
};

SlotGeom slot_geom(const same_ctx *ctx, int32_t m, int64_t nb) {
    SlotGeom s;
    s.ld = (nb + 63) / 64 * 64;
    s.states = align_up((size_t)ctx->g.n * (size_t)node_state_bytes(m, s.ld, ctx->g.quad_bytes));
    s.bytes = s.states + align_up((size_t)ctx->g.n * (size_t)s.ld);
    return s;
}

}  // namespace

extern "C" {

const char *same_last_error(void) { return g_last_error.c_str(); }

int same_create(int32_t n_nodes, const int32_t *parent_ptr, const int32_t *parent_idx,
                const int32_t *card, double dirichlet_prior, same_ctx **out) {
    return same_create_ex(n_nodes, parent_ptr, parent_idx, card, dirichlet_prior, nullptr, out);
}

int same_create_ex(int32_t n_nodes, const int32_t *parent_ptr, const int32_t *parent_idx,
                   const int32_t *card, double dirichlet_prior, const same_options_t *opts,
                   same_ctx **out) {
    if (!out) return set_error(SAME_EINVAL, "out is null");
    int64_t table_limit = same::kDefaultTableLimit;
    if (opts && opts->table_limit >= 0) table_limit = opts->table_limit;
    if (opts && opts->table_limit < -1) return set_error(SAME_EINVAL, "table_limit must be >= -1");
    if (opts && opts->tile_bytes < 0) return set_error(SAME_EINVAL, "tile_bytes must be >= 0");
    int64_t lds_limit = same::kDefaultLdsBytes;
    if (opts && opts->lds_limit >= 0) lds_limit = opts->lds_limit;
    if (opts && (opts->lds_limit < -1 || opts->lds_limit > same::kLdsBudgetBytes))
        return set_error(SAME_EINVAL, "lds_limit must be -1 or in [0, 32768]");
    if (opts && opts->packed_indices != 0 && opts->packed_indices != 1)
        return set_error(SAME_EINVAL, "packed_indices must be 0 or 1");
    const bool packed = !opts || opts->packed_indices != 0;
    if (opts && opts->first_fit_colours != 0 && opts->first_fit_colours != 1)
        return set_error(SAME_EINVAL, "first_fit_colours must be 0 or 1");
    const bool balance = !opts || opts->first_fit_colours == 0;
    if (opts && opts->state_bits != 0 && opts->state_bits != 4)
        return set_error(SAME_EINVAL, "state_bits must be 0 or 4");
    const int32_t state_bits = opts ? opts->state_bits : 0;
    *out = nullptr;
    if (!(dirichlet_prior > 0.0)) return set_error(SAME_EINVAL, "dirichlet_prior must be > 0");
    same_ctx *ctx = new (std::nothrow) same_ctx();
    if (!ctx) return set_error(SAME_ENOMEM, "out of host memory");
    std::string err;
    int rc;
    try {
        rc = same::compile_graph(n_nodes, parent_ptr, parent_idx, card, ctx->g, err, table_limit,
                                 lds_limit, packed, balance, state_bits);
    } catch (const std::bad_alloc &) {
        rc = SAME_ENOMEM;
        err = "out of host memory";
    }
    if (rc) {
        delete ctx;
        return set_error(rc, err);
    }
    ctx->alpha = dirichlet_prior;
    if (opts && opts->tile_bytes > 0) ctx->tile_bytes = (double)opts->tile_bytes;
    ctx->ws_table = 0;
    ctx->ws_cond = align_up(ctx->ws_table + (size_t)ctx->g.table_floats * sizeof(float));
    ctx->ws_counts = align_up(ctx->ws_cond + (size_t)ctx->g.cond_words * sizeof(uint32_t));
    ctx->ws_gamma = align_up(ctx->ws_counts + (size_t)ctx->g.off[n_nodes] * sizeof(int32_t));
    ctx->ws_total = align_up(ctx->ws_gamma + (size_t)ctx->g.off[n_nodes] * sizeof(double));
    *out = ctx;
    return SAME_OK;
}

void same_destroy(same_ctx *ctx) {
    if (!ctx) return;
    for (auto &r : ctx->timing.pending) {
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.end);
    }
    for (auto &r : ctx->sres) free_stream_res(r);
    for (auto &t : ctx->dev) free_tables(t);
    delete ctx;
}

int same_layout(const same_ctx *ctx, same_layout_t *out, int64_t *cpt_off, int32_t *color) {
    if (!ctx || !out) return set_error(SAME_EINVAL, "ctx and out must be non-null");
    const same::Compiled &g = ctx->g;
    out->n_nodes = g.n;
    out->n_colors = g.n_colors;
    out->cpt_total = g.off[g.n];
    out->n_rows = g.n_rows;
    out->state_bytes = g.state_bytes;
    out->state_bits = g.state_bits;
    out->max_card = g.max_card;
    const int32_t L = same::kLaunchClasses;
    int32_t launches = 0;
    for (int32_t c = 0; c < g.n_colors; ++c)
        for (int32_t k = 0; k < L; ++k) {
            const int32_t cnt = g.launch[c * (L + 1) + k + 1] - g.launch[c * (L + 1) + k];
            launches += cnt > 0 ? 1 : 0;
        }
    out->sweep_launches = launches;
    int32_t tn = 0;
    for (int32_t i = 0; i < g.n; ++i) tn += g.mode[i] == same::kModeTable ? 1 : 0;
    out->table_nodes = tn;
    if (cpt_off) std::memcpy(cpt_off, g.off.data(), sizeof(int64_t) * (g.n + 1));
    if (color) std::memcpy(color, g.color.data(), sizeof(int32_t) * g.n);
    return SAME_OK;
}

int same_workspace_size(const same_ctx *ctx, size_t *bytes) {
    if (!ctx || !bytes) return set_error(SAME_EINVAL, "ctx and bytes must be non-null");
    *bytes = ctx->ws_total;
    return SAME_OK;
}

int same_sweep(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts, int32_t m,
               int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed, uint32_t sweep_id,
               void *workspace, void *stream) {
    return do_sweep(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, 0, 0, nullptr,
                    workspace, stream);
}

int same_sweep_debug(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts,
                     int32_t m, int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed,
                     uint32_t sweep_id, int64_t win_begin, int64_t win, float *probs,
                     void *workspace, void *stream) {
    if (win <= 0) return set_error(SAME_EINVAL, "win must be positive");
    return do_sweep(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, win_begin, win,
                    probs, workspace, stream);
}

int same_debug_thresholds(same_ctx *ctx, const float *cpts, int64_t *node_off, int32_t *node_kt,
                          int64_t *words, uint32_t *cond_out, void *workspace, void *stream) {
    if (!ctx || !node_off || !node_kt || !words)
        return set_error(SAME_EINVAL, "ctx, node_off, node_kt and words must be non-null");
    const same::Compiled &g = ctx->g;
    for (int32_t i = 0; i < g.n; ++i) {
        const int32_t *d = g.desc.data() + g.desc_off[i];
        const bool tab = g.mode[i] == same::kModeTable;
        node_off[i] = tab ? (int64_t)d[5] : -1;
        node_kt[i] = tab ? d[7] : 0;
    }
    *words = g.cond_words;
    if (!cond_out || g.cond_words == 0) return SAME_OK;
    if (!cpts || !workspace) return set_error(SAME_EINVAL, "cpts and workspace must be non-null");
    if (!aligned(cond_out, 4)) return set_error(SAME_EALIGN, "cond_out must be 4-byte aligned");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    same::DeviceTables *t = nullptr;
    int rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    uint32_t *cond = (uint32_t *)((char *)workspace + ctx->ws_cond);
    rc = check_hip(same::launch_build_thresholds(*t, cpts, cond, s), "threshold build launch");
    if (rc) return rc;
    return check_hip(hipMemcpyAsync(cond_out, cond, (size_t)g.cond_words * sizeof(uint32_t),
                                    hipMemcpyDeviceToDevice, s),
                     "threshold copy");
}

int same_counts(same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld,
                int32_t *mb_counts, int32_t *totals, void *workspace, void *stream) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!mb_counts || !workspace) return set_error(SAME_EINVAL, "mb_counts and workspace must be non-null");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    if ((double)n_cols * (double)m >= 2147483648.0)
        return set_error(SAME_ESIZE, "n_cols * m must stay below 2^31");
    same::DeviceTables *t = nullptr;
    rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    const int64_t total = ctx->g.off[ctx->g.n];
    int32_t *newc = (int32_t *)((char *)workspace + ctx->ws_counts);
    rc = check_hip(same::launch_fill_zero(newc, total, s), "count clear launch");
    if (rc) return rc;
    rc = check_hip(same::launch_counts(*t, states, ctx->g.state_bits, m, 0, n_cols, ld, newc, s),
                   "count launch");
    if (rc) return rc;
    return check_hip(same::launch_moving_sum(newc, mb_counts, totals, total, s), "moving-sum launch");
}

int same_sample_cpts(same_ctx *ctx, const int32_t *totals, float *cpts_out, uint64_t seed,
                     uint32_t update_id, void *workspace, void *stream) {
    if (!ctx || !totals || !cpts_out || !workspace)
        return set_error(SAME_EINVAL, "ctx, totals, cpts_out and workspace must be non-null");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    same::DeviceTables *t = nullptr;
    int rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    const int64_t total = ctx->g.off[ctx->g.n];
    double *gv = (double *)((char *)workspace + ctx->ws_gamma);
    rc = check_hip(same::launch_gamma(totals, ctx->alpha, (uint32_t)seed, (uint32_t)(seed >> 32), update_id,
                                      nullptr, gv, total, s),
                   "gamma launch");
    if (rc) return rc;
    return check_hip(same::launch_normalize(*t, gv, cpts_out, ctx->g.n_rows, s), "normalize launch");
}

int same_sweep_plan(const same_ctx *ctx, int32_t m, int64_t n_cols, int64_t *tile_cols_out,
                    int32_t *launches) {
    if (!ctx || !tile_cols_out || !launches) return set_error(SAME_EINVAL, "null pointer argument");
    if (m < 1 || n_cols < 0) return set_error(SAME_EINVAL, "need m >= 1 and n_cols >= 0");
    if (n_cols == 0) {
        *tile_cols_out = 0;
        *launches = 0;
        return SAME_OK;
    }
    const int64_t T = tile_cols(ctx, m, n_cols);
    same_layout_t lay;
    same_layout(ctx, &lay, nullptr, nullptr);
    *tile_cols_out = T;
    *launches = (int32_t)(((n_cols + T - 1) / T) * lay.sweep_launches);
    return SAME_OK;
}

int same_step(same_ctx *ctx, void *states, const uint8_t *obs, float *cpts, int32_t m,
              int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed, uint32_t sweep_id,
              int32_t *mb_counts, int32_t *totals, uint32_t update_id, void *workspace,
              void *stream) {
    return do_step(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id, mb_counts, totals,
                   update_id, workspace, stream);
}

int same_stream_slots_size(const same_ctx *ctx, int32_t m, int64_t nb, size_t *bytes) {
    if (!ctx || !bytes) return set_error(SAME_EINVAL, "ctx and bytes must be non-null");
    if (m < 1 || m > 65535 || nb < 4) return set_error(SAME_EINVAL, "need 1 <= m <= 65535 and nb >= 4");
    *bytes = 2 * slot_geom(ctx, m, nb).bytes;
    return SAME_OK;
}

}  // extern "C"

namespace {

// One out-of-core pass (layout and overlap as documented for same_stream_pass):
// per minibatch b the upload, then compute(b, device states, device obs,
// columns, first column) on `stream`, then (with download) the copy back.
template <typename F>
int stream_pass_impl(same_ctx *ctx, void *host_states, const uint8_t *host_obs, int64_t host_ld,
                     int64_t n_cols, int64_t nb, int32_t m, void *slots, void *stream, bool download,
                     F &&compute) {
    const SlotGeom sg = slot_geom(ctx, m, nb);
    StreamRes *sr = nullptr;
    int rc = stream_res_for_current_device(ctx, &sr);
    if (rc) return rc;
    hipStream_t cs = (hipStream_t)stream;
    const size_t sb = (size_t)ctx->g.quad_bytes;  // bytes of one column of a quad row
    const int64_t rows = (int64_t)ctx->g.n * replica_quads(m);
    const int64_t M = (n_cols + nb - 1) / nb;
    for (int64_t b = 0; b < M; ++b) {
        const int s = (int)(b & 1);
        const int64_t c0 = b * nb;
        const int64_t cols = n_cols - c0 < nb ? n_cols - c0 : nb;
        char *slot = (char *)slots + s * sg.bytes;
        void *d_states = slot;
        uint8_t *d_obs = (uint8_t *)(slot + sg.states);
        // upload (after the slot's previous minibatch has left it)
        if (sr->slot_used[s] && (rc = check_hip(hipStreamWaitEvent(sr->up, sr->ev_down[s], 0), "wait")))
            return rc;
        rc = check_hip(hipMemcpy2DAsync(d_states, sg.ld * sb, (char *)host_states + c0 * sb, host_ld * sb,
                                        cols * sb, rows, hipMemcpyHostToDevice, sr->up),
                       "state upload");
        if (!rc)
            rc = check_hip(hipMemcpy2DAsync(d_obs, sg.ld, host_obs + c0, host_ld, cols, ctx->g.n,
                                            hipMemcpyHostToDevice, sr->up),
                           "obs upload");
        if (!rc) rc = check_hip(hipEventRecord(sr->ev_up[s], sr->up), "event");
        if (!rc) rc = check_hip(hipStreamWaitEvent(cs, sr->ev_up[s], 0), "wait");
        if (rc) return rc;
        rc = compute(b, d_states, d_obs, cols, c0, sg.ld);
        if (rc) return rc;
        rc = check_hip(hipEventRecord(sr->ev_comp[s], cs), "event");
        if (rc) return rc;
        if (!download) {
            rc = check_hip(hipEventRecord(sr->ev_down[s], cs), "event");
        } else {
            rc = check_hip(hipStreamWaitEvent(sr->down, sr->ev_comp[s], 0), "wait");
            if (!rc)
                rc = check_hip(hipMemcpy2DAsync((char *)host_states + c0 * sb, host_ld * sb, d_states,
                                                sg.ld * sb, cols * sb, rows, hipMemcpyDeviceToHost, sr->down),
                               "state download");
            if (!rc) rc = check_hip(hipEventRecord(sr->ev_down[s], sr->down), "event");
        }
        if (rc) return rc;
        sr->slot_used[s] = true;
    }
    // the caller's stream completes only after the last downloads
    for (int s = 0; s < 2; ++s)
        if (sr->slot_used[s] && (rc = check_hip(hipStreamWaitEvent(cs, sr->ev_down[s], 0), "wait")))
            return rc;
    return SAME_OK;
}

int check_stream_args(same_ctx *ctx, const void *host_states, const uint8_t *host_obs, int64_t host_ld,
                      int64_t n_cols, int64_t nb, int32_t m, const void *cpts, const void *counts,
                      const void *totals, uint32_t pass_id, int32_t flags, const void *slots,
                      const void *workspace) {
    if (!ctx) return set_error(SAME_EINVAL, "ctx is null");
    if (!host_states || !host_obs || !cpts || !counts || !totals || !slots || !workspace)
        return set_error(SAME_EINVAL, "null pointer argument");
    if (m < 1 || m > 65535) return set_error(SAME_EINVAL, "m must be in [1, 65535]");
    if (nb < 4 || nb % 4 != 0) return set_error(SAME_EALIGN, "nb must be a positive multiple of 4");
    if (n_cols < 0 || host_ld < n_cols) return set_error(SAME_EINVAL, "need 0 <= n_cols <= host_ld");
    if (flags & ~SAME_STREAM_COUNTS_ONLY) return set_error(SAME_EINVAL, "unknown flags");
    if (!aligned(slots, kAlign)) return set_error(SAME_EALIGN, "slots must be 256-byte aligned");
    const int64_t M = n_cols > 0 ? (n_cols + nb - 1) / nb : 0;
    if ((double)M * (double)pass_id + M > 4294967295.0)
        return set_error(SAME_ESIZE, "pass_id * minibatches exceeds the update-id range");
    return SAME_OK;
}

}  // namespace

extern "C" {

int same_stream_pass(same_ctx *ctx, void *host_states, const uint8_t *host_obs, int64_t host_ld,
                     int64_t n_cols, int64_t nb, int32_t m, float *cpts, int32_t *mb_counts,
                     int32_t *totals, uint64_t seed, uint32_t pass_id, int32_t flags, void *slots,
                     void *workspace, void *stream) {
    int rc = check_stream_args(ctx, host_states, host_obs, host_ld, n_cols, nb, m, cpts, mb_counts, totals,
                               pass_id, flags, slots, workspace);
    if (rc || n_cols == 0) return rc;
    const int64_t M = (n_cols + nb - 1) / nb;
    const int64_t total = ctx->g.off[ctx->g.n];
    const bool counts_only = (flags & SAME_STREAM_COUNTS_ONLY) != 0;
    return stream_pass_impl(
        ctx, host_states, host_obs, host_ld, n_cols, nb, m, slots, stream, !counts_only,
        [&](int64_t b, void *d_states, uint8_t *d_obs, int64_t cols, int64_t c0, int64_t ld) {
            int32_t *mb = mb_counts + b * total;
            if (counts_only) return same_counts(ctx, d_states, m, cols, ld, mb, totals, workspace, stream);
            return do_step(ctx, d_states, d_obs, cpts, m, cols, ld, c0, seed, pass_id, mb, totals,
                           (uint32_t)(pass_id * M + b), workspace, stream);
        });
}

int same_counts_ema(same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld, double decay,
                    double *totals, void *workspace, void *stream) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!totals || !workspace) return set_error(SAME_EINVAL, "totals and workspace must be non-null");
    if (!(decay >= 0.0 && decay <= 1.0)) return set_error(SAME_EINVAL, "decay must be in [0, 1]");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    if (!aligned(totals, 8)) return set_error(SAME_EALIGN, "totals must be 8-byte aligned");
    if ((double)n_cols * (double)m >= 2147483648.0)
        return set_error(SAME_ESIZE, "n_cols * m must stay below 2^31");
    same::DeviceTables *t = nullptr;
    rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    const int64_t total = ctx->g.off[ctx->g.n];
    int32_t *newc = (int32_t *)((char *)workspace + ctx->ws_counts);
    rc = check_hip(same::launch_fill_zero(newc, total, s), "count clear launch");
    if (rc) return rc;
    rc = check_hip(same::launch_counts(*t, states, ctx->g.state_bits, m, 0, n_cols, ld, newc, s),
                   "count launch");
    if (rc) return rc;
    return check_hip(same::launch_ema(newc, totals, decay, total, s), "moving-sum launch");
}

int same_counts_noalloc(same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld,
                        int32_t *mb_counts, int32_t *totals, void *stream) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!mb_counts) return set_error(SAME_EINVAL, "mb_counts must be non-null");
    if ((double)n_cols * (double)m >= 2147483648.0)
        return set_error(SAME_ESIZE, "n_cols * m must stay below 2^31");
    const int64_t total = ctx->g.off[ctx->g.n];
    if (total > same::kScratchCountEntries)
        return set_error(SAME_ESIZE, "cpt_total exceeds the " + std::to_string(same::kScratchCountEntries) +
                                         " entries of the allocation-free count scratch");
    int device = -1;
    rc = check_hip(hipGetDevice(&device), "hipGetDevice");
    if (rc) return rc;
    // the structure tables must already be on this device: uploading them
    // would allocate
    same::DeviceTables *t = nullptr;
    {
        std::lock_guard<std::mutex> lock(ctx->mu);
        if ((int)ctx->dev.size() > device && ctx->dev[device].device == device) t = &ctx->dev[device];
    }
    if (!t)
        return set_error(SAME_EINVAL, "the context's tables are not on this device yet: make one allocating call "
                                      "(e.g. same_counts) on it first");
    int32_t *newc = nullptr;
    rc = check_hip(same::scratch_counts(device, &newc), "hipGetSymbolAddress");
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    rc = check_hip(same::launch_fill_zero(newc, total, s), "count clear launch");
    if (rc) return rc;
    rc = check_hip(same::launch_counts(*t, states, ctx->g.state_bits, m, 0, n_cols, ld, newc, s), "count launch");
    if (rc) return rc;
    return check_hip(same::launch_moving_sum(newc, mb_counts, totals, total, s), "moving-sum launch");
}

int same_sample_cpts_ema(same_ctx *ctx, const double *totals, float *cpts_out, uint64_t seed, uint32_t update_id,
                         void *workspace, void *stream) {
    if (!ctx || !totals || !cpts_out || !workspace)
        return set_error(SAME_EINVAL, "ctx, totals, cpts_out and workspace must be non-null");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    same::DeviceTables *t = nullptr;
    int rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    hipStream_t s = (hipStream_t)stream;
    const int64_t total = ctx->g.off[ctx->g.n];
    double *gv = (double *)((char *)workspace + ctx->ws_gamma);
    rc = check_hip(same::launch_gamma(totals, ctx->alpha, (uint32_t)seed, (uint32_t)(seed >> 32), update_id,
                                      nullptr, gv, total, s),
                   "gamma launch");
    if (rc) return rc;
    return check_hip(same::launch_normalize(*t, gv, cpts_out, ctx->g.n_rows, s), "normalize launch");
}

int same_stream_pass_ema(same_ctx *ctx, void *host_states, const uint8_t *host_obs, int64_t host_ld,
                         int64_t n_cols, int64_t nb, int32_t m, float *cpts, double *totals, double decay,
                         uint64_t seed, uint32_t pass_id, int32_t flags, void *slots, void *workspace,
                         void *stream) {
    int rc = check_stream_args(ctx, host_states, host_obs, host_ld, n_cols, nb, m, cpts, totals, totals, pass_id,
                               flags, slots, workspace);
    if (rc || n_cols == 0) return rc;
    if (!(decay >= 0.0 && decay <= 1.0)) return set_error(SAME_EINVAL, "decay must be in [0, 1]");
    const int64_t M = (n_cols + nb - 1) / nb;
    const bool counts_only = (flags & SAME_STREAM_COUNTS_ONLY) != 0;
    return stream_pass_impl(
        ctx, host_states, host_obs, host_ld, n_cols, nb, m, slots, stream, !counts_only,
        [&](int64_t b, void *d_states, uint8_t *d_obs, int64_t cols, int64_t c0, int64_t ld) {
            if (!counts_only) {
                int r2 = do_sweep(ctx, d_states, d_obs, cpts, m, cols, ld, c0, seed, pass_id, 0, 0, nullptr,
                                  workspace, stream);
                if (r2) return r2;
            }
            int r2 = same_counts_ema(ctx, d_states, m, cols, ld, decay, totals, workspace, stream);
            if (r2 || counts_only) return r2;
            return same_sample_cpts_ema(ctx, totals, cpts, seed, (uint32_t)(pass_id * M + b), workspace, stream);
        });
}

}  // extern "C"

extern "C" int same_expand_observed(same_ctx *ctx, const int64_t *row_ptr, const int32_t *col_idx,
                                    const void *values, int64_t nnz, int32_t m, int64_t n_cols, int64_t ld,
                                    void *states, uint8_t *obs, void *stream) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!row_ptr || !obs) return set_error(SAME_EINVAL, "row_ptr and obs must be non-null");
    if (nnz < 0) return set_error(SAME_EINVAL, "nnz must be >= 0");
    if (nnz > 0 && (!col_idx || !values)) return set_error(SAME_EINVAL, "col_idx and values must be non-null");
    if (!aligned(obs, 4)) return set_error(SAME_EALIGN, "obs must be 4-byte aligned");
    return check_hip(same::launch_expand(row_ptr, ctx->g.n, col_idx, values, nnz, m, n_cols, ld,
                                         ctx->g.state_bits, states, obs, (hipStream_t)stream),
                     "expand launch");
}

extern "C" int same_init_latent(same_ctx *ctx, void *states, const uint8_t *obs, int32_t m, int64_t n_cols,
                                int64_t ld, int64_t col_offset, uint64_t seed, void *stream) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!obs) return set_error(SAME_EINVAL, "obs is null");
    if (!aligned(obs, 4)) return set_error(SAME_EALIGN, "obs must be 4-byte aligned");
    if (col_offset < 0 || col_offset % 4 != 0)
        return set_error(SAME_EALIGN, "col_offset must be a non-negative multiple of 4");
    if (((col_offset + n_cols) >> 2) > (int64_t)0xFFFFFFFFll)
        return set_error(SAME_ESIZE, "global column index exceeds the Philox counter range (2^34 columns)");
    same::DeviceTables *t = nullptr;
    rc = tables_for_current_device(ctx, &t);
    if (rc) return rc;
    return check_hip(same::launch_init_latent(*t, ctx->g.n, m, n_cols, ld, col_offset, (uint32_t)seed,
                                              (uint32_t)(seed >> 32), ctx->g.state_bits, states, obs,
                                              (hipStream_t)stream),
                     "latent init launch");
}

namespace {
int check_hits_args(same_ctx *ctx, const void *states, const void *target, int32_t m, int64_t n_cols, int64_t ld,
                    int32_t *hits) {
    int rc = check_minibatch(ctx, states, m, n_cols, ld);
    if (rc) return rc;
    if (!target || !hits) return set_error(SAME_EINVAL, "target and hits must be non-null");
    if (!aligned(target, 4 * (size_t)ctx->g.state_bytes))
        return set_error(SAME_EALIGN, "target must be aligned to 4 state elements");
    if (!aligned(hits, 16)) return set_error(SAME_EALIGN, "hits must be 16-byte aligned");
    return SAME_OK;
}
}  // namespace

extern "C" int same_accumulate_hits(same_ctx *ctx, const void *states, const void *target, int32_t m,
                                    int64_t n_cols, int64_t ld, int32_t *hits, void *stream) {
    int rc = check_hits_args(ctx, states, target, m, n_cols, ld, hits);
    if (rc) return rc;
    return check_hip(same::launch_hits(states, target, ctx->g.n, m, n_cols, ld, ctx->g.state_bits, hits,
                                       (hipStream_t)stream),
                     "hits launch");
}

extern "C" int same_predict(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts, const void *target,
                            int32_t m, int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed,
                            uint32_t sweep_id0, int32_t n_sweeps, int32_t *hits, void *workspace, void *stream) {
    int rc = check_hits_args(ctx, states, target, m, n_cols, ld, hits);
    if (rc) return rc;
    if (n_sweeps < 0) return set_error(SAME_EINVAL, "n_sweeps must be >= 0");
    for (int32_t s = 0; s < n_sweeps; ++s) {
        rc = do_sweep(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, sweep_id0 + (uint32_t)s, 0, 0,
                      nullptr, workspace, stream);
        if (rc) return rc;
        rc = check_hip(same::launch_hits(states, target, ctx->g.n, m, n_cols, ld, ctx->g.state_bits, hits,
                                         (hipStream_t)stream),
                       "hits launch");
        if (rc) return rc;
    }
    return SAME_OK;
}

extern "C" int same_grow_replicas(same_ctx *ctx, const void *states, int32_t m, void *dst, int32_t m2, int64_t ld,
                                  void *stream) {
    int rc = check_minibatch(ctx, states, m, ld, ld);
    if (rc) return rc;
    rc = check_minibatch(ctx, dst, m2, ld, ld);
    if (rc) return rc;
    if (m2 < m) return set_error(SAME_EINVAL, "m2 must be >= m");
    const char *a = (const char *)states, *b = (const char *)dst;
    const int32_t qb = ctx->g.quad_bytes;
    if (a < b + (size_t)(ctx->g.n * node_state_bytes(m2, ld, qb)) &&
        b < a + (size_t)(ctx->g.n * node_state_bytes(m, ld, qb)))
        return set_error(SAME_EINVAL, "states and dst must not overlap");
    return check_hip(same::launch_grow(states, m, dst, m2, ctx->g.n, ld, ctx->g.state_bits, (hipStream_t)stream),
                     "replica growth launch");
}

extern "C" int same_kernel_timing(same_ctx *ctx, int32_t enable) {
    if (!ctx) return set_error(SAME_EINVAL, "null context");
    std::lock_guard<std::mutex> lock(ctx->mu);
    int rc = collect_timing(ctx);
    ctx->timing.on = enable != 0;
    for (int32_t k = 0; k < same::kLaunchClasses; ++k) {
        ctx->timing.ms[k] = 0.0;
        ctx->timing.launches[k] = 0;
        ctx->timing.node_samples[k] = 0.0;
    }
    ctx->timing.phase_ms = 0.0;
    ctx->timing.phases = 0;
    return rc;
}

extern "C" int same_kernel_times(same_ctx *ctx, same_kernel_times_t *out) {
    if (!ctx || !out) return set_error(SAME_EINVAL, "null argument");
    std::lock_guard<std::mutex> lock(ctx->mu);
    int rc = collect_timing(ctx);
    for (int32_t k = 0; k < same::kLaunchClasses; ++k) {
        out->ms[k] = ctx->timing.ms[k];
        out->launches[k] = ctx->timing.launches[k];
        out->node_samples[k] = ctx->timing.node_samples[k];
    }
    out->phase_ms = ctx->timing.phase_ms;
    out->phases = ctx->timing.phases;
    return rc;
}

namespace {

// Device layout of the compact-pass slots: two dense slots (states + obs),
// two staging buffers of the largest compact minibatch, the chunk prefix
// sums of the current minibatch and the per-(minibatch, node) offsets.
struct CompactGeom {
    SlotGeom dense;
    size_t staging = 0, prefix = 0, offsets = 0, bytes = 0;
    int64_t chunks = 0;
};

CompactGeom compact_geom(const same_ctx *ctx, int32_t m, int64_t nb, int64_t n_cols, int64_t max_block) {
    CompactGeom c;
    c.dense = slot_geom(ctx, m, nb);
    const int64_t M = (n_cols + nb - 1) / nb;
    c.chunks = (nb + kCompactChunkCols - 1) / kCompactChunkCols;
    c.staging = align_up((size_t)max_block * ctx->g.state_bytes + 8);
    c.prefix = align_up((size_t)ctx->g.n * (size_t)c.chunks * sizeof(int32_t));
    c.offsets = align_up((size_t)(M * ctx->g.n + 1) * sizeof(int64_t));
    c.bytes = 2 * c.dense.bytes + 2 * c.staging + c.prefix + c.offsets;
    return c;
}

int check_compact_args(same_ctx *ctx, const uint8_t *obs_dev, int64_t ld_dev, int64_t n_cols, int64_t nb,
                       int32_t m) {
    if (!ctx || !obs_dev) return set_error(SAME_EINVAL, "ctx and obs_dev must be non-null");
    if (m < 1 || m > 65535) return set_error(SAME_EINVAL, "m must be in [1, 65535]");
    if (nb < 4 || nb % 4 != 0) return set_error(SAME_EALIGN, "nb must be a positive multiple of 4");
    if (n_cols < 0 || ld_dev < n_cols || ld_dev % 4 != 0)
        return set_error(SAME_EINVAL, "need 0 <= n_cols <= ld_dev, ld_dev a multiple of 4");
    if (!aligned(obs_dev, 4)) return set_error(SAME_EALIGN, "obs_dev must be 4-byte aligned");
    return SAME_OK;
}

}  // namespace

extern "C" {

int same_stream_compact_layout(same_ctx *ctx, const uint8_t *obs_dev, int64_t ld_dev, int64_t n_cols, int64_t nb,
                               int32_t m, int64_t *lat_off, size_t *slot_bytes, void *workspace, void *stream) {
    int rc = check_compact_args(ctx, obs_dev, ld_dev, n_cols, nb, m);
    if (rc) return rc;
    if (!lat_off || !slot_bytes || !workspace) return set_error(SAME_EINVAL, "null pointer argument");
    if (!aligned(workspace, kAlign)) return set_error(SAME_EALIGN, "workspace must be 256-byte aligned");
    const int32_t n = ctx->g.n;
    const int64_t M = n_cols > 0 ? (n_cols + nb - 1) / nb : 0;
    hipStream_t s = (hipStream_t)stream;
    // per node counts in the workspace's count scratch (cpt_total >= 2n entries)
    int32_t *counts = (int32_t *)((char *)workspace + ctx->ws_counts);
    std::vector<int32_t> host((size_t)n);
    int64_t run = 0, max_block = 0;
    for (int64_t b = 0; b < M; ++b) {
        const int64_t c0 = b * nb, cols = n_cols - c0 < nb ? n_cols - c0 : nb;
        rc = check_hip(same::launch_compact_node_counts(obs_dev, ld_dev, c0, cols, n, counts, s), "count launch");
        if (!rc) rc = check_hip(hipMemcpyAsync(host.data(), counts, (size_t)n * sizeof(int32_t),
                                               hipMemcpyDeviceToHost, s), "count copy");
        if (!rc) rc = check_hip(hipStreamSynchronize(s), "hipStreamSynchronize");
        if (rc) return rc;
        const int64_t start = run;
        for (int32_t i = 0; i < n; ++i) {
            lat_off[b * n + i] = run;
            run += (int64_t)m * host[i];
        }
        max_block = std::max(max_block, run - start);
    }
    lat_off[M * n] = run;
    *slot_bytes = compact_geom(ctx, m, nb, n_cols, max_block).bytes;
    return SAME_OK;
}

int same_stream_pass_compact(same_ctx *ctx, void *lat_host, const int64_t *lat_off, const uint8_t *obs_dev,
                             const void *data_dev, int64_t ld_dev, int64_t n_cols, int64_t nb, int32_t m,
                             float *cpts, int32_t *mb_counts, int32_t *totals, uint64_t seed, uint32_t pass_id,
                             int32_t flags, void *slots, void *workspace, void *stream) {
    int rc = check_compact_args(ctx, obs_dev, ld_dev, n_cols, nb, m);
    if (rc) return rc;
    if (!lat_host || !lat_off || !data_dev || !cpts || !mb_counts || !totals || !slots || !workspace)
        return set_error(SAME_EINVAL, "null pointer argument");
    if (flags & ~SAME_STREAM_COUNTS_ONLY) return set_error(SAME_EINVAL, "unknown flags");
    if (!aligned(slots, kAlign) || !aligned(workspace, kAlign))
        return set_error(SAME_EALIGN, "slots and workspace must be 256-byte aligned");
    if (!aligned(data_dev, 4 * (size_t)ctx->g.state_bytes))
        return set_error(SAME_EALIGN, "data_dev must be aligned to 4 state elements");
    if (n_cols == 0) return SAME_OK;
    const int32_t n = ctx->g.n;
    const int64_t M = (n_cols + nb - 1) / nb;
    if ((double)M * (double)pass_id + M > 4294967295.0)
        return set_error(SAME_ESIZE, "pass_id * minibatches exceeds the update-id range");
    int64_t max_block = 0;
    for (int64_t b = 0; b < M; ++b) max_block = std::max(max_block, lat_off[(b + 1) * n] - lat_off[b * n]);
    const CompactGeom cg = compact_geom(ctx, m, nb, n_cols, max_block);
    StreamRes *sr = nullptr;
    rc = stream_res_for_current_device(ctx, &sr);
    if (rc) return rc;
    hipStream_t cs = (hipStream_t)stream;
    const size_t sb = (size_t)ctx->g.state_bytes;
    const int64_t total = ctx->g.off[n];
    const bool counts_only = (flags & SAME_STREAM_COUNTS_ONLY) != 0;
    char *base = (char *)slots;
    char *staging[2] = {base + 2 * cg.dense.bytes, base + 2 * cg.dense.bytes + cg.staging};
    int32_t *prefix = (int32_t *)(base + 2 * cg.dense.bytes + 2 * cg.staging);
    int64_t *d_off = (int64_t *)((char *)prefix + cg.prefix);
    // the offsets on the device (the kernels subtract each minibatch's first)
    rc = check_hip(hipMemcpyAsync(d_off, lat_off, (size_t)(M * n + 1) * sizeof(int64_t), hipMemcpyHostToDevice, cs),
                   "offset upload");
    if (rc) return rc;
    for (int64_t b = 0; b < M; ++b) {
        const int sl = (int)(b & 1);
        const int64_t c0 = b * nb, cols = n_cols - c0 < nb ? n_cols - c0 : nb;
        char *slot = base + sl * cg.dense.bytes;
        void *d_states = slot;
        uint8_t *d_obs = (uint8_t *)(slot + cg.dense.states);
        const int64_t blk0 = lat_off[b * n], blk = lat_off[(b + 1) * n] - blk0;
        // upload the compact block (after the staging buffer's previous block left it)
        if (sr->slot_used[sl] && (rc = check_hip(hipStreamWaitEvent(sr->up, sr->ev_down[sl], 0), "wait")))
            return rc;
        rc = check_hip(hipMemcpyAsync(staging[sl], (char *)lat_host + blk0 * sb, (size_t)blk * sb,
                                      hipMemcpyHostToDevice, sr->up), "latent upload");
        if (!rc) rc = check_hip(hipEventRecord(sr->ev_up[sl], sr->up), "event");
        if (!rc) rc = check_hip(hipStreamWaitEvent(cs, sr->ev_up[sl], 0), "wait");
        if (rc) return rc;
        // chunk ranks, then the dense slot
        rc = check_hip(same::launch_compact_counts(obs_dev, ld_dev, c0, cols, n, prefix, true, cs), "count launch");
        if (!rc)
            rc = check_hip(same::launch_expand_compact(obs_dev, data_dev, ld_dev, c0, cols, n, m, prefix,
                                                       d_off + b * n, blk0, staging[sl], d_states, d_obs,
                                                       cg.dense.ld, ctx->g.state_bits, cs),
                           "expand launch");
        if (rc) return rc;
        int32_t *mb = mb_counts + b * total;
        if (counts_only) rc = same_counts(ctx, d_states, m, cols, cg.dense.ld, mb, totals, workspace, stream);
        else
            rc = do_step(ctx, d_states, d_obs, cpts, m, cols, cg.dense.ld, c0, seed, pass_id, mb, totals,
                         (uint32_t)(pass_id * M + b), workspace, stream);
        if (rc) return rc;
        if (counts_only) {
            rc = check_hip(hipEventRecord(sr->ev_down[sl], cs), "event");
        } else {
            rc = check_hip(same::launch_gather_compact(obs_dev, ld_dev, c0, cols, n, m, prefix, d_off + b * n,
                                                       blk0, d_states, cg.dense.ld, staging[sl],
                                                       ctx->g.state_bits, cs),
                           "gather launch");
            if (!rc) rc = check_hip(hipEventRecord(sr->ev_comp[sl], cs), "event");
            if (!rc) rc = check_hip(hipStreamWaitEvent(sr->down, sr->ev_comp[sl], 0), "wait");
            if (!rc)
                rc = check_hip(hipMemcpyAsync((char *)lat_host + blk0 * sb, staging[sl], (size_t)blk * sb,
                                              hipMemcpyDeviceToHost, sr->down), "latent download");
            if (!rc) rc = check_hip(hipEventRecord(sr->ev_down[sl], sr->down), "event");
        }
        if (rc) return rc;
        sr->slot_used[sl] = true;
    }
    for (int sl = 0; sl < 2; ++sl)
        if (sr->slot_used[sl] && (rc = check_hip(hipStreamWaitEvent(cs, sr->ev_down[sl], 0), "wait")))
            return rc;
    return SAME_OK;
}

}  // extern "C"

// ------------------------------------------------ replayable step graphs

// A captured sequence of SAME steps over one resident minibatch.
struct same_graph {
    int device = -1;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
};

namespace {

constexpr int32_t kMaxGraphSteps = 64;

void free_graph(same_graph *g) {
    if (!g) return;
    if (g->exec) (void)hipGraphExecDestroy(g->exec);
    if (g->graph) (void)hipGraphDestroy(g->graph);
    delete g;
}

}  // namespace

extern "C" {

int same_step_graph(same_ctx *ctx, void *states, const uint8_t *obs, float *cpts, int32_t m, int64_t n_cols,
                    int64_t ld, int64_t col_offset, uint64_t seed, int32_t *mb_counts, int32_t *totals,
                    uint32_t *ids, uint32_t update_stride, int32_t steps, void *workspace, same_graph **out) {
    if (!out) return set_error(SAME_EINVAL, "out is null");
    *out = nullptr;
    int rc = check_sweep_args(ctx, states, obs, cpts, m, n_cols, ld, col_offset, 0, 0, nullptr, workspace);
    if (rc) return rc;
    if (!mb_counts || !totals || !ids) return set_error(SAME_EINVAL, "mb_counts, totals and ids must be non-null");
    if (!aligned(ids, 4)) return set_error(SAME_EALIGN, "ids must be 4-byte aligned");
    if (steps < 1 || steps > kMaxGraphSteps) return set_error(SAME_EINVAL, "steps must be in [1, 64]");
    if (n_cols < 1) return set_error(SAME_EINVAL, "n_cols must be positive");
    if ((double)n_cols * (double)m >= 2147483648.0) return set_error(SAME_ESIZE, "n_cols * m must stay below 2^31");
    // what is set up synchronously on first use happens before the capture
    same::DeviceTables *t = nullptr;
    rc = tables_for_current_device(ctx, &t);
    StreamRes *sr = nullptr;
    if (!rc) rc = stream_res_for_current_device(ctx, &sr);
    if (rc) return rc;
    same_graph *g = new (std::nothrow) same_graph();
    if (!g) return set_error(SAME_ENOMEM, "out of host memory");
    rc = check_hip(hipGetDevice(&g->device), "hipGetDevice");
    hipStream_t cs = nullptr;
    if (!rc) rc = check_hip(hipStreamCreateWithFlags(&cs, hipStreamNonBlocking), "hipStreamCreateWithFlags");
    if (rc) {
        free_graph(g);
        return rc;
    }
    // per-launch timing records events; none go into the graph
    const bool timing = ctx->timing.on;
    ctx->timing.on = false;
    rc = check_hip(hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
    if (!rc) {
        for (int32_t k = 0; k < steps && !rc; ++k) {
            rc = do_step(ctx, states, obs, cpts, m, n_cols, ld, col_offset, seed, 0, mb_counts, totals, 0,
                         workspace, cs, ids);
            if (!rc) rc = check_hip(same::launch_advance_ids(ids, 1, update_stride, cs), "id advance launch");
        }
        // the capture ends whether or not a launch failed
        const int rc_end = check_hip(hipStreamEndCapture(cs, &g->graph), "hipStreamEndCapture");
        if (!rc) rc = rc_end;
    }
    ctx->timing.on = timing;
    (void)hipStreamDestroy(cs);
    if (!rc) rc = check_hip(hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0), "hipGraphInstantiate");
    if (rc) {
        free_graph(g);
        return rc;
    }
    *out = g;
    return SAME_OK;
}

int same_graph_launch(same_graph *g, void *stream) {
    if (!g || !g->exec) return set_error(SAME_EINVAL, "graph is null");
    int device = -1;
    int rc = check_hip(hipGetDevice(&device), "hipGetDevice");
    if (rc) return rc;
    if (device != g->device) return set_error(SAME_EINVAL, "the graph was captured on another device");
    return check_hip(hipGraphLaunch(g->exec, (hipStream_t)stream), "hipGraphLaunch");
}

void same_graph_destroy(same_graph *g) { free_graph(g); }

}  // extern "C"
