// Internal launch interface between the C ABI (api.cpp) and the gfx950
// kernels (kernels.hip).  Plain device pointers only.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "graph.hpp"

namespace same {

// Device copies of the compiled structure tables (one set per device).
struct DeviceTables {
    int device = -1;
    int32_t *desc = nullptr;       // sweep descriptor stream
    int32_t *desc_off = nullptr;   // [n]
    int32_t *order = nullptr;      // colour-ordered nodes
    int32_t *cdesc = nullptr;      // count descriptor stream: [K, n_par, nbins, cpt_off, (p, stride)*]
    int32_t *cdesc_off = nullptr;  // [n]
    int32_t *cwork = nullptr;      // count work items (node, first bin)
    int32_t n_cwork = 0;
    Segment *segs = nullptr;
    int32_t *blk_seg = nullptr;    // table-build block -> segment
    int32_t *blk_first = nullptr;  // table-build block -> first group
    int32_t n_build_blocks = 0;
    int32_t *row_off = nullptr;    // [n_rows]
    int32_t *row_k = nullptr;      // [n_rows]
    int32_t *cprog = nullptr;      // threshold build programs
    int32_t *cprog_off = nullptr;
    int32_t *cblk_prog = nullptr;  // threshold-build block -> program
    int32_t *cblk_first = nullptr; // threshold-build block -> first configuration
    int32_t n_cond_blocks = 0;
};

// Kernel arguments of the sweep (passed by value).
struct SweepParams {
    const int32_t *desc;
    const int32_t *desc_off;
    const int32_t *order;
    int32_t begin;                 // first entry of order[] in this launch
    const float *table;            // regrouped k-vector tables (workspace)
    const uint32_t *cond;          // threshold tables (workspace)
    void *states;
    const uint8_t *obs;
    int32_t m;
    int64_t n_cols, ld, col_offset;
    uint32_t key0, key1, sweep_id;
    // block geometry, set by the launcher: a launch covers `count` nodes x
    // `n_slabs` slabs (a column chunk of quads_per_block quads x a replica
    // range of reps_per_block); see block_work in kernels.hip
    int64_t quads_per_block;
    int32_t reps_per_block;
    int32_t count;
    int32_t rsplit;
    int64_t n_slabs;
    int64_t win_begin, win;        // debug window (win == 0: none)
    int32_t reverse;               // 1: slabs in descending order (see block_work)
    float *probs;
    int32_t max_card;
    // nullable: when set, the sweep id is read from ids[0] on the device at
    // launch time instead of sweep_id (replayed HIP graphs of a step)
    const uint32_t *ids;
};

hipError_t launch_build_tables(const DeviceTables &t, const float *cpts, float *table,
                               hipStream_t stream);

hipError_t launch_build_thresholds(const DeviceTables &t, const float *cpts, uint32_t *cond,
                                   hipStream_t stream);

// launch_build_tables, launch_build_thresholds and (zero_count > 0) a clear of
// zero[0 .. zero_count) in one launch.
hipError_t launch_prepare(const DeviceTables &t, const float *cpts, float *table, uint32_t *cond, int32_t *zero,
                          int64_t zero_count, hipStream_t stream);

// Nodes order[begin .. begin+count) of one colour, all of launch class klass
// (0: fast kernel, tables staged in lds_bytes of LDS; 1: fast kernel, tables
// in global memory; 2: wide kernel; 3: generic kernel).
hipError_t launch_sweep(SweepParams P, int32_t begin, int32_t count, int32_t klass,
                        int32_t lds_bytes, int32_t state_bits, hipStream_t stream);

hipError_t launch_fill_zero(int32_t *p, int64_t count, hipStream_t stream);

// Entries of the file-scope count scratch of the allocation-free count entry
// point (int32; 8 MiB per device).
constexpr int64_t kScratchCountEntries = int64_t(1) << 21;

// Device address of that scratch on `device`, which must be the current
// device; resolved with hipGetSymbolAddress on the first call per device.
// Allocates nothing.
hipError_t scratch_counts(int device, int32_t **out);

// Histograms of every node's family (the count work items of t) over the
// columns [col0, col0 + n_cols) of states [n][m][ld].
hipError_t launch_counts(const DeviceTables &t, const void *states, int32_t state_bits,
                         int32_t m, int64_t col0, int64_t n_cols, int64_t ld, int32_t *counts,
                         hipStream_t stream);

// Dense minibatch from CSR known entries (rows = nodes): clears obs, then
// one thread per entry writes obs and every replica's state.
hipError_t launch_expand(const int64_t *row_ptr, int32_t n, const int32_t *col_idx, const void *values,
                         int64_t nnz, int32_t m, int64_t n_cols, int64_t ld, int32_t state_bits,
                         void *states, uint8_t *obs, hipStream_t stream);

// Random initial states of the latent entries (Philox tag 2).
hipError_t launch_init_latent(const DeviceTables &t, int32_t n, int32_t m, int64_t n_cols, int64_t ld,
                              int64_t col_offset, uint32_t key0, uint32_t key1, int32_t state_bits,
                              void *states, const uint8_t *obs, hipStream_t stream);

// Held-out prediction: hits[i][j] += replicas whose state equals target[i][j] >= 0.
hipError_t launch_hits(const void *states, const void *target, int32_t n, int32_t m, int64_t n_cols, int64_t ld,
                       int32_t state_bits, int32_t *hits, hipStream_t stream);

// Compact host state of the out-of-core passes: latent columns per (node,
// chunk of 1024 columns) of the minibatch [c0, c0 + cols) of obs [n][obs_ld]
// into counts [n][chunks] (with prefix, turned into per-node exclusive
// prefix sums); the dense slot from the device-resident known data and the
// compact latent states (node i's block at lat_states + node_off[i] - off0);
// and the latent states back into compact form.
hipError_t launch_compact_counts(const uint8_t *obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t n,
                                 int32_t *counts, bool prefix, hipStream_t stream);
// Latent columns of each node of the minibatch into counts [n].
hipError_t launch_compact_node_counts(const uint8_t *obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t n,
                                      int32_t *counts, hipStream_t stream);
hipError_t launch_expand_compact(const uint8_t *obs, const void *data, int64_t obs_ld, int64_t c0, int64_t cols,
                                 int32_t n, int32_t m, const int32_t *prefix, const int64_t *node_off, int64_t off0,
                                 const void *lat_states, void *states, uint8_t *obs_slot, int64_t slot_ld,
                                 int32_t state_bits, hipStream_t stream);
hipError_t launch_gather_compact(const uint8_t *obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t n, int32_t m,
                                 const int32_t *prefix, const int64_t *node_off, int64_t off0, const void *states,
                                 int64_t slot_ld, void *lat_states, int32_t state_bits, hipStream_t stream);

// SAME annealing: dst (m2 replicas) from src (m replicas), replica r of dst
// taking replica r mod m; both in the state-quad layout with leading dimension ld.
hipError_t launch_grow(const void *src, int32_t m, void *dst, int32_t m2, int32_t n, int64_t ld,
                       int32_t state_bits, hipStream_t stream);

hipError_t launch_moving_sum(const int32_t *newc, int32_t *mb, int32_t *totals, int64_t total,
                             hipStream_t stream);

// ids (nullable): the update id is read from ids[1] on the device instead.
hipError_t launch_gamma(const int32_t *totals, double alpha, uint32_t key0, uint32_t key1,
                        uint32_t update_id, const uint32_t *ids, double *g, int64_t total,
                        hipStream_t stream);
hipError_t launch_gamma(const double *totals, double alpha, uint32_t key0, uint32_t key1,
                        uint32_t update_id, const uint32_t *ids, double *g, int64_t total,
                        hipStream_t stream);

// launch_moving_sum (totals non-null) followed by launch_gamma on the
// updated totals, in one launch.
hipError_t launch_moving_sum_gamma(const int32_t *newc, int32_t *mb, int32_t *totals, double alpha, uint32_t key0,
                                   uint32_t key1, uint32_t update_id, const uint32_t *ids, double *g, int64_t total,
                                   hipStream_t stream);

// ids[0] += d0, ids[1] += d1 (one thread; the last node of a graphed step).
hipError_t launch_advance_ids(uint32_t *ids, uint32_t d0, uint32_t d1, hipStream_t stream);

// Exponential moving sum: totals = decay * totals + newc (fp64).
hipError_t launch_ema(const int32_t *newc, double *totals, double decay, int64_t total, hipStream_t stream);

hipError_t launch_normalize(const DeviceTables &t, const double *g, float *cpts, int64_t n_rows,
                            hipStream_t stream);

}  // namespace same
