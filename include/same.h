/*
 * same.h -- C ABI of libsame, an MI355X (gfx950) implementation of SAME Gibbs
 * sampling for discrete Bayesian networks (Seita, Chen & Canny, arXiv
 * 1511.06416).
 *
 * The problem (Sec. 1): a Bayesian network of known structure whose nodes take
 * discrete states and whose conditional probability tables (CPTs) Theta are
 * unknown; the data are a node x case matrix in which some entries are
 * missing.  The sampler draws the missing states Z and the CPTs from
 * P(Z, Theta | D).  SAME (Sec. 3, Eq. 1) replicates the latent states m times,
 * all tied to one Theta.  The data are processed in same-sized minibatches of
 * columns (Sec. 4); per minibatch the library runs one chromatic Gibbs sweep
 * over the m replicas (Sec. 4, colour groups of the moralized graph visited
 * in order), counts (parent configuration, state) pairs, keeps the exact
 * moving sum of the per-minibatch counts, and resamples every CPT row from
 * Dirichlet(prior + counts).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Graph:  nodes 0..n-1; parent lists in CSR form (parent_ptr[n+1],
 *         parent_idx[parent_ptr[n]]).  The listed parent order fixes the CPT
 *         row radix: row u = sum_j x_{pa_j} * stride_j with the LAST listed
 *         parent fastest.
 * CPTs:   one flat fp32 array of cpt_total entries; node i owns
 *         [cpt_off[i], cpt_off[i+1]) = R_i rows of K_i entries, entry
 *         cpt_off[i] + u*K_i + k = P(x_i = k | parents in configuration u).
 * States: device array [n][mq][ld][4] of int8 (every K_i <= 127) or int16
 *         (some K_i >= 128), mq = ceil(m / 4): replica r of node i at
 *         minibatch column j, written states[i][r][j] below, is element
 *         ((i * mq + r / 4) * ld + j) * 4 + r % 4.  The four replicas
 *         4q .. 4q + 3 of one column (a state quad) are adjacent, so the
 *         sweep reads and writes them with one access.  With 4-bit states
 *         (same_options_t.state_bits = 4) the array is [n][mq][ld] of 16-bit
 *         words, one state quad each, replica 4q + s in bits 4s .. 4s + 3.  Column j of a
 *         minibatch is global column col_offset + j.  Observed entries must
 *         hold the observed value in every replica.  Values must lie in
 *         [0, K_i) (out-of-range values are undefined behaviour).  Slots
 *         r >= m of the last quad are padding and may hold anything: the
 *         sweep reads them as state 0 and writes valid draws there, and
 *         counts, hits and replica growth skip them.
 * Obs:    device array [n][ld] of uint8, 1 = observed, 0 = latent; shared by
 *         the m replicas.  Columns [n_cols, ld) are never drawn or counted.
 * Counts: int32, laid out like the CPTs.
 * Memory: the caller owns every state, obs, CPT, count and workspace buffer
 *         (device memory; PyTorch tensors in the Python binding).  The
 *         library owns only the context and its small per-device structure
 *         tables, uploaded synchronously on the first device call.
 * Streams: `stream` is a hipStream_t passed as void* (NULL = null stream);
 *         device work is enqueued asynchronously on it.  Argument errors are
 *         detected and returned before anything is enqueued.
 * Errors: functions return SAME_OK (0) or a negative SAME_E* code;
 *         same_last_error() gives a message for the calling thread's last
 *         failure.  A context is used by one host thread at a time.
 * Random numbers: Philox4x32-10 (Salmon et al., SC'11) keyed by the 64-bit
 *         seed; the Gibbs draw of node i, replica r, global column g in sweep
 *         s takes word r&3 of the block at counter {g, i, r>>2, s} (one block
 *         per column and quad of replicas; g < 2^32); the Gamma
 *         attempt t of CPT entry e at update q uses counter {e, t, 1<<24, q};
 *         the initial latent state uses {g>>2, i, r | 2<<24, 0}.
 */
#ifndef SAME_H
#define SAME_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct same_ctx same_ctx;

enum {
    SAME_OK = 0,
    SAME_EINVAL = -1,  /* bad argument (null pointer, m < 1, n_cols > ld, ...) */
    SAME_EGRAPH = -2,  /* cycle, self-loop, duplicate or out-of-range parent */
    SAME_ECARD = -3,   /* a cardinality outside [2, 32767] */
    SAME_ESIZE = -4,   /* a size that overflows the library's int32 indexing */
    SAME_ENOMEM = -5,  /* host or device allocation failed */
    SAME_EHIP = -6,    /* a HIP runtime call failed (message has the HIP error) */
    SAME_EALIGN = -7   /* col_offset or ld not a multiple of 4, misaligned pointer */
};

typedef struct {
    int32_t n_nodes;
    int32_t n_colors;     /* colour groups of the moralized graph */
    int64_t cpt_total;    /* CPT entries */
    int64_t n_rows;       /* CPT rows (distributions) */
    int32_t state_bytes;  /* bytes of one state in the element arrays (CSR values, targets,
                             compact host states): 1, or 2 for 16-bit states */
    int32_t max_card;     /* largest K_i */
    int32_t sweep_launches;  /* sweep kernel launches per same_sweep call */
    int32_t table_nodes;     /* nodes drawing from precomputed threshold tables */
    int32_t state_bits;      /* bits per state in the states array: 4, 8 or 16 (see States) */
} same_layout_t;

/*
 * Builds a context for one network (Sec. 1 problem statement; Sec. 4 colour
 * groups).  Host only: validates the DAG, orders it topologically, builds the
 * moralized graph (parents joined, directions dropped), colours it first-fit
 * over a Kahn topological order that takes the smallest ready id and then
 * balances the colour groups (Sec. 4 asks for groups of balanced size):
 * repeatedly, the first node -- scanning groups from the largest (ties:
 * lower colour), nodes by ascending id -- that can move to a group at least
 * two nodes smaller (scanning from the smallest, ties: lower colour) without
 * a moral neighbour there moves to it, until no such move is left; lays out
 * the CPTs and the per-node Markov-blanket tables.  dirichlet_prior (> 0) is
 * the Dirichlet parameter added to every count in same_sample_cpts.  The
 * arrays are copied; the caller may free them after the call.
 */
int same_create(int32_t n_nodes, const int32_t *parent_ptr, const int32_t *parent_idx,
                const int32_t *card, double dirichlet_prior, same_ctx **out);

/* Build options for same_create_ex. */
typedef struct {
    /* Largest (blanket configurations) x (thresholds per configuration) for
     * which a node's full conditional is precomputed into a table of CDF
     * thresholds (one table per CPT update; the draw becomes one table read).
     * -1 selects the default (6144, so that a table fits the default LDS
     * staging budget below); 0 disables the tables, so every node
     * forms its conditional from CPT entries during the sweep.  Either way the
     * sweep draws from the same conditional with the same uniforms. */
    int64_t table_limit;
    /* Target bytes of states + obs per column tile of a sweep (0: default,
     * one tile = the whole minibatch).  Tiles are at least 1024 columns wide.
     * Results do not depend on it. */
    int64_t tile_bytes;
    /* LDS staging budget of a sweep block (bytes): a node's table record up
     * to this size is copied into LDS before drawing; a larger record stages
     * its smallest CPT groups up to this size and reads the rest from global
     * memory.  -1 selects the default (24576); at most 32768; 0 stages
     * nothing.  Such a record is laid out with its staged groups first, and
     * the fp32 product of a conditional is formed in record order, so the
     * budget can change a conditional in its last bits: draws agree except
     * where a uniform lies within rounding of a CDF boundary. */
    int64_t lds_limit;
    /* 1 (default): blanket indices of nodes with K <= 8 and records below
     * 2^16 rows use packed 16-bit arithmetic; 0: every product-mode node uses
     * the 32-bit path.  Results do not depend on it. */
    int32_t packed_indices;
    /* 0 (default): the first-fit colouring is balanced by single-node moves
     * between colour groups that keep it proper (see same_create); 1: the
     * first-fit colouring as it is.  The colouring fixes the order of the
     * sequential scan the sweep equals, so it changes the sample path. */
    int32_t first_fit_colours;
    /* 0 (default): 8-bit states (16-bit when some K > 127); 4: 4-bit states,
     * a state quad in one 16-bit word (every K must be <= 16, else
     * SAME_ECARD).  The states array's format follows (see States); results
     * do not depend on it. */
    int32_t state_bits;
} same_options_t;

/* same_create with options (opts may be NULL for the defaults). */
int same_create_ex(int32_t n_nodes, const int32_t *parent_ptr, const int32_t *parent_idx,
                   const int32_t *card, double dirichlet_prior, const same_options_t *opts,
                   same_ctx **out);

/* Frees the context and its device tables (on every device it used). */
void same_destroy(same_ctx *ctx);

/*
 * Copies out the layout; cpt_off (n+1 entries) and color (n entries) are
 * optional.  Host only.
 */
int same_layout(const same_ctx *ctx, same_layout_t *out, int64_t *cpt_off, int32_t *color);

/*
 * Bytes of device workspace that same_sweep, same_sweep_debug, same_counts
 * and same_sample_cpts need (one buffer serves all of them; 256-byte aligned
 * base required).  The workspace holds the sweep's regrouped CPT tables, the
 * new-count histogram and the fp64 Gamma variates; its contents need not be
 * preserved between calls.  Host only.
 */
int same_workspace_size(const same_ctx *ctx, size_t *bytes);

/*
 * One chromatic Gibbs sweep over one minibatch, in place (Sec. 4: colour
 * groups in ascending order; inside a group every (node, column, replica) is
 * independent).  For every latent entry the full conditional
 *   P(x_i = k | rest) ~ theta_i(k | x_pa(i)) * prod_{h in ch(i)} theta_h(x_h | x_pa(h), x_i = k)
 * is formed from max(theta, FLT_MIN) and a state is drawn by inverse CDF: with
 * S_k the running sum of the weights and Z = S_{K-1}, the smallest k with
 * u*Z < S_k, else the largest k with positive weight (u = 24-bit uniform).
 * Nodes whose Markov blanket has few configurations (see same_options_t) read
 * integer thresholds ceil(2^24 S_k / Z) precomputed in fp64 for every blanket
 * configuration; the others multiply fp32 CPT entries (relative error below
 * (1 + children) * 2^-24 per weight) at every draw.
 * states (in/out, the layout above), obs [n][ld], cpts [cpt_total]: device
 * pointers.
 * col_offset and ld must be multiples of 4 and states/obs 4-byte aligned.
 * seed and sweep_id select the Philox stream.  The colour groups launch in
 * order on `stream`.  Inside a group, the nodes whose tables are read from
 * global memory (launch class 1) run on a side stream that the context keeps
 * per device, forked from and joined back into `stream` with events, beside
 * the group's LDS-staged launch; the call's work is still ordered on `stream`
 * as a whole.  Sweeps issued on several streams of one context share that side
 * stream, so their class-1 launches run in issue order.
 */
int same_sweep(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts, int32_t m,
               int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed, uint32_t sweep_id,
               void *workspace, void *stream);

/*
 * same_sweep that also writes the fp32 conditionals of columns
 * [win_begin, win_begin + win) to probs[((i*m + r)*win + (j - win_begin))*max_card + k]
 * (device pointer, n*m*win*max_card floats); entries of observed columns and
 * k >= K_i are left untouched.  For parity checks.
 */
int same_sweep_debug(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts,
                     int32_t m, int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed,
                     uint32_t sweep_id, int64_t win_begin, int64_t win, float *probs,
                     void *workspace, void *stream);

/*
 * Parity/debug: the CDF threshold tables same_sweep draws from for the CPTs
 * `cpts` (nodes whose Markov blanket has few configurations; see
 * same_options_t.table_limit).  Such a node's table has one row of KT uint32
 * words per configuration of its Markov blanket -- its parents, children and
 * the children's other parents, each once, in ascending node id, the last
 * one varying fastest -- holding T_k = ceil(2^24 S_k / Z) for k < K - 1 and
 * 2^24 after that, where S_k / Z is the cumulative conditional of Sec. 4's
 * Gibbs draw (own CPT entry times the children's entries) formed in fp64.
 * The sweep's draw with 24-bit uniform u24 is #{k : T_k <= u24}.
 * Host outputs: node_off[n] (word offset of node i's table, -1 for nodes that
 * form their conditional from CPT entries), node_kt[n] (KT, 0 for those) and
 * *words (total table words).  cond_out (device, nullable, 4-byte aligned,
 * *words entries) receives the tables, built on `stream` in the workspace
 * and copied out.  Errors: SAME_EINVAL for null ctx, outputs or (with
 * cond_out) cpts/workspace; SAME_EALIGN; SAME_EHIP.
 */
int same_debug_thresholds(same_ctx *ctx, const float *cpts, int64_t *node_off, int32_t *node_kt,
                          int64_t *words, uint32_t *cond_out, void *workspace, void *stream);

/*
 * Sufficient statistics and their moving sum (Sec. 4): histogram of
 * (parent configuration, state) over columns [0, n_cols) and all m replicas of
 * states (the layout above).  mb_counts [cpt_total] holds this minibatch's previous
 * counts on entry (zeros on its first visit) and its new counts on return;
 * totals [cpt_total] (nullable) += new - previous.  Device pointers.  Counts
 * are exact (integer) and independent of launch order; n_cols * m * (number
 * of minibatches) must stay below 2^31.
 */
int same_counts(same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld,
                int32_t *mb_counts, int32_t *totals, void *workspace, void *stream);

/*
 * same_counts for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same histogram and moving sum, with the new-count histogram held in a
 * library-owned device array of 2^21 int32 entries (8 MiB, one per device,
 * kept until the process ends) instead of the workspace.  No workspace
 * argument; the call allocates nothing and clears the array with a kernel
 * (no memset).  Preconditions: cpt_total <= 2^21 (else SAME_ESIZE), and the
 * context's structure tables already on the current device, i.e. some other
 * device call of this context (same_counts, same_sweep, ...) has run on it
 * (else SAME_EINVAL).  Every call on one device shares the array, which keeps
 * the last call's contents: calls that overlap on one device (other streams,
 * other threads, other contexts) race and must be ordered by the caller.
 * Other arguments and errors as same_counts.
 */
int same_counts_noalloc(same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld,
                        int32_t *mb_counts, int32_t *totals, void *stream);

/*
 * Dirichlet resample of every CPT row (Sec. 4: counts plus the Dirichlet
 * prior are the Dirichlet parameters from which the CPTs are sampled):
 * g_e ~ Gamma(prior + totals[e], 1) (Marsaglia & Tsang, in fp64), then
 * cpts_out[e] = fp32(g_e / sum of g over e's row).  update_id selects the
 * Philox stream (one id per resample).  Device pointers.
 */
int same_sample_cpts(same_ctx *ctx, const int32_t *totals, float *cpts_out, uint64_t seed,
                     uint32_t update_id, void *workspace, void *stream);

/*
 * How same_sweep splits a minibatch of n_cols columns with m replicas: the
 * column-tile width and the number of sweep-kernel launches per call (for
 * profiling; host only).
 */
int same_sweep_plan(const same_ctx *ctx, int32_t m, int64_t n_cols, int64_t *tile_cols,
                    int32_t *launches);

/*
 * One whole SAME step over one minibatch (Sec. 4, Fig. 1): same_sweep, then
 * same_counts into mb_counts and totals, then same_sample_cpts writing cpts in
 * place with update_id.  The result equals those three calls in that order.
 * With a tile_bytes option the sweep and the counts run tile by tile, so the
 * count pass reads the tile the sweep just visited.  Device pointers; cpts is
 * read by the sweep and rewritten by the resample.
 */
int same_step(same_ctx *ctx, void *states, const uint8_t *obs, float *cpts, int32_t m,
              int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed, uint32_t sweep_id,
              int32_t *mb_counts, int32_t *totals, uint32_t update_id, void *workspace,
              void *stream);

/*
 * Out-of-core passes (Sec. 4: the sampler keeps only model-sized state on the
 * device and streams the data; Sec. 6: the GPU's memory, not the data size,
 * limits the problem).  The data stay in host memory -- pinned (page-locked)
 * for the copies to overlap -- laid out like a device minibatch but with the
 * full column range: states [n][mq][host_ld][4], obs [n][host_ld], column j is
 * global column j.  Minibatch b covers columns [b*nb, min((b+1)*nb, n_cols)).
 *
 * same_stream_pass runs one pass over all M = ceil(n_cols / nb) minibatches:
 * per minibatch b it copies the minibatch to the device (upload stream), runs
 * same_sweep (col_offset b*nb, sweep_id = pass_id), same_counts into
 * mb_counts[b] and totals, and same_sample_cpts (update_id = pass_id*M + b)
 * on `stream`, then copies the new states back to the host (download stream).
 * Two device slots alternate, so the upload of b+1 and the download of b-1
 * overlap the compute of b.  With flags & SAME_STREAM_COUNTS_ONLY it only
 * uploads and counts (the count-only pre-pass that initialises mb_counts and
 * totals before the first sweep; mb_counts and totals must be zero on entry).
 *
 * cpts [cpt_total] (device, in/out), mb_counts [M][cpt_total] and totals
 * [cpt_total] (device) persist between passes.  slots (device, at least
 * same_stream_slots_size bytes, 256-byte aligned) holds the two slots;
 * workspace is the same_workspace_size buffer.  nb must be a multiple of 4.
 * The call returns when everything is enqueued; the host states are final
 * once `stream` has been synchronised.  The caller must not touch the host
 * buffers or `stream`'s work until then.
 */
enum { SAME_STREAM_COUNTS_ONLY = 1 };

int same_stream_slots_size(const same_ctx *ctx, int32_t m, int64_t nb, size_t *bytes);

int same_stream_pass(same_ctx *ctx, void *host_states, const uint8_t *host_obs, int64_t host_ld,
                     int64_t n_cols, int64_t nb, int32_t m, float *cpts, int32_t *mb_counts,
                     int32_t *totals, uint64_t seed, uint32_t pass_id, int32_t flags, void *slots,
                     void *workspace, void *stream);

/*
 * Out-of-core passes with compact host state (Sec. 4: the data are typically
 * sparse and only model-sized state need live on the device; Sec. 6: the
 * GPU's memory, not the data, limits the problem).  The known data stay on
 * the device -- obs_dev [n][ld_dev] (1 = observed) and data_dev [n][ld_dev]
 * (the observed values, state type; latent entries ignored) for all n_cols
 * columns -- and the host keeps only the m replicas' latent states,
 * compacted: for minibatch b (columns [b*nb, min((b+1)*nb, n_cols))) and
 * node i with L latent columns in it, replica r's states at those columns in
 * ascending order are lat_host[lat_off[b*n + i] + r*L + k], k < L.  Per
 * minibatch only the compact block crosses PCIe each way (the dense
 * same_stream_pass moves every state and the obs bytes).
 *
 * same_stream_compact_layout fills lat_off[M*n + 1] (host) from obs_dev (a
 * device pass over the obs array, synchronous on `stream`) and the bytes
 * *slot_bytes of device memory the passes need (two dense minibatch slots,
 * two staging buffers of the largest compact block, offsets and scratch).
 * same_stream_pass_compact then runs one pass exactly as same_stream_pass --
 * per minibatch: upload of the compact block, expansion into the dense slot,
 * same_sweep (col_offset b*nb, sweep_id pass_id), same_counts into
 * mb_counts[b] and totals, same_sample_cpts (update_id pass_id*M + b),
 * compaction and download -- with the same results; SAME_STREAM_COUNTS_ONLY
 * uploads, expands and counts (the pre-pass).  lat_host should be pinned
 * memory for the copies to overlap the compute; nb a multiple of 4, ld_dev a
 * multiple of 4 with n_cols <= ld_dev, obs_dev 4-byte and data_dev 4-element
 * aligned, slots and workspace 256-byte aligned.  Errors as same_stream_pass.
 */
int same_stream_compact_layout(same_ctx *ctx, const uint8_t *obs_dev, int64_t ld_dev, int64_t n_cols, int64_t nb,
                               int32_t m, int64_t *lat_off, size_t *slot_bytes, void *workspace, void *stream);

int same_stream_pass_compact(same_ctx *ctx, void *lat_host, const int64_t *lat_off, const uint8_t *obs_dev,
                             const void *data_dev, int64_t ld_dev, int64_t n_cols, int64_t nb, int32_t m,
                             float *cpts, int32_t *mb_counts, int32_t *totals, uint64_t seed, uint32_t pass_id,
                             int32_t flags, void *slots, void *workspace, void *stream);

/*
 * Exponential moving sum of the counts (Sec. 4: for datasets too large to keep
 * every minibatch's counts, the counts are maintained as an exponential
 * moving sum, so memory scales with the model, not the data).
 *
 * same_counts_ema: the (parent configuration, state) histogram of the
 * minibatch (as same_counts) folded into fp64 totals [cpt_total] as
 * totals = decay * totals + new (the product rounded before the sum), with
 * decay in [0, 1].  decay = 1 - 1/M keeps the totals on the scale of the exact
 * moving sum over M minibatches (its fixed point for equal minibatches is M
 * times one minibatch's counts); decay = 0 keeps only the newest minibatch.
 *
 * same_sample_cpts_ema: the Dirichlet resample of same_sample_cpts from fp64
 * totals: g_e ~ Gamma(prior + totals[e], 1), cpts_out[e] = fp32(g_e / row sum).
 *
 * same_stream_pass_ema: same_stream_pass with the exponential moving sum in
 * place of the per-minibatch counts: per minibatch b, same_sweep,
 * same_counts_ema and same_sample_cpts_ema (update_id = pass_id * M + b); with
 * SAME_STREAM_COUNTS_ONLY only same_counts_ema (the pre-pass).  No
 * per-minibatch count storage.  Device pointers as in same_stream_pass;
 * totals is fp64, 8-byte aligned.  Errors as same_counts / same_stream_pass,
 * plus SAME_EINVAL for decay outside [0, 1].
 */
int same_counts_ema(same_ctx *ctx, const void *states, int32_t m, int64_t n_cols, int64_t ld,
                    double decay, double *totals, void *workspace, void *stream);

int same_sample_cpts_ema(same_ctx *ctx, const double *totals, float *cpts_out, uint64_t seed,
                         uint32_t update_id, void *workspace, void *stream);

int same_stream_pass_ema(same_ctx *ctx, void *host_states, const uint8_t *host_obs, int64_t host_ld,
                         int64_t n_cols, int64_t nb, int32_t m, float *cpts, double *totals,
                         double decay, uint64_t seed, uint32_t pass_id, int32_t flags, void *slots,
                         void *workspace, void *stream);

/*
 * Dense minibatch from its known entries (Sec. 4: the sampler takes a
 * typically sparse data matrix with rows = variables and columns = cases, and
 * forms m copies of the known data per minibatch).  The known entries are in
 * CSR form by node: row i holds entries [row_ptr[i], row_ptr[i+1]) of col_idx
 * (minibatch column, ascending within the row) and values (int8 or int16 like
 * the states); nnz = row_ptr[n].  obs [n][ld] is cleared, then for every
 * entry with col_idx in [0, n_cols): obs[i][j] = 1 and states[i][r][j] = value
 * for every replica r < m.  Entries with a column outside [0, n_cols) are
 * skipped; of repeated columns in a row the last entry is kept.  Latent
 * entries of states are left as they are (see same_init_latent).  All
 * pointers are device pointers owned by the caller; values must lie in
 * [0, K_i).  Errors: SAME_EINVAL for null pointers or bad sizes, SAME_EALIGN
 * for misaligned states/obs or ld, SAME_EHIP for launch failures.
 */
int same_expand_observed(same_ctx *ctx, const int64_t *row_ptr, const int32_t *col_idx,
                         const void *values, int64_t nnz, int32_t m, int64_t n_cols, int64_t ld,
                         void *states, uint8_t *obs, void *stream);

/*
 * Random initial states of the latent entries (Sec. 5.2: the sampler starts
 * from a random initialisation): for every node i, replica r < m and column
 * j < n_cols with obs[i][j] == 0, states[i][r][j] = floor(U * K_i) with U the
 * 24-bit uniform (w >> 8) * 2^-24 of word g & 3 of the Philox block at counter
 * {g >> 2, i, r | 2 << 24, 0}, g = col_offset + j (computed exactly as
 * ((w >> 8) * K_i) >> 24).  Observed entries are left as they are.  Device
 * pointers; col_offset a multiple of 4.  Errors as same_sweep's.
 */
int same_init_latent(same_ctx *ctx, void *states, const uint8_t *obs, int32_t m, int64_t n_cols,
                     int64_t ld, int64_t col_offset, uint64_t seed, void *stream);

/*
 * Held-out prediction (Sec. 6, testing phase): with the CPTs frozen, the
 * states a test entry takes over repeated sweeps estimate the probability of
 * its true state.  same_accumulate_hits adds, for every entry (i, j < n_cols)
 * with target[i][j] >= 0, the number of replicas r < m with
 * states[i][r][j] == target[i][j] to hits[i][j].  target [n][ld] has the
 * state type (-1: not a test entry; test entries must be latent in the obs
 * the sweeps use); hits [n][ld] is int32, 16-byte aligned.  Device pointers
 * owned by the caller; the caller zeroes hits before the first call.
 *
 * same_predict runs n_sweeps sweeps (same_sweep with sweep ids sweep_id0,
 * sweep_id0 + 1, ...) with cpts unchanged and accumulates the hits after each;
 * hits / (n_sweeps * m) is then the estimated probability of each test
 * entry's true state.  states is updated in place.  Errors as same_sweep's,
 * plus SAME_EINVAL for null target/hits or n_sweeps < 0 and SAME_EALIGN for
 * a misaligned target or hits.
 */
int same_accumulate_hits(same_ctx *ctx, const void *states, const void *target, int32_t m,
                         int64_t n_cols, int64_t ld, int32_t *hits, void *stream);

int same_predict(same_ctx *ctx, void *states, const uint8_t *obs, const float *cpts,
                 const void *target, int32_t m, int64_t n_cols, int64_t ld, int64_t col_offset,
                 uint64_t seed, uint32_t sweep_id0, int32_t n_sweeps, int32_t *hits,
                 void *workspace, void *stream);

/*
 * SAME annealing (Sec. 3: the replication factor m acts as a temperature and
 * can be raised during sampling to anneal the sampler): copies states (m
 * replicas) into dst (m2 >= m replicas), both in the state layout with
 * leading dimension ld.  Replica r < m is copied and replica r >= m starts as
 * a copy of replica r mod m, a valid state of the enlarged SAME joint (every
 * copy agrees with the known data); dst's padding slots follow the same rule.
 * All ld columns are copied.  After growing, the counts of the minibatch must be recomputed
 * over the m2 replicas (same_counts with zeroed previous counts, or the
 * count-only pre-pass).  Device pointers owned by the caller; states and dst
 * must not overlap.  Errors: SAME_EINVAL (null, m2 < m, overlap), SAME_EALIGN,
 * SAME_ESIZE, SAME_EHIP.
 */
int same_grow_replicas(same_ctx *ctx, const void *states, int32_t m, void *dst, int32_t m2, int64_t ld,
                       void *stream);

/*
 * Measurement of the sweep kernels.  same_kernel_timing(ctx, 1) clears the
 * totals and makes every later sweep of ctx bracket each of its kernel
 * launches with a pair of HIP events on the launch stream; (ctx, 0) clears
 * them and stops.  same_kernel_times waits for the recorded launches and
 * returns, per launch class (0: tables staged in LDS, whole or in part, 1:
 * tables in global memory, 2: 32-bit index path, 3: K > 16), the summed
 * device milliseconds, the number of kernel launches and the (node, column,
 * replica) slots those launches covered since timing was enabled, and the
 * summed device milliseconds of the colour phases (one per colour group and
 * column tile: from before the group's first launch to after its last, on
 * the caller's stream).  A group's class-1 launch runs beside its class-0
 * launch (see same_sweep), so the per-class sums count their shared time
 * twice and phase_ms is the sweep's own device time.  Host calls; the waits
 * make them unsuitable inside a captured or latency-critical sequence.
 */
typedef struct {
    double ms[4];
    int64_t launches[4];
    double phase_ms;
    int64_t phases;
    double node_samples[4];
} same_kernel_times_t;

int same_kernel_timing(same_ctx *ctx, int32_t enable);
int same_kernel_times(same_ctx *ctx, same_kernel_times_t *out);

/*
 * Replayable step graphs (Sec. 4 fuses colour groups into few large kernel
 * calls to hide the GPU's per-kernel overhead; on a small minibatch the
 * launches of one step -- table builds, one or two sweep launches per
 * colour group, counts, moving sum, Gamma and normalisation -- cost more
 * than their work).  same_step_graph captures `steps` consecutive same_step
 * calls over one resident minibatch into a HIP graph; same_graph_launch
 * replays it on `stream` with one launch.
 *
 * ids (device, two uint32 words, 4-byte aligned, caller-owned) carries the
 * sweep id (ids[0]) and the update id (ids[1]).  Step k of a replay reads
 * them on the device as they stand when it starts, runs exactly what
 * same_step(..., sweep_id = ids[0], ..., update_id = ids[1], ...) runs, and
 * then adds 1 to ids[0] and update_stride to ids[1] (a final one-thread
 * kernel).  So a replay from ids = {s, u} equals the eager calls with sweep
 * ids s, s+1, ... and update ids u, u + update_stride, ...  (update_stride M
 * gives the ids of a resident pass over M minibatches, where minibatch b's
 * graph starts from {pass, pass * M + b}).
 *
 * The graph keeps the pointers it was captured with: states, obs, cpts,
 * mb_counts, totals, ids and workspace must stay valid, and in place, while
 * it is replayed.  It holds kernel nodes and their stream-order
 * dependencies only (no memory-set or copy nodes).  Capture uses the
 * context's per-device side stream (see same_sweep), so no other call of this
 * context may run while same_step_graph runs; per-launch timing
 * (same_kernel_timing) does not apply to replays.  Replays on one device
 * must be ordered by the caller like the eager calls they stand for.
 * Errors: SAME_EINVAL (null arguments, n_cols < 1, steps outside [1, 64], a
 * launch on a device other than the capture's), SAME_EALIGN, SAME_ESIZE, and
 * the argument errors of same_step; SAME_EHIP if the capture or
 * instantiation fails.  same_graph_destroy frees the graph (null is a no-op).
 */
typedef struct same_graph same_graph;

int same_step_graph(same_ctx *ctx, void *states, const uint8_t *obs, float *cpts, int32_t m,
                    int64_t n_cols, int64_t ld, int64_t col_offset, uint64_t seed,
                    int32_t *mb_counts, int32_t *totals, uint32_t *ids, uint32_t update_stride,
                    int32_t steps, void *workspace, same_graph **out);
int same_graph_launch(same_graph *graph, void *stream);
void same_graph_destroy(same_graph *graph);

/* Message for the calling thread's last failed call ("" if none). */
const char *same_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SAME_H */
