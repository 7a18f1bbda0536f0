/*
 * Reference oracle for SAME Gibbs sampling on discrete Bayesian networks
 * (Seita, Chen & Canny, "Fast Parallel SAME Gibbs Sampling on General
 * Discrete Bayesian Networks", arXiv 1511.06416).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, double-precision CPU
 * statement of what one SAME Gibbs sweep computes.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark load it; the product
 * library never links, includes or calls it, and it shares no code, header,
 * table or constant generator with the product.
 *
 * What it computes, and where the paper defines it:
 *   - the problem: sample latent states Z and CPTs Theta from P(Z, Theta | D)
 *     for a discrete Bayesian network of known structure with partially
 *     observed data; Z are multinomial, Theta Dirichlet (Sec. 1);
 *   - SAME: m latent copies of every data case tied to one Theta (Sec. 3, Eq. 1);
 *   - chromatic Gibbs: colour the moralized graph, visit colour groups in
 *     order; this equals a sequential-scan Gibbs sampler over the permutation
 *     "colour 1 nodes, then colour 2 nodes, ..." (Sec. 4, chromatic
 *     partitioning paragraph).  The oracle therefore IS that sequential scan;
 *   - per-minibatch counts and their exact moving sum over the M minibatches
 *     (Sec. 4, minibatch paragraph);
 *   - Dirichlet resampling of the CPTs from counts plus prior (Sec. 4, SAME
 *     paragraph).
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - CPT layout: node i owns entries [off_i, off_i + R_i*K_i), R_i = prod of
 *     parent cardinalities; row u = sum_j x_{pa_j} * stride_j in the listed
 *     parent order with the LAST parent fastest; entry = off_i + u*K_i + k.
 *   - Colouring: first-fit greedy over a Kahn topological order that always
 *     takes the smallest ready node id; each node gets the smallest colour not
 *     used by an already coloured moral neighbour; then the groups are
 *     balanced by single-node moves that keep the colouring proper
 *     (balance_colouring).
 *   - Random numbers: Philox4x32-10 (Salmon, Moraes, Dror & Shaw, SC'11).
 *     Gibbs draw for node i, replica r, global column g, sweep s uses word
 *     (r & 3) of Philox(ctr = {g, i, (r>>2) | (0<<24), s}, key = {seed_lo, seed_hi});
 *     U24(w) = (w >> 8) * 2^-24.
 *   - Draw rule (inverse CDF): w_k = exp(l_k - max l), S_k = w_0 + ... + w_k,
 *     Z = S_{K-1}; pick the smallest k with u*Z < S_k, else the largest k with
 *     w_k > 0.  A draw is "flagged" when u lies within 1e-6 of a CDF boundary
 *     S_k/Z, k < K-1.
 *   - CPT entries are used as max(theta, FLT_MIN), so a zero entry is a very
 *     small positive weight rather than -inf.
 *   - Dirichlet prior: theta_row ~ Dir(alpha + T_row), T the moving-sum counts
 *     summed over the m replicas.
 *   - Gamma variates: Marsaglia & Tsang (ACM TOMS 26(3), 2000) with the
 *     shape<1 boost Gamma(a) = Gamma(a+1) * U^(1/a); attempt t of entry e at
 *     update q uses Philox(ctr = {e, t, 1<<24, q}); normal by Box-Muller from
 *     words 0 and 1, acceptance uniform from word 2, boost uniform from word 3.
 */
#include <float.h>
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_OK 0
#define OR_EINVAL -1
#define OR_EGRAPH -2
#define OR_ECARD -3
#define OR_ESIZE -4
#define OR_ENOMEM -5

#define TAG_GIBBS 0u
#define TAG_GAMMA 1u
#define GAMMA_MAX_ATTEMPTS 256
#define FLAG_BAND 1e-6

/* ------------------------------------------------------------------ */
/* Philox4x32-10, written from its published definition (SC'11).       */
/* ------------------------------------------------------------------ */

static void mulhilo32(uint32_t a, uint32_t b, uint32_t *hi, uint32_t *lo) {
    uint64_t p = (uint64_t)a * (uint64_t)b;
    *hi = (uint32_t)(p >> 32);
    *lo = (uint32_t)p;
}

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint32_t hi0, lo0, hi1, lo1;
        mulhilo32(M0, c0, &hi0, &lo0);
        mulhilo32(M1, c2, &hi1, &lo1);
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += W0;
        k1 += W1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

static uint32_t philox_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                            int word) {
    uint32_t ctr[4] = {c0, c1, c2, c3};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    return out[word];
}

/*
 * The Gibbs uniform of one (node, replica, global column, sweep): word r & 3
 * of the block at counter {g, node, (r >> 2) | TAG_GIBBS << 24, sweep}, so
 * that one block serves four replicas of one column.
 */
double oracle_gibbs_uniform(uint64_t seed, int32_t node, int32_t replica, int64_t gcol,
                            uint32_t sweep_id) {
    uint32_t w = philox_word(seed, (uint32_t)gcol, (uint32_t)node,
                             ((uint32_t)replica >> 2) | (TAG_GIBBS << 24), sweep_id, (int)(replica & 3));
    return (double)(w >> 8) * (1.0 / 16777216.0);
}

/* ------------------------------------------------------------------ */
/* Graph: validation, topological order, moral graph, colouring,      */
/* CPT layout (Sec. 1 CPT definition; Sec. 4 chromatic partitioning).  */
/* ------------------------------------------------------------------ */

typedef struct {
    int32_t n;
    const int32_t *pptr, *pidx, *card;
    int64_t *off;     /* [n+1] CPT offsets */
    int64_t *rows;    /* [n]   R_i */
    int64_t *stride;  /* [nnz] stride of parent slot j in node i's row index */
    int32_t *cptr;    /* [n+1] children CSR */
    int32_t *cidx;    /* [nnz] child node */
    int32_t *cslot;   /* [nnz] slot of the parent in that child's parent list */
} graph_t;

static void graph_free(graph_t *g) {
    free(g->off); free(g->rows); free(g->stride);
    free(g->cptr); free(g->cidx); free(g->cslot);
    memset(g, 0, sizeof(*g));
}

/* Validates the DAG and fills the CPT layout and children lists. */
static int graph_build(graph_t *g, int32_t n, const int32_t *pptr, const int32_t *pidx,
                       const int32_t *card) {
    memset(g, 0, sizeof(*g));
    if (n <= 0 || !pptr || !card) return OR_EINVAL;
    if (pptr[0] != 0) return OR_EGRAPH;
    for (int32_t i = 0; i < n; ++i)
        if (pptr[i + 1] < pptr[i]) return OR_EGRAPH;
    int32_t nnz = pptr[n];
    if (nnz > 0 && !pidx) return OR_EINVAL;
    for (int32_t i = 0; i < n; ++i) {
        if (card[i] < 2 || card[i] > 32767) return OR_ECARD;
        for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) {
            int32_t p = pidx[a];
            if (p < 0 || p >= n || p == i) return OR_EGRAPH;
            for (int32_t b = pptr[i]; b < a; ++b)
                if (pidx[b] == p) return OR_EGRAPH;
        }
    }
    g->n = n; g->pptr = pptr; g->pidx = pidx; g->card = card;
    g->off = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
    g->rows = (int64_t *)calloc((size_t)n, sizeof(int64_t));
    g->stride = (int64_t *)calloc((size_t)nnz + 1, sizeof(int64_t));
    g->cptr = (int32_t *)calloc((size_t)n + 1, sizeof(int32_t));
    g->cidx = (int32_t *)calloc((size_t)nnz + 1, sizeof(int32_t));
    g->cslot = (int32_t *)calloc((size_t)nnz + 1, sizeof(int32_t));
    if (!g->off || !g->rows || !g->stride || !g->cptr || !g->cidx || !g->cslot) {
        graph_free(g);
        return OR_ENOMEM;
    }
    for (int32_t i = 0; i < n; ++i) {
        int64_t r = 1;
        for (int32_t a = pptr[i + 1] - 1; a >= pptr[i]; --a) { /* last parent fastest */
            g->stride[a] = r;
            r *= card[pidx[a]];
            if (r > ((int64_t)1 << 31)) { graph_free(g); return OR_ESIZE; }
        }
        g->rows[i] = r;
        g->off[i + 1] = g->off[i] + r * card[i];
        if (g->off[i + 1] >= ((int64_t)1 << 31)) { graph_free(g); return OR_ESIZE; }
    }
    /* children lists, children of each node in ascending child id */
    for (int32_t h = 0; h < n; ++h)
        for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) g->cptr[pidx[a] + 1]++;
    for (int32_t i = 0; i < n; ++i) g->cptr[i + 1] += g->cptr[i];
    int32_t *fill = (int32_t *)calloc((size_t)n, sizeof(int32_t));
    if (!fill) { graph_free(g); return OR_ENOMEM; }
    for (int32_t h = 0; h < n; ++h)
        for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) {
            int32_t p = pidx[a];
            int32_t pos = g->cptr[p] + fill[p]++;
            g->cidx[pos] = h;
            g->cslot[pos] = a - pptr[h];
        }
    free(fill);
    /* cycle check with Kahn's algorithm */
    int32_t *indeg = (int32_t *)calloc((size_t)n, sizeof(int32_t));
    char *done = (char *)calloc((size_t)n, 1);
    if (!indeg || !done) { free(indeg); free(done); graph_free(g); return OR_ENOMEM; }
    for (int32_t i = 0; i < n; ++i) indeg[i] = pptr[i + 1] - pptr[i];
    int32_t emitted = 0;
    for (;;) {
        int32_t v = -1;
        for (int32_t i = 0; i < n; ++i)
            if (!done[i] && indeg[i] == 0) { v = i; break; }
        if (v < 0) break;
        done[v] = 1;
        emitted++;
        for (int32_t a = g->cptr[v]; a < g->cptr[v + 1]; ++a) indeg[g->cidx[a]]--;
    }
    free(indeg); free(done);
    if (emitted != n) { graph_free(g); return OR_EGRAPH; }
    return OR_OK;
}

/*
 * Balancing of a proper colouring (Sec. 4 asks for colour groups of balanced
 * size): repeatedly move one node from a larger group to a group at least two
 * smaller, when none of its moral neighbours is in that group (so the
 * colouring stays proper).  Which move: groups by decreasing size (ties:
 * lower colour first), inside a group nodes by ascending id, targets by
 * increasing size (ties: lower colour first); the first valid move is made
 * and the search starts again.  Every move lowers the sum of squared group
 * sizes, so this ends; no group empties.  adj is the dense moral adjacency.
 */
static void balance_colouring(int32_t n, const char *adj, int32_t ncol, int32_t *col) {
    int32_t *size = (int32_t *)calloc((size_t)ncol, sizeof(int32_t));
    int32_t *by_desc = (int32_t *)calloc((size_t)ncol, sizeof(int32_t));
    int32_t *by_asc = (int32_t *)calloc((size_t)ncol, sizeof(int32_t));
    for (;;) {
        for (int32_t c = 0; c < ncol; ++c) size[c] = 0;
        for (int32_t v = 0; v < n; ++v) size[col[v]]++;
        /* the two orders, by insertion sort */
        for (int32_t c = 0; c < ncol; ++c) by_desc[c] = by_asc[c] = c;
        for (int32_t i = 1; i < ncol; ++i)
            for (int32_t j = i; j > 0; --j) {
                int32_t x = by_desc[j - 1], y = by_desc[j];
                if (size[y] > size[x] || (size[y] == size[x] && y < x)) {
                    by_desc[j - 1] = y; by_desc[j] = x;
                }
                x = by_asc[j - 1]; y = by_asc[j];
                if (size[y] < size[x] || (size[y] == size[x] && y < x)) {
                    by_asc[j - 1] = y; by_asc[j] = x;
                }
            }
        int moved = 0;
        for (int32_t ia = 0; ia < ncol && !moved; ++ia) {
            int32_t a = by_desc[ia];
            for (int32_t v = 0; v < n && !moved; ++v) {
                if (col[v] != a) continue;
                for (int32_t ib = 0; ib < ncol; ++ib) {
                    int32_t b = by_asc[ib];
                    if (size[b] + 1 >= size[a]) break;
                    int clash = 0;
                    for (int32_t w = 0; w < n; ++w)
                        if (adj[(size_t)v * n + w] && col[w] == b) { clash = 1; break; }
                    if (!clash) { col[v] = b; moved = 1; break; }
                }
            }
        }
        if (!moved) break;
    }
    free(size); free(by_desc); free(by_asc);
}

/*
 * Topological order (Kahn, smallest ready id first), moral graph and the
 * colouring: first-fit over the topological order, then (balance != 0) the
 * balancing above.  Outputs: cpt_off[n+1], topo[n], color[n], *n_colors.
 * Any output pointer may be NULL.
 */
int oracle_graph_ex(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                    int32_t balance, int64_t *cpt_off, int32_t *topo, int32_t *color, int32_t *n_colors);

int oracle_graph(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                 int64_t *cpt_off, int32_t *topo, int32_t *color, int32_t *n_colors) {
    return oracle_graph_ex(n, pptr, pidx, card, 1, cpt_off, topo, color, n_colors);
}

int oracle_graph_ex(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                    int32_t balance, int64_t *cpt_off, int32_t *topo, int32_t *color, int32_t *n_colors) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    if (cpt_off)
        for (int32_t i = 0; i <= n; ++i) cpt_off[i] = g.off[i];

    /* moral graph: parent-child edges plus edges between co-parents */
    char *adj = (char *)calloc((size_t)n * (size_t)n, 1);
    int32_t *order = (int32_t *)calloc((size_t)n, sizeof(int32_t));
    int32_t *indeg = (int32_t *)calloc((size_t)n, sizeof(int32_t));
    int32_t *col = (int32_t *)calloc((size_t)n, sizeof(int32_t));
    char *done = (char *)calloc((size_t)n, 1);
    char *used = (char *)calloc((size_t)n + 1, 1);
    if (!adj || !order || !indeg || !col || !done || !used) {
        free(adj); free(order); free(indeg); free(col); free(done); free(used);
        graph_free(&g);
        return OR_ENOMEM;
    }
    for (int32_t h = 0; h < n; ++h)
        for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) {
            int32_t p = pidx[a];
            adj[(size_t)p * n + h] = adj[(size_t)h * n + p] = 1;
            for (int32_t b = pptr[h]; b < pptr[h + 1]; ++b) {
                int32_t q = pidx[b];
                if (q != p) adj[(size_t)p * n + q] = adj[(size_t)q * n + p] = 1;
            }
        }
    for (int32_t i = 0; i < n; ++i) indeg[i] = pptr[i + 1] - pptr[i];
    for (int32_t t = 0; t < n; ++t) {
        int32_t v = -1;
        for (int32_t i = 0; i < n; ++i)
            if (!done[i] && indeg[i] == 0) { v = i; break; }
        done[v] = 1;
        order[t] = v;
        for (int32_t a = g.cptr[v]; a < g.cptr[v + 1]; ++a) indeg[g.cidx[a]]--;
    }
    for (int32_t i = 0; i < n; ++i) col[i] = -1;
    int32_t ncol = 0;
    for (int32_t t = 0; t < n; ++t) {
        int32_t v = order[t];
        memset(used, 0, (size_t)n + 1);
        for (int32_t w = 0; w < n; ++w)
            if (adj[(size_t)v * n + w] && col[w] >= 0) used[col[w]] = 1;
        int32_t c = 0;
        while (used[c]) c++;
        col[v] = c;
        if (c + 1 > ncol) ncol = c + 1;
    }
    if (balance) balance_colouring(n, adj, ncol, col);
    if (topo) memcpy(topo, order, sizeof(int32_t) * (size_t)n);
    if (color) memcpy(color, col, sizeof(int32_t) * (size_t)n);
    if (n_colors) *n_colors = ncol;
    free(adj); free(order); free(indeg); free(col); free(done); free(used);
    graph_free(&g);
    return OR_OK;
}

/* Moral-graph adjacency as a dense n*n byte matrix (tests only). */
int oracle_moral(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                 uint8_t *adj) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    memset(adj, 0, (size_t)n * (size_t)n);
    for (int32_t h = 0; h < n; ++h)
        for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) {
            int32_t p = pidx[a];
            adj[(size_t)p * n + h] = adj[(size_t)h * n + p] = 1;
            for (int32_t b = pptr[h]; b < pptr[h + 1]; ++b) {
                int32_t q = pidx[b];
                if (q != p) adj[(size_t)p * n + q] = adj[(size_t)q * n + p] = 1;
            }
        }
    graph_free(&g);
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Markov-blanket conditional and the inverse-CDF draw.                */
/* ------------------------------------------------------------------ */

static double log_entry(const float *theta, int64_t e) {
    double t = (double)theta[e];
    if (t < (double)FLT_MIN) t = (double)FLT_MIN;
    return log(t);
}

/* State of node v in the chain; the chain is addressed by base + v*vstride. */
static int32_t state_at(const void *states, int32_t state_bytes, int64_t idx) {
    if (state_bytes == 1) return (int32_t)((const int8_t *)states)[idx];
    return (int32_t)((const int16_t *)states)[idx];
}

static int64_t row_of(const graph_t *g, int32_t node, const void *states, int32_t sb,
                      int64_t base, int64_t vstride) {
    int64_t u = 0;
    for (int32_t a = g->pptr[node]; a < g->pptr[node + 1]; ++a)
        u += (int64_t)state_at(states, sb, base + (int64_t)g->pidx[a] * vstride) * g->stride[a];
    return u;
}

/*
 * Log of the unnormalised full conditional of node i for each state k
 * (product of the node's own CPT entry and the CPT entries of its children,
 * i.e. the factors of the joint that mention x_i).  The chain's state of node
 * v is states[base + v*vstride].
 */
static void log_conditional(const graph_t *g, const float *theta, int32_t i, const void *states,
                            int32_t sb, int64_t base, int64_t vstride, double *l) {
    int32_t K = g->card[i];
    int64_t u = row_of(g, i, states, sb, base, vstride);
    for (int32_t k = 0; k < K; ++k) l[k] = log_entry(theta, g->off[i] + u * K + k);
    for (int32_t a = g->cptr[i]; a < g->cptr[i + 1]; ++a) {
        int32_t h = g->cidx[a];
        int32_t slot = g->cslot[a];
        int64_t s = g->stride[g->pptr[h] + slot];
        int64_t uh = row_of(g, h, states, sb, base, vstride);
        int32_t xi = state_at(states, sb, base + (int64_t)i * vstride);
        int64_t uh_minus_i = uh - (int64_t)xi * s;
        int32_t xh = state_at(states, sb, base + (int64_t)h * vstride);
        int32_t Kh = g->card[h];
        for (int32_t k = 0; k < K; ++k)
            l[k] += log_entry(theta, g->off[h] + (uh_minus_i + (int64_t)k * s) * Kh + xh);
    }
}

/*
 * Inverse-CDF draw from non-negative weights w[K]: S_k = w_0 + ... + w_k,
 * Z = S_{K-1}; the smallest k with u*Z < S_k, else the largest k with w_k > 0.
 * Writes the normalised weights into p (may be NULL) and the boundary flag.
 */
static int32_t draw_from_weights(const double *w, int32_t K, double u, double *p, int *flagged) {
    if (K < 1) return -1;
    double Sbuf[64];
    double *S = K <= 64 ? Sbuf : (double *)malloc(sizeof(double) * (size_t)K);
    double acc = 0.0;
    for (int32_t k = 0; k < K; ++k) {
        acc += w[k];
        S[k] = acc;
    }
    double Z = S[K - 1];
    int32_t pick = -1;
    for (int32_t k = 0; k < K; ++k)
        if (u * Z < S[k]) { pick = k; break; }
    if (pick < 0)
        for (int32_t k = K - 1; k >= 0; --k)
            if (w[k] > 0.0) { pick = k; break; }
    if (flagged) {
        int f = 0;
        for (int32_t k = 0; k < K - 1; ++k)
            if (fabs(u - S[k] / Z) < FLAG_BAND) f = 1;
        *flagged = f;
    }
    if (p)
        for (int32_t k = 0; k < K; ++k) p[k] = w[k] / Z;
    if (K > 64) free(S);
    return pick;
}

/* Weights w_k = exp(l_k - max l) from log weights, then the draw above. */
static int32_t draw_from_logits(const double *l, int32_t K, double u, double *p, int *flagged) {
    if (K < 1) return -1;
    double mx = l[0];
    for (int32_t k = 1; k < K; ++k)
        if (l[k] > mx) mx = l[k];
    double wbuf[64];
    double *w = K <= 64 ? wbuf : (double *)malloc(sizeof(double) * (size_t)K);
    for (int32_t k = 0; k < K; ++k) w[k] = exp(l[k] - mx);
    int32_t pick = draw_from_weights(w, K, u, p, flagged);
    if (K > 64) free(w);
    return pick;
}

/*
 * Normalised full conditional of `node` for one chain given as a state
 * vector x[n] (int32).  Returns K or a negative error.
 */
int oracle_conditional(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                       const float *theta, const int32_t *x, int32_t node, double *p_out) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    if (node < 0 || node >= n) { graph_free(&g); return OR_EINVAL; }
    int16_t *xs = (int16_t *)malloc(sizeof(int16_t) * (size_t)n);
    double *l = (double *)malloc(sizeof(double) * (size_t)card[node]);
    if (!xs || !l) { free(xs); free(l); graph_free(&g); return OR_ENOMEM; }
    for (int32_t v = 0; v < n; ++v) xs[v] = (int16_t)x[v];
    log_conditional(&g, theta, node, xs, 2, 0, 1, l);
    draw_from_logits(l, card[node], 0.0, p_out, NULL);
    int32_t K = card[node];
    free(xs); free(l);
    graph_free(&g);
    return K;
}

/*
 * The same normalised conditional for `count` state vectors X[count][n]
 * (int32), into P[count][K_node]: the graph is built once for all of them.
 */
int oracle_conditionals(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                        const float *theta, const int32_t *X, int64_t count, int32_t node, double *P) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    if (node < 0 || node >= n) { graph_free(&g); return OR_EINVAL; }
    const int32_t K = card[node];
    int16_t *xs = (int16_t *)malloc(sizeof(int16_t) * (size_t)n);
    double *l = (double *)malloc(sizeof(double) * (size_t)K);
    if (!xs || !l) { free(xs); free(l); graph_free(&g); return OR_ENOMEM; }
    for (int64_t c = 0; c < count; ++c) {
        for (int32_t v = 0; v < n; ++v) xs[v] = (int16_t)X[c * n + v];
        log_conditional(&g, theta, node, xs, 2, 0, 1, l);
        draw_from_logits(l, K, 0.0, P + c * K, NULL);
    }
    free(xs); free(l);
    graph_free(&g);
    return K;
}

/* The draw rule alone, for hand-built (weights, u) cases.  Weights must be >= 0. */
int32_t oracle_draw(const double *weights, int32_t K, double u, int32_t *flagged) {
    int f = 0;
    int32_t pick = draw_from_weights(weights, K, u, NULL, &f);
    if (flagged) *flagged = f;
    return pick;
}

/* ------------------------------------------------------------------ */
/* One SAME Gibbs sweep over one minibatch (Sec. 3 Eq. 1; Sec. 4).      */
/* ------------------------------------------------------------------ */

/*
 * states: [n][m][ld] (int8 when state_bytes == 1, int16 when 2), updated in
 * place; obs: [n][ld], 1 = observed.  Column j < n_cols is global column
 * col_offset + j.  color[n] gives the colour of every node; colours are
 * visited in ascending order and, inside a colour, nodes in ascending id,
 * which is the sequential scan the colour-parallel sampler equals.
 * flags (nullable): [n][m][ld] bytes, set to 1 for flagged draws, 0 for other
 * latent draws, untouched for observed entries.
 * probs (nullable): conditionals for columns [win_begin, win_begin + win):
 * probs[((i*m + r)*win + (j - win_begin))*kmax + k]; observed entries are
 * left untouched.
 * Returns the number of latent draws (>= 0) or a negative error.
 */
int64_t oracle_sweep(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                     const float *theta, const int32_t *color, int32_t state_bytes, void *states,
                     const uint8_t *obs, int32_t m, int64_t n_cols, int64_t ld, int64_t col_offset,
                     uint64_t seed, uint32_t sweep_id, uint8_t *flags, int64_t win_begin,
                     int64_t win, double *probs, int32_t kmax, int32_t n_threads) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    if (state_bytes != 1 && state_bytes != 2) { graph_free(&g); return OR_EINVAL; }
    if (m < 1 || n_cols < 0 || ld < n_cols || !color) { graph_free(&g); return OR_EINVAL; }
    if (probs && kmax < 1) { graph_free(&g); return OR_EINVAL; }
    int32_t ncol = 0;
    for (int32_t i = 0; i < n; ++i) {
        if (color[i] < 0) { graph_free(&g); return OR_EINVAL; }
        if (color[i] + 1 > ncol) ncol = color[i] + 1;
    }
    int32_t Kmax = 0;
    for (int32_t i = 0; i < n; ++i)
        if (card[i] > Kmax) Kmax = card[i];
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
    int64_t draws = 0;
    const int64_t vstride = (int64_t)m * ld; /* distance between nodes of one chain */
    for (int32_t c = 0; c < ncol; ++c) {
        for (int32_t i = 0; i < n; ++i) {
            if (color[i] != c) continue;
            int32_t K = card[i];
            int64_t local = 0;
#pragma omp parallel reduction(+ : local)
            {
            double *l = (double *)malloc(sizeof(double) * (size_t)Kmax);
            double *p = (double *)malloc(sizeof(double) * (size_t)Kmax);
#pragma omp for schedule(static)
            for (int64_t j = 0; j < n_cols; ++j) {
                if (obs[(int64_t)i * ld + j]) continue;
                for (int32_t r = 0; r < m; ++r) {
                    int64_t base = (int64_t)r * ld + j;
                    log_conditional(&g, theta, i, states, state_bytes, base, vstride, l);
                    double u = oracle_gibbs_uniform(seed, i, r, col_offset + j, sweep_id);
                    int f = 0;
                    int32_t x = draw_from_logits(l, K, u, p, &f);
                    int64_t at = (int64_t)i * vstride + base;
                    if (state_bytes == 1) ((int8_t *)states)[at] = (int8_t)x;
                    else ((int16_t *)states)[at] = (int16_t)x;
                    if (flags) flags[at] = (uint8_t)f;
                    if (probs && j >= win_begin && j < win_begin + win) {
                        double *dst = probs + (((int64_t)i * m + r) * win + (j - win_begin)) * kmax;
                        for (int32_t k = 0; k < K && k < kmax; ++k) dst[k] = p[k];
                    }
                    local++;
                }
            }
            free(l);
            free(p);
            }
            draws += local;
        }
    }
    graph_free(&g);
    return draws;
}

/* ------------------------------------------------------------------ */
/* Sufficient statistics (Sec. 4): histogram of (parent row, state).    */
/* ------------------------------------------------------------------ */

/* counts[cpt_total] is overwritten with the counts of states[n][m][ld] over
 * columns j < n_cols and all replicas; observed and sampled entries alike. */
int oracle_counts(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                  int32_t state_bytes, const void *states, int32_t m, int64_t n_cols, int64_t ld,
                  int64_t *counts, int32_t n_threads) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    if (state_bytes != 1 && state_bytes != 2) { graph_free(&g); return OR_EINVAL; }
    if (m < 1 || n_cols < 0 || ld < n_cols) { graph_free(&g); return OR_EINVAL; }
#ifdef _OPENMP
    if (n_threads > 0) omp_set_num_threads(n_threads);
#else
    (void)n_threads;
#endif
    memset(counts, 0, sizeof(int64_t) * (size_t)g.off[n]);
    const int64_t vstride = (int64_t)m * ld;
#pragma omp parallel for schedule(dynamic, 1)
    for (int32_t i = 0; i < n; ++i) {
        int32_t K = card[i];
        for (int32_t r = 0; r < m; ++r)
            for (int64_t j = 0; j < n_cols; ++j) {
                int64_t base = (int64_t)r * ld + j;
                int64_t u = row_of(&g, i, states, state_bytes, base, vstride);
                int32_t x = state_at(states, state_bytes, (int64_t)i * vstride + base);
                counts[g.off[i] + u * K + x] += 1;
            }
    }
    graph_free(&g);
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Gamma and Dirichlet (Sec. 4: counts plus prior are the Dirichlet     */
/* parameters from which the CPTs are sampled).                         */
/* ------------------------------------------------------------------ */

static double u24_open0(uint32_t w) { return ((double)(w >> 8) + 1.0) * (1.0 / 16777216.0); }
static double u24(uint32_t w) { return (double)(w >> 8) * (1.0 / 16777216.0); }

/* One Gamma(shape, 1) variate for flat CPT entry `entry` at update `update_id`. */
double oracle_gamma(double shape, uint64_t seed, uint32_t entry, uint32_t update_id,
                    int32_t *attempts_out) {
    const double two_pi = 6.283185307179586476925286766559;
    int boost = shape < 1.0;
    double b = boost ? shape + 1.0 : shape;
    double d = b - 1.0 / 3.0;
    double c = 1.0 / sqrt(9.0 * d);
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    for (int32_t t = 0; t < GAMMA_MAX_ATTEMPTS; ++t) {
        uint32_t ctr[4] = {entry, (uint32_t)t, TAG_GAMMA << 24, update_id};
        uint32_t w[4];
        oracle_philox4x32_10(ctr, key, w);
        double u1 = u24_open0(w[0]);
        double u2 = u24(w[1]);
        double z = sqrt(-2.0 * log(u1)) * cos(two_pi * u2);
        double v = 1.0 + c * z;
        if (v <= 0.0) continue;
        v = v * v * v;
        double ua = u24_open0(w[2]);
        if (log(ua) < 0.5 * z * z + d - d * v + d * log(v)) {
            double gval = d * v;
            if (boost) gval *= pow(u24_open0(w[3]), 1.0 / shape);
            if (attempts_out) *attempts_out = t + 1;
            return gval;
        }
    }
    if (attempts_out) *attempts_out = GAMMA_MAX_ATTEMPTS;
    return d;
}

/*
 * theta_out[e] = fp32( g_e / sum of g over e's CPT row ), g_e ~ Gamma(alpha +
 * totals[e]).  A row whose Gamma variates all underflow to zero becomes
 * uniform.  gamma_out (nullable) receives the fp64 variates.  totals are
 * integer counts (oracle_dirichlet) or fp64 moving sums (oracle_dirichlet_f64).
 */
static int dirichlet_impl(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                          const int64_t *itot, const double *dtot, double alpha, uint64_t seed,
                          uint32_t update_id, float *theta_out, double *gamma_out);

int oracle_dirichlet(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                     const int64_t *totals, double alpha, uint64_t seed, uint32_t update_id,
                     float *theta_out, double *gamma_out) {
    return dirichlet_impl(n, pptr, pidx, card, totals, NULL, alpha, seed, update_id, theta_out, gamma_out);
}

int oracle_dirichlet_f64(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                         const double *totals, double alpha, uint64_t seed, uint32_t update_id,
                         float *theta_out, double *gamma_out) {
    return dirichlet_impl(n, pptr, pidx, card, NULL, totals, alpha, seed, update_id, theta_out, gamma_out);
}

static int dirichlet_impl(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                          const int64_t *itot, const double *dtot, double alpha, uint64_t seed,
                          uint32_t update_id, float *theta_out, double *gamma_out) {
    graph_t g;
    int rc = graph_build(&g, n, pptr, pidx, card);
    if (rc) return rc;
    if (!(alpha > 0.0)) { graph_free(&g); return OR_EINVAL; }
    double *gv = (double *)malloc(sizeof(double) * (size_t)g.off[n]);
    if (!gv) { graph_free(&g); return OR_ENOMEM; }
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < g.off[n]; ++e)
        gv[e] = oracle_gamma(alpha + (itot ? (double)itot[e] : dtot[e]), seed, (uint32_t)e, update_id, NULL);
    for (int32_t i = 0; i < n; ++i) {
        int32_t K = card[i];
        for (int64_t u = 0; u < g.rows[i]; ++u) {
            int64_t e0 = g.off[i] + u * K;
            double s = 0.0;
            for (int32_t k = 0; k < K; ++k) s += gv[e0 + k];
            for (int32_t k = 0; k < K; ++k)
                theta_out[e0 + k] = (float)(s > 0.0 ? gv[e0 + k] / s : 1.0 / K);
        }
    }
    if (gamma_out) memcpy(gamma_out, gv, sizeof(double) * (size_t)g.off[n]);
    free(gv);
    graph_free(&g);
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Data ingest: the (typically sparse) node x case matrix of known     */
/* entries (Sec. 4) and the random initial latent states (Sec. 5.2).   */
/* ------------------------------------------------------------------ */

#define TAG_INIT 2u

static void put_state(void *states, int32_t state_bytes, int64_t idx, int32_t v) {
    if (state_bytes == 1) ((int8_t *)states)[idx] = (int8_t)v;
    else ((int16_t *)states)[idx] = (int16_t)v;
}

/*
 * Dense minibatch from its known entries (Sec. 4: the sampler takes a
 * typically sparse matrix with rows = variables and columns = cases, and forms
 * m copies of the known data).  Row i of the sparse matrix holds entries
 * [row_ptr[i], row_ptr[i+1]) with column indices col_idx (relative to the
 * minibatch) and values (state_bytes: 1 = int8, 2 = int16).  obs[n][ld] is set
 * to 0, then for every entry with a column in [0, n_cols): obs[i][j] = 1 and
 * states[i][r][j] = value for r < m.  A row listing a column twice keeps the
 * later entry.  Latent entries of states are not touched.
 */
int oracle_expand(int32_t n, int64_t n_cols, int32_t m, int64_t ld, const int64_t *row_ptr,
                  const int32_t *col_idx, const void *values, int32_t state_bytes, void *states,
                  uint8_t *obs) {
    if (n <= 0 || m < 1 || n_cols < 0 || ld < n_cols || (state_bytes != 1 && state_bytes != 2))
        return OR_EINVAL;
    memset(obs, 0, (size_t)n * (size_t)ld);
    for (int32_t i = 0; i < n; ++i) {
        for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
            int64_t j = col_idx[e];
            if (j < 0 || j >= n_cols) continue;
            int32_t v = state_bytes == 1 ? ((const int8_t *)values)[e] : ((const int16_t *)values)[e];
            obs[(int64_t)i * ld + j] = 1;
            for (int32_t r = 0; r < m; ++r) put_state(states, state_bytes, ((int64_t)i * m + r) * ld + j, v);
        }
    }
    return OR_OK;
}

/*
 * Random initial latent states (Sec. 5.2: the sampler starts from a random
 * initialisation).  For node i, replica r and column j < n_cols with
 * obs[i][j] == 0: states[i][r][j] = floor(U * K_i), U = (w >> 8) * 2^-24 with
 * w word (g & 3) of Philox(ctr = {g >> 2, i, r | (2 << 24), 0}),
 * g = col_offset + j.  floor(U * K_i) is formed exactly as ((w >> 8) * K_i) >> 24.
 */
int oracle_init_latent(int32_t n, const int32_t *card, int64_t n_cols, int32_t m, int64_t ld,
                       int64_t col_offset, uint64_t seed, int32_t state_bytes, void *states,
                       const uint8_t *obs) {
    if (n <= 0 || m < 1 || n_cols < 0 || ld < n_cols || (state_bytes != 1 && state_bytes != 2))
        return OR_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        for (int32_t r = 0; r < m; ++r)
            for (int64_t j = 0; j < n_cols; ++j) {
                if (obs[(int64_t)i * ld + j]) continue;
                int64_t g = col_offset + j;
                uint32_t w = philox_word(seed, (uint32_t)(g >> 2), (uint32_t)i,
                                         (uint32_t)r | (TAG_INIT << 24), 0u, (int)(g & 3));
                int32_t v = (int32_t)(((uint64_t)(w >> 8) * (uint64_t)card[i]) >> 24);
                put_state(states, state_bytes, ((int64_t)i * m + r) * ld + j, v);
            }
    return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Held-out prediction (Sec. 6).                                       */
/* ------------------------------------------------------------------ */

static int32_t get_state(const void *a, int32_t state_bytes, int64_t idx) {
    return state_bytes == 1 ? ((const int8_t *)a)[idx] : ((const int16_t *)a)[idx];
}

/*
 * With the CPTs frozen, the states a test entry takes over n sweeps estimate
 * the probability of its true state (Sec. 6, testing phase).  One call adds,
 * for every entry (i, j < n_cols) with target[i][j] >= 0 (target [n][ld] in
 * the state type, -1 = not a test entry), the number of replicas r < m with
 * states[i][r][j] == target[i][j] to hits[i][j] (int32 [n][ld]).
 */
int oracle_accumulate_hits(int32_t n, int64_t n_cols, int32_t m, int64_t ld, int32_t state_bytes,
                           const void *states, const void *target, int32_t *hits) {
    if (n <= 0 || m < 1 || n_cols < 0 || ld < n_cols || (state_bytes != 1 && state_bytes != 2))
        return OR_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n_cols; ++j) {
            int32_t t = get_state(target, state_bytes, (int64_t)i * ld + j);
            if (t < 0) continue;
            for (int32_t r = 0; r < m; ++r)
                if (get_state(states, state_bytes, ((int64_t)i * m + r) * ld + j) == t) hits[(int64_t)i * ld + j] += 1;
        }
    return OR_OK;
}

/*
 * Exponential moving sum of the counts (Sec. 4 footnote: for datasets whose
 * per-minibatch counts are not kept): totals[e] = decay * totals[e] + newc[e]
 * in fp64, the product rounded before the sum.
 */
void oracle_ema(int64_t total, double decay, const int64_t *newc, double *totals) {
    for (int64_t e = 0; e < total; ++e) {
        double p = decay * totals[e];
        totals[e] = p + (double)newc[e];
    }
}

/* ------------------------------------------------------------------ */
/* SAME annealing (Sec. 3): more replicas as the sampler proceeds.      */
/* ------------------------------------------------------------------ */

/*
 * The replication factor acts as a temperature that can be raised during
 * sampling (Sec. 3).  dst [n][m2][ld] (m2 >= m) takes replica r of states
 * [n][m][ld] for r < m, and a copy of replica r mod m for r >= m (a valid
 * state of the enlarged SAME joint: every copy of a column agrees with its
 * known data).  All ld columns are copied.
 */
int oracle_grow_replicas(int32_t n, int32_t m, int32_t m2, int64_t ld, int32_t state_bytes, const void *states,
                         void *dst) {
    if (n <= 0 || m < 1 || m2 < m || ld < 0 || (state_bytes != 1 && state_bytes != 2)) return OR_EINVAL;
    for (int32_t i = 0; i < n; ++i)
        for (int32_t r = 0; r < m2; ++r)
            memcpy((char *)dst + ((int64_t)i * m2 + r) * ld * state_bytes,
                   (const char *)states + ((int64_t)i * m + r % m) * ld * state_bytes, (size_t)ld * state_bytes);
    return OR_OK;
}
