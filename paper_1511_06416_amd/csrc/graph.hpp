// Host graph compiler of libsame: validation, topological order, moralized
// graph, colour groups, CPT layout and the per-node Markov-blanket tables the
// sweep kernels read (Sec. 1 CPT definition; Sec. 4 chromatic partitioning).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace same {

// One node's Markov-blanket view in the regrouped sweep tables.
//
// The sweep forms, for every state k of node i, the product of node i's own
// CPT entry and one entry of each child's CPT.  Both factors are read as
// "k-vectors": KP consecutive floats (K_i values padded to a power of two)
// holding max(theta, FLT_MIN) scaled by a power of two so that the vector's
// maximum lies in [0.5, 1) (the scale is common to all k, so the conditional
// is unchanged and the scaling is exact).
//   own k-vector of row u:        table[own_off + u*KP]
//   child h k-vector of (u', x_h): table[ctab_off + (u'*K_h + x_h)*KP]
// where u' is h's row index over its parents other than i, in the radix of
// those parents (last listed fastest).
struct ChildTab {
    int32_t node;      // i
    int32_t child;     // h
    int32_t slot;      // position of i in h's parent list
    int64_t off;       // float offset of the k-vector table
    int64_t groups;    // (R_h / K_i) * K_h
};

// A contiguous run of k-vectors the table-build kernel writes.
struct Segment {
    int64_t dst;       // float offset of group 0
    int64_t src;       // CPT entry offset of the source node (i for own, h for child)
    int32_t n_groups;
    int32_t K;         // values per group (K_i)
    int32_t KP;        // padded length
    int32_t Kh;        // child cardinality (1 for an own segment)
    int32_t s;         // stride of i in h's row index (0 for own)
    int32_t own;       // 1: own rows of node i
};

struct Compiled {
    int32_t n = 0;
    std::vector<int32_t> pptr, pidx, card;
    std::vector<int64_t> off;        // [n+1] CPT offsets
    std::vector<int64_t> rows;       // [n]   R_i
    std::vector<int64_t> pstride;    // [nnz] stride of each parent slot
    std::vector<int32_t> topo;       // Kahn order, smallest ready id first
    std::vector<int32_t> color;      // [n]
    int32_t n_colors = 0;
    std::vector<std::vector<int32_t>> groups;  // nodes of each colour, ascending
    int32_t state_bytes = 1;
    int32_t max_card = 0;
    int64_t n_rows = 0;

    // regrouped sweep tables
    std::vector<int32_t> kp;         // [n]
    std::vector<int64_t> own_off;    // [n]
    std::vector<ChildTab> ctabs;
    int64_t table_floats = 0;
    std::vector<Segment> segments;

    // flat descriptor stream read by the sweep kernel, and per-node offsets
    //   [K, KP, own_off, n_par, n_child,
    //    (par_node, par_mult) * n_par,
    //    per child: (h, ctab_off, xh_mult, n_cop, (cop_node, cop_mult) * n_cop)]
    // par_mult = parent stride * KP; xh_mult = KP; cop_mult = compact stride * K_h * KP
    std::vector<int32_t> desc;
    std::vector<int32_t> desc_off;   // [n]
    // same for the count kernel: [K, n_par, n_bins, cpt_off, (par_node, stride) * n_par]
    std::vector<int32_t> cdesc;
    std::vector<int32_t> cdesc_off;  // [n]

    // colour-ordered node list (colour 0 nodes, then colour 1, ...) and the
    // start of each colour in it, and each colour's largest KP
    std::vector<int32_t> order;
    std::vector<int32_t> color_start;  // [n_colors+1]
    std::vector<int32_t> color_kp;     // [n_colors]

    // CPT rows, for the Dirichlet normalisation: entry offset and K of each row
    std::vector<int32_t> row_off, row_k;
};

// Returns 0 or a negative SAME_E* code with a message in err.
int compile_graph(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                  Compiled &out, std::string &err);

}  // namespace same
