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

// Sweep modes (descriptor field 2).
enum SweepMode : int32_t {
    kModeKP2 = 0,    // product of k-vectors, KP = 2
    kModeKP4 = 1,
    kModeKP8 = 2,
    kModeTable = 3,  // precomputed CDF thresholds per blanket configuration
    kModeKP16 = 4,   // product path with KP = 16
    kModeGeneric = 5, // K > 16: extended-exponent product path
    kModeKP6 = 6     // product path with KP = 6 (K = 5, 6)
};

// Launch classes (one kernel each):
//   0 fast path with LDS staging: the node's whole table record (k-vectors
//     or thresholds) when it fits the budget, else the record's smallest
//     k-vector groups (a prefix of the record); staged groups are indexed in
//     bytes, the rest are read from global memory with packed 16-bit indices
//     in units of one k-vector;
//   1 fast path with nothing staged (threshold tables beyond the budget, or
//     no k-vector group that fits): packed 16-bit indices in units of one
//     k-vector (or one threshold row);
//   2 wide path: product modes up to KP = 16 with 32-bit float indices;
//   3 generic path (K > 16).
constexpr int32_t kLaunchClasses = 4;
constexpr int64_t kLdsBudgetBytes = 32768;   // largest LDS staging budget per block
constexpr int64_t kDefaultLdsBytes = 24576;  // default budget: 6 blocks per CU (measured best)
// default threshold-table limit (entries): a table then fits the default LDS
// budget, so no threshold node gathers from global memory (measured best)
constexpr int64_t kDefaultTableLimit = kDefaultLdsBytes / 4;
constexpr int32_t kDescHeader = 16;
constexpr int64_t kPackedLimit = 65536;      // packed indices are 16-bit
constexpr int32_t kCountLdsBins = 8192;      // bins of the count kernel's LDS histogram
constexpr int64_t kCountSplitBins = 4 * kCountLdsBins;  // largest CPT counted in ranges

// Sweep descriptor of a node (int32 words at desc_off[i]):
//   [0] K  [1] KP  [2] mode  [3] tab_begin  [4] tab_len (floats)
//   [5] cond_off  [6] cond_len (threshold words)  [7] KT
//   [8] n_fast  [9] fast (relative word index of the fast group list)
//   [10] n_wide [11] wide (relative word index of the wide group list)
//   [12] launch class
//   [13] staged groups: the first [13] groups of the fast list are read from
//        LDS (byte indices), the rest from global memory; in table mode 1
//        when the threshold table is staged
//   [14] words a block copies into LDS before drawing (multiple of 4)
//   [15] product modes of classes 0 and 1: relative word index of the flat
//        list, the fast list's entries in list order, four words each after
//        a four-word header [E, 0, 0, 0]: [node, mult, group base, flags]
//        with flags 1 = first entry of its group, 2 = last, 4 = staged
//        group; an empty group is one entry of the node itself with mult 0
// A group list is a sequence of groups [n_e, base, (node, mult) * n_e]; the
// group's index is base + sum of mult * state over its entries.
//   wide list (every node): group 0 is the node's own row (entries: its
//     parents), then one group per child h (entries: h itself, then h's
//     other parents); indices are float offsets into the node's table record.
//   fast list (classes 0 and 1): product modes hold the same groups; the
//     table mode holds one group over the Markov blanket (ascending id, last
//     fastest) indexing the threshold rows.  Class 0 counts in bytes, class 1
//     in k-vectors (KP floats) or threshold rows (KT words); base and mult are
//     stored packed twice (v | v << 16) for the 2 x 16-bit lane arithmetic,
//     and every index of the list stays below 2^16.

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
    int32_t state_bytes = 1;   // bytes of one state in the non-quad arrays (values, targets, compact states)
    int32_t state_bits = 8;    // bits per state in a state quad: 4, 8 or 16
    int32_t quad_bytes = 4;    // bytes of one state quad (four replicas of a column): 2, 4 or 8
    int32_t max_card = 0;
    int64_t n_rows = 0;

    // regrouped sweep tables
    std::vector<int32_t> kp;         // [n]
    std::vector<int64_t> own_off;    // [n]
    std::vector<ChildTab> ctabs;
    int64_t table_floats = 0;
    std::vector<Segment> segments;

    // per-node table records and the sweep descriptors (layout above)
    std::vector<int64_t> tab_begin, tab_len;  // [n], floats
    std::vector<int32_t> lds_bytes;           // [n], 0: tables read from global memory
    // record layout: group_order[i] lists the groups (0 = own rows, 1 + c =
    // child c) in record order; the first stage_groups[i] of them, of
    // stage_floats[i] floats, are the part a block stages in LDS
    std::vector<std::vector<int32_t>> group_order;
    std::vector<int32_t> stage_groups;
    std::vector<int64_t> stage_floats;
    std::vector<int32_t> desc;
    std::vector<int32_t> desc_off;   // [n]

    // precomputed conditional tables: for a node in table mode (at most
    // kPackedLimit blanket configurations), every
    // configuration of its Markov blanket (blanket nodes in ascending id, last
    // fastest) holds KT uint32 thresholds T_k = ceil(2^24 * S_k / Z), k < K-1,
    // padded with 2^24; the draw is #{k : T_k <= u24}.
    int64_t cond_words = 0;
    // build program per table node, read by the threshold-build kernel:
    //   [K, KT, cond_off, n_cfg, n_bl, bl_card * n_bl, own_cpt_off, n_par,
    //    (bl_pos, stride) * n_par, n_child,
    //    per child: (cpt_off_h, K_h, s_i, xh_pos, n_cop, (bl_pos, stride) * n_cop)]
    std::vector<int32_t> cprog;
    std::vector<int32_t> cprog_off;  // per table node
    std::vector<int32_t> cprog_nodes;
    // same for the count kernel: [K, n_par, n_bins, cpt_off, (par_node, stride) * n_par]
    std::vector<int32_t> cdesc;
    std::vector<int32_t> cdesc_off;  // [n]
    // count work items (node, first bin): one per node, and one per range of
    // kCountLdsBins bins for a CPT larger than the count kernel's LDS
    // histogram, up to kCountSplitBins bins (each range's blocks read the
    // node's rows again); a larger CPT has one item with first bin -1, whose
    // blocks add to global memory directly
    std::vector<int32_t> cwork;

    // colour-ordered node list (colour 0 nodes, then colour 1, ...; inside a
    // colour grouped by launch class) and, per colour, the start of each class
    // range: launch[c*5 + k] .. launch[c*5 + k + 1] for class k < 4
    std::vector<int32_t> order;
    std::vector<int32_t> launch;       // [n_colors * (kLaunchClasses + 1)]
    std::vector<int32_t> launch_lds;   // [n_colors * kLaunchClasses]
    std::vector<int32_t> mode;         // [n]
    std::vector<int32_t> klass;        // [n] launch class

    // CPT rows, for the Dirichlet normalisation: entry offset and K of each row
    std::vector<int32_t> row_off, row_k;
};

// Returns 0 or a negative SAME_E* code with a message in err.
// table_limit: largest KT * (number of blanket configurations) for which a
// node gets a precomputed threshold table (0 disables the table path).
// lds_limit: LDS staging budget per block in bytes (class 0): the largest
// record staged whole, and the most a larger record stages of its groups.
// packed: false sends every product-mode node to the wide class.
// balance: false keeps the first-fit colouring (no balancing moves).
// state_bits: 0 picks 8-bit states (16-bit when some K > 127); 4 asks for
// 4-bit states (every K <= 16, else SAME_ECARD).
int compile_graph(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                  Compiled &out, std::string &err, int64_t table_limit = kDefaultTableLimit,
                  int64_t lds_limit = kDefaultLdsBytes, bool packed = true, bool balance = true,
                  int32_t state_bits = 0);

}  // namespace same
