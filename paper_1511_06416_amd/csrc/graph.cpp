// Host graph compiler of libsame (see graph.hpp).
#include "graph.hpp"

#include <algorithm>
#include <functional>
#include <queue>

#include "../../include/same.h"

namespace same {

namespace {

constexpr int64_t kI32Max = (int64_t(1) << 31) - 1;

int32_t padded_k(int32_t K) {
    if (K <= 2) return 2;
    if (K <= 4) return 4;
    if (K <= 8) return 8;
    if (K <= 16) return 16;
    return (K + 3) & ~3;
}

int fail(std::string &err, int code, const std::string &msg) {
    err = msg;
    return code;
}

}  // namespace

int compile_graph(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                  Compiled &g, std::string &err) {
    if (n <= 0) return fail(err, SAME_EINVAL, "n_nodes must be positive");
    if (!pptr || !card) return fail(err, SAME_EINVAL, "parent_ptr and card must be non-null");
    if (pptr[0] != 0) return fail(err, SAME_EGRAPH, "parent_ptr[0] must be 0");
    for (int32_t i = 0; i < n; ++i)
        if (pptr[i + 1] < pptr[i]) return fail(err, SAME_EGRAPH, "parent_ptr must be non-decreasing");
    const int32_t nnz = pptr[n];
    if (nnz > 0 && !pidx) return fail(err, SAME_EINVAL, "parent_idx is null");

    g = Compiled();
    g.n = n;
    g.pptr.assign(pptr, pptr + n + 1);
    g.pidx.assign(pidx ? pidx : pptr, pidx ? pidx + nnz : pptr);
    g.card.assign(card, card + n);

    for (int32_t i = 0; i < n; ++i) {
        if (card[i] < 2 || card[i] > 32767)
            return fail(err, SAME_ECARD, "node " + std::to_string(i) + ": cardinality " +
                                             std::to_string(card[i]) + " outside [2, 32767]");
        std::vector<int32_t> seen(g.pidx.begin() + pptr[i], g.pidx.begin() + pptr[i + 1]);
        for (int32_t p : seen) {
            if (p < 0 || p >= n)
                return fail(err, SAME_EGRAPH, "node " + std::to_string(i) + ": parent out of range");
            if (p == i) return fail(err, SAME_EGRAPH, "node " + std::to_string(i) + ": self-loop");
        }
        std::sort(seen.begin(), seen.end());
        if (std::adjacent_find(seen.begin(), seen.end()) != seen.end())
            return fail(err, SAME_EGRAPH, "node " + std::to_string(i) + ": duplicate parent");
        g.max_card = std::max(g.max_card, card[i]);
    }
    g.state_bytes = g.max_card <= 127 ? 1 : 2;

    // children with the slot they occupy in the child's parent list
    std::vector<std::vector<std::pair<int32_t, int32_t>>> kids(n);
    for (int32_t h = 0; h < n; ++h)
        for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) kids[g.pidx[a]].push_back({h, a - pptr[h]});

    // Kahn topological order, smallest ready id first
    {
        std::vector<int32_t> indeg(n);
        std::priority_queue<int32_t, std::vector<int32_t>, std::greater<int32_t>> ready;
        for (int32_t i = 0; i < n; ++i) {
            indeg[i] = pptr[i + 1] - pptr[i];
            if (indeg[i] == 0) ready.push(i);
        }
        while (!ready.empty()) {
            int32_t v = ready.top();
            ready.pop();
            g.topo.push_back(v);
            for (auto &c : kids[v])
                if (--indeg[c.first] == 0) ready.push(c.first);
        }
        if ((int32_t)g.topo.size() != n) return fail(err, SAME_EGRAPH, "the graph has a cycle");
    }

    // CPT layout: last listed parent fastest
    g.off.assign(n + 1, 0);
    g.rows.assign(n, 0);
    g.pstride.assign(nnz, 0);
    for (int32_t i = 0; i < n; ++i) {
        int64_t r = 1;
        for (int32_t a = pptr[i + 1] - 1; a >= pptr[i]; --a) {
            g.pstride[a] = r;
            r *= card[g.pidx[a]];
            if (r > kI32Max) return fail(err, SAME_ESIZE, "node " + std::to_string(i) + ": too many CPT rows");
        }
        g.rows[i] = r;
        g.off[i + 1] = g.off[i] + r * card[i];
        if (g.off[i + 1] > kI32Max) return fail(err, SAME_ESIZE, "CPT total exceeds 2^31 entries");
        g.n_rows += r;
    }

    // moralized graph as sorted neighbour lists: parent-child plus co-parents
    std::vector<std::vector<int32_t>> nb(n);
    for (int32_t h = 0; h < n; ++h)
        for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) {
            int32_t p = g.pidx[a];
            nb[p].push_back(h);
            nb[h].push_back(p);
            for (int32_t b = a + 1; b < pptr[h + 1]; ++b) {
                nb[p].push_back(g.pidx[b]);
                nb[g.pidx[b]].push_back(p);
            }
        }
    for (auto &v : nb) {
        std::sort(v.begin(), v.end());
        v.erase(std::unique(v.begin(), v.end()), v.end());
    }

    // first-fit colouring in topological order
    g.color.assign(n, -1);
    for (int32_t v : g.topo) {
        std::vector<char> taken(nb[v].size() + 1, 0);
        for (int32_t w : nb[v]) {
            int32_t c = g.color[w];
            if (c >= 0 && c < (int32_t)taken.size()) taken[c] = 1;
        }
        int32_t c = 0;
        while (taken[c]) ++c;
        g.color[v] = c;
        g.n_colors = std::max(g.n_colors, c + 1);
    }
    g.groups.assign(g.n_colors, {});
    for (int32_t i = 0; i < n; ++i) g.groups[g.color[i]].push_back(i);
    g.color_start.assign(1, 0);
    for (int32_t c = 0; c < g.n_colors; ++c) {
        int32_t kp = 2;
        for (int32_t i : g.groups[c]) {
            g.order.push_back(i);
            kp = std::max(kp, padded_k(card[i]));
        }
        g.color_start.push_back((int32_t)g.order.size());
        g.color_kp.push_back(kp);
    }

    // regrouped sweep tables and the segments that build them
    g.kp.resize(n);
    g.own_off.resize(n);
    // every k-vector table starts on a 64-byte boundary so that the sweep can
    // read a group with float2/float4 loads
    auto align16 = [](int64_t v) { return (v + 15) & ~int64_t(15); };
    int64_t pos = 0;
    for (int32_t i = 0; i < n; ++i) {
        g.kp[i] = padded_k(card[i]);
        pos = align16(pos);
        g.own_off[i] = pos;
        Segment s{pos, g.off[i], (int32_t)g.rows[i], card[i], g.kp[i], 1, 0, 1};
        g.segments.push_back(s);
        pos += g.rows[i] * g.kp[i];
    }
    std::vector<std::vector<int32_t>> ctab_of(n);  // indices into ctabs per node
    for (int32_t i = 0; i < n; ++i) {
        for (auto &c : kids[i]) {
            int32_t h = c.first;
            ChildTab t;
            t.node = i;
            t.child = h;
            t.slot = c.second;
            t.groups = g.rows[h] / card[i] * card[h];
            pos = align16(pos);
            t.off = pos;
            int64_t s_i = g.pstride[pptr[h] + c.second];
            Segment s{pos, g.off[h], (int32_t)t.groups, card[i], g.kp[i], card[h], (int32_t)s_i, 0};
            g.segments.push_back(s);
            pos += t.groups * g.kp[i];
            ctab_of[i].push_back((int32_t)g.ctabs.size());
            g.ctabs.push_back(t);
        }
    }
    g.table_floats = pos;
    if (pos > kI32Max) return fail(err, SAME_ESIZE, "sweep tables exceed 2^31 floats");

    // descriptor streams
    g.desc_off.resize(n);
    g.cdesc_off.resize(n);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t KP = g.kp[i];
        g.desc_off[i] = (int32_t)g.desc.size();
        g.desc.push_back(card[i]);
        g.desc.push_back(KP);
        g.desc.push_back((int32_t)g.own_off[i]);
        g.desc.push_back(pptr[i + 1] - pptr[i]);
        g.desc.push_back((int32_t)kids[i].size());
        for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) {
            g.desc.push_back(g.pidx[a]);
            int64_t mult = g.pstride[a] * KP;
            if (mult > kI32Max) return fail(err, SAME_ESIZE, "row stride overflow");
            g.desc.push_back((int32_t)mult);
        }
        for (int32_t t : ctab_of[i]) {
            const ChildTab &ct = g.ctabs[t];
            const int32_t h = ct.child, Kh = card[h];
            g.desc.push_back(h);
            g.desc.push_back((int32_t)ct.off);
            g.desc.push_back(KP);
            g.desc.push_back(pptr[h + 1] - pptr[h] - 1);
            // compact strides over h's parents without i, last listed fastest
            int64_t r = 1;
            std::vector<std::pair<int32_t, int64_t>> cops;
            for (int32_t a = pptr[h + 1] - 1; a >= pptr[h]; --a) {
                if (a - pptr[h] == ct.slot) continue;
                cops.push_back({g.pidx[a], r});
                r *= card[g.pidx[a]];
            }
            std::reverse(cops.begin(), cops.end());
            for (auto &cp : cops) {
                int64_t mult = cp.second * Kh * KP;
                if (mult > kI32Max) return fail(err, SAME_ESIZE, "child stride overflow");
                g.desc.push_back(cp.first);
                g.desc.push_back((int32_t)mult);
            }
        }
        g.cdesc_off[i] = (int32_t)g.cdesc.size();
        g.cdesc.push_back(card[i]);
        g.cdesc.push_back(pptr[i + 1] - pptr[i]);
        g.cdesc.push_back((int32_t)(g.rows[i] * card[i]));
        g.cdesc.push_back((int32_t)g.off[i]);
        for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) {
            g.cdesc.push_back(g.pidx[a]);
            g.cdesc.push_back((int32_t)g.pstride[a]);
        }
    }
    if ((int64_t)g.desc.size() > kI32Max) return fail(err, SAME_ESIZE, "descriptor overflow");

    // CPT rows
    g.row_off.reserve(g.n_rows);
    g.row_k.reserve(g.n_rows);
    for (int32_t i = 0; i < n; ++i)
        for (int64_t u = 0; u < g.rows[i]; ++u) {
            g.row_off.push_back((int32_t)(g.off[i] + u * card[i]));
            g.row_k.push_back(card[i]);
        }
    return SAME_OK;
}

}  // namespace same
