// Host graph compiler of libsame (see graph.hpp).
#include "graph.hpp"

#include <algorithm>
#include <functional>
#include <queue>
#include <set>

#include "../../include/same.h"

namespace same {

namespace {

constexpr int64_t kI32Max = (int64_t(1) << 31) - 1;

int32_t padded_k(int32_t K) {
    if (K <= 2) return 2;
    if (K <= 4) return 4;
    if (K <= 6) return 6;
    if (K <= 8) return 8;
    if (K <= 16) return 16;
    return (K + 3) & ~3;
}

int fail(std::string &err, int code, const std::string &msg) {
    err = msg;
    return code;
}

}  // namespace

int32_t thresholds_per_config(int32_t K) {
    int32_t t = 1;
    while (t < K - 1) t <<= 1;
    return t;
}

// Balanced colour groups (Sec. 4 colours the moralized graph with groups of
// balanced size): single-node moves from a group to one at least two nodes
// smaller, allowed only when the node has no moral neighbour in the target
// group.  The move taken is the first found scanning source groups from the
// largest (ties: lower colour), their nodes by ascending id, and target
// groups from the smallest (ties: lower colour); then the scan restarts.
// Each move lowers the sum of squared group sizes, so the loop ends, and
// no group empties.  nbc[v][c] counts v's neighbours of colour c.
static void balance_colours(const std::vector<std::vector<int32_t>> &nb, int32_t n_colors, std::vector<int32_t> &color) {
    const int32_t n = (int32_t)color.size();
    if (n_colors < 2) return;
    std::vector<std::vector<int32_t>> nbc(n, std::vector<int32_t>(n_colors, 0));
    std::vector<std::set<int32_t>> members(n_colors);
    for (int32_t v = 0; v < n; ++v) {
        members[color[v]].insert(v);
        for (int32_t w : nb[v]) nbc[v][color[w]]++;
    }
    std::vector<int32_t> desc(n_colors), asc(n_colors);
    for (;;) {
        for (int32_t c = 0; c < n_colors; ++c) desc[c] = asc[c] = c;
        auto sz = [&](int32_t c) { return (int32_t)members[c].size(); };
        std::stable_sort(desc.begin(), desc.end(), [&](int32_t x, int32_t y) { return sz(x) > sz(y); });
        std::stable_sort(asc.begin(), asc.end(), [&](int32_t x, int32_t y) { return sz(x) < sz(y); });
        int32_t mv = -1, to = -1;
        for (int32_t a : desc) {
            for (int32_t v : members[a]) {
                for (int32_t b : asc) {
                    if (sz(b) + 1 >= sz(a)) break;
                    if (nbc[v][b] == 0) {
                        mv = v;
                        to = b;
                        break;
                    }
                }
                if (mv >= 0) break;
            }
            if (mv >= 0) break;
        }
        if (mv < 0) return;
        const int32_t from = color[mv];
        members[from].erase(mv);
        members[to].insert(mv);
        color[mv] = to;
        for (int32_t w : nb[mv]) {
            nbc[w][from]--;
            nbc[w][to]++;
        }
    }
}

int compile_graph(int32_t n, const int32_t *pptr, const int32_t *pidx, const int32_t *card,
                  Compiled &g, std::string &err, int64_t table_limit, int64_t lds_limit, bool packed,
                  bool balance, int32_t state_bits) {
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
    if (state_bits == 4) {
        if (g.max_card > 16) return fail(err, SAME_ECARD, "4-bit states need every cardinality <= 16");
        g.state_bits = 4;
    } else {
        g.state_bits = g.max_card <= 127 ? 8 : 16;
    }
    g.state_bytes = g.state_bits == 16 ? 2 : 1;
    g.quad_bytes = g.state_bits / 2;

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
    if (balance) balance_colours(nb, g.n_colors, g.color);
    g.groups.assign(g.n_colors, {});
    for (int32_t i = 0; i < n; ++i) g.groups[g.color[i]].push_back(i);

    // regrouped sweep tables and the segments that build them: one contiguous
    // record per node (its own k-vectors and one table per child), every
    // record and sub-table on a 64-byte boundary so that the sweep can read a
    // group with float2/float4 loads and stage a record in LDS.  A record
    // larger than lds_limit puts the groups it can stage first (smallest
    // first, up to lds_limit bytes), so that the staged part is a prefix of
    // the record.
    g.kp.resize(n);
    g.own_off.resize(n);
    g.tab_begin.resize(n);
    g.tab_len.resize(n);
    g.group_order.assign(n, {});
    g.stage_groups.assign(n, 0);
    g.stage_floats.assign(n, 0);
    auto align16 = [](int64_t v) { return (v + 15) & ~int64_t(15); };
    int64_t pos = 0;
    std::vector<std::vector<int32_t>> ctab_of(n);  // indices into ctabs per node (children order)
    for (int32_t i = 0; i < n; ++i) {
        g.kp[i] = padded_k(card[i]);
        // group sizes in floats: 0 = own rows, 1 + c = child c (kids order)
        std::vector<int64_t> gsz;
        gsz.push_back(align16(g.rows[i] * g.kp[i]));
        for (auto &c : kids[i]) gsz.push_back(align16(g.rows[c.first] / card[i] * card[c.first] * g.kp[i]));
        int64_t total = 0;
        for (int64_t v : gsz) total += v;
        std::vector<int32_t> &order = g.group_order[i];
        if (total * 4 <= lds_limit) {
            for (int32_t t = 0; t < (int32_t)gsz.size(); ++t) order.push_back(t);
            g.stage_groups[i] = (int32_t)gsz.size();
            g.stage_floats[i] = total;
        } else {
            std::vector<int32_t> by_size(gsz.size());
            for (int32_t t = 0; t < (int32_t)gsz.size(); ++t) by_size[t] = t;
            std::stable_sort(by_size.begin(), by_size.end(),
                             [&](int32_t a, int32_t b) { return gsz[a] < gsz[b]; });
            std::vector<char> staged(gsz.size(), 0);
            int64_t cum = 0;
            for (int32_t t : by_size) {
                if ((cum + gsz[t]) * 4 > lds_limit) break;
                cum += gsz[t];
                staged[t] = 1;
                g.stage_groups[i] += 1;
            }
            g.stage_floats[i] = cum;
            for (int32_t t = 0; t < (int32_t)gsz.size(); ++t)
                if (staged[t]) order.push_back(t);
            for (int32_t t = 0; t < (int32_t)gsz.size(); ++t)
                if (!staged[t]) order.push_back(t);
        }
        pos = align16(pos);
        g.tab_begin[i] = pos;
        std::vector<int64_t> at(gsz.size());
        for (int32_t t : order) {
            at[t] = pos;
            pos += gsz[t];
        }
        g.own_off[i] = at[0];
        g.segments.push_back(Segment{at[0], g.off[i], (int32_t)g.rows[i], card[i], g.kp[i], 1, 0, 1});
        for (size_t ci = 0; ci < kids[i].size(); ++ci) {
            const auto &c = kids[i][ci];
            int32_t h = c.first;
            ChildTab t;
            t.node = i;
            t.child = h;
            t.slot = c.second;
            t.groups = g.rows[h] / card[i] * card[h];
            t.off = at[ci + 1];
            int64_t s_i = g.pstride[pptr[h] + c.second];
            g.segments.push_back(
                Segment{t.off, g.off[h], (int32_t)t.groups, card[i], g.kp[i], card[h], (int32_t)s_i, 0});
            ctab_of[i].push_back((int32_t)g.ctabs.size());
            g.ctabs.push_back(t);
        }
        g.tab_len[i] = pos - g.tab_begin[i];
    }
    g.table_floats = pos;
    if (pos > kI32Max) return fail(err, SAME_ESIZE, "sweep tables exceed 2^31 floats");

    // Markov blankets (parents, children, co-parents; ascending id) and modes
    std::vector<std::vector<int32_t>> blanket(n);
    g.mode.assign(n, kModeKP2);
    for (int32_t i = 0; i < n; ++i) {
        std::vector<int32_t> &b = blanket[i];
        for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) b.push_back(g.pidx[a]);
        for (auto &c : kids[i]) {
            int32_t h = c.first;
            b.push_back(h);
            for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a)
                if (g.pidx[a] != i) b.push_back(g.pidx[a]);
        }
        std::sort(b.begin(), b.end());
        b.erase(std::unique(b.begin(), b.end()), b.end());
        const int32_t K = card[i];
        int32_t mode = K <= 2 ? kModeKP2 : K <= 4 ? kModeKP4 : K <= 6 ? kModeKP6 : K <= 8 ? kModeKP8
                     : K <= 16 ? kModeKP16 : kModeGeneric;
        if (table_limit > 0 && K <= 9) {
            int64_t cfg = 1;
            for (int32_t v : b) {
                cfg *= card[v];
                if (cfg * thresholds_per_config(K) > table_limit) break;
            }
            if (cfg * thresholds_per_config(K) <= table_limit && cfg <= kPackedLimit && b.size() <= 24)
                mode = kModeTable;
        }
        g.mode[i] = mode;
    }

    // threshold tables and their build programs
    std::vector<int64_t> cond_off(n, -1);
    {
        int64_t cpos = 0;
        for (int32_t i = 0; i < n; ++i) {
            if (g.mode[i] != kModeTable) continue;
            const int32_t K = card[i], KT = thresholds_per_config(K);
            const std::vector<int32_t> &b = blanket[i];
            int64_t ncfg = 1;
            for (int32_t v : b) ncfg *= card[v];
            cpos = (cpos + 15) & ~int64_t(15);
            cond_off[i] = cpos;
            auto pos_of = [&](int32_t v) {
                return (int32_t)(std::lower_bound(b.begin(), b.end(), v) - b.begin());
            };
            g.cprog_nodes.push_back(i);
            g.cprog_off.push_back((int32_t)g.cprog.size());
            std::vector<int32_t> &P = g.cprog;
            P.push_back(K);
            P.push_back(KT);
            P.push_back((int32_t)cpos);
            P.push_back((int32_t)ncfg);
            P.push_back((int32_t)b.size());
            for (int32_t v : b) P.push_back(card[v]);
            P.push_back((int32_t)g.off[i]);
            P.push_back(pptr[i + 1] - pptr[i]);
            for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) {
                P.push_back(pos_of(g.pidx[a]));
                P.push_back((int32_t)g.pstride[a]);
            }
            P.push_back((int32_t)kids[i].size());
            for (auto &c : kids[i]) {
                const int32_t h = c.first;
                P.push_back((int32_t)g.off[h]);
                P.push_back(card[h]);
                P.push_back((int32_t)g.pstride[pptr[h] + c.second]);
                P.push_back(pos_of(h));
                P.push_back(pptr[h + 1] - pptr[h] - 1);
                for (int32_t a = pptr[h]; a < pptr[h + 1]; ++a) {
                    if (g.pidx[a] == i) continue;
                    P.push_back(pos_of(g.pidx[a]));
                    P.push_back((int32_t)g.pstride[a]);
                }
            }
            cpos += ncfg * KT;
            if (cpos > kI32Max) return fail(err, SAME_ESIZE, "threshold tables exceed 2^31 words");
        }
        g.cond_words = (cpos + 15) & ~int64_t(15);  // whole float4s for the LDS staging copy
    }

    // descriptor streams
    g.desc_off.resize(n);
    g.cdesc_off.resize(n);
    g.lds_bytes.assign(n, 0);
    g.klass.assign(n, 0);
    for (int32_t i = 0; i < n; ++i) {
        const int32_t KP = g.kp[i], K = card[i];
        const bool tab = g.mode[i] == kModeTable;
        const std::vector<int32_t> &b = blanket[i];
        const int32_t KT = tab ? thresholds_per_config(K) : 0;
        int64_t ncfg = 1;
        if (tab)
            for (int32_t v : b) ncfg *= card[v];
        const int64_t cond_len = tab ? ncfg * KT : 0;

        // launch class and the unit of the fast list's indices (bytes)
        int32_t klass;
        int64_t unit = 0;
        int32_t n_staged = 0;   // fast-list groups (or the threshold table) read from LDS
        int64_t stage_words = 0;  // words the block copies into LDS
        if (g.mode[i] == kModeGeneric) {
            klass = 3;
        } else if (g.mode[i] == kModeKP16) {
            klass = 2;
        } else {
            const int64_t bytes = tab ? cond_len * 4 : g.tab_len[i] * 4;
            // index unit of the global fast list: a threshold row, a k-vector,
            // or 8 bytes for KP = 6 (24-byte k-vectors in 64-byte aligned groups)
            const int64_t row_bytes = tab ? (int64_t)KT * 4 : KP == 6 ? 8 : (int64_t)KP * 4;
            if (!packed && !tab) {
                klass = 2;
            } else if (bytes <= lds_limit) {
                klass = 0;
                unit = 1;
                n_staged = tab ? 1 : g.stage_groups[i];
                stage_words = tab ? ((cond_len + 3) & ~int64_t(3)) : g.tab_len[i];
            } else if (bytes / row_bytes <= kPackedLimit) {
                // staged groups (if any) count bytes, the others k-vectors
                unit = row_bytes;
                if (!tab) {
                    n_staged = g.stage_groups[i];
                    stage_words = g.stage_floats[i];
                }
                klass = n_staged > 0 ? 0 : 1;
            } else {
                klass = 2;  // product modes only: tables always fit 16-bit rows
            }
            g.lds_bytes[i] = (int32_t)(stage_words * 4);  // staged in float4s
        }
        g.klass[i] = klass;

        const int32_t base = (int32_t)g.desc.size();
        g.desc_off[i] = base;
        g.desc.resize(base + kDescHeader, 0);
        g.desc[base + 0] = K;
        g.desc[base + 1] = KP;
        g.desc[base + 2] = g.mode[i];
        g.desc[base + 3] = (int32_t)g.tab_begin[i];
        g.desc[base + 4] = (int32_t)g.tab_len[i];
        g.desc[base + 5] = (int32_t)cond_off[i];
        g.desc[base + 6] = (int32_t)cond_len;
        g.desc[base + 7] = KT;
        g.desc[base + 12] = klass;
        g.desc[base + 13] = n_staged;
        g.desc[base + 14] = (int32_t)stage_words;

        // product-path groups in float offsets: own row, then one per child
        struct Group {
            int64_t base;
            std::vector<std::pair<int32_t, int64_t>> ent;
        };
        std::vector<Group> groups;
        {
            Group own{g.own_off[i] - g.tab_begin[i], {}};
            for (int32_t a2 = pptr[i]; a2 < pptr[i + 1]; ++a2)
                own.ent.push_back({g.pidx[a2], g.pstride[a2] * KP});
            groups.push_back(own);
        }
        for (int32_t t : ctab_of[i]) {
            const ChildTab &ct = g.ctabs[t];
            const int32_t h = ct.child, Kh = card[h];
            Group cg{ct.off - g.tab_begin[i], {{h, (int64_t)KP}}};
            // h's parents other than i, compact strides (last listed fastest)
            int64_t r = 1;
            std::vector<std::pair<int32_t, int64_t>> cops;
            for (int32_t a2 = pptr[h + 1] - 1; a2 >= pptr[h]; --a2) {
                if (a2 - pptr[h] == ct.slot) continue;
                cops.push_back({g.pidx[a2], r * Kh * KP});
                r *= card[g.pidx[a2]];
            }
            std::reverse(cops.begin(), cops.end());
            cg.ent.insert(cg.ent.end(), cops.begin(), cops.end());
            groups.push_back(cg);
        }
        {
            // record order: the staged groups first
            std::vector<Group> ordered;
            for (int32_t t : g.group_order[i]) ordered.push_back(groups[t]);
            groups.swap(ordered);
        }
        auto emit = [&](const Group &gr, int64_t div, bool packed) -> bool {
            auto word = [&](int64_t v) -> int64_t {
                v /= div;
                return packed ? (v | (v << 16)) : v;
            };
            if (gr.base % div || (packed && gr.base / div >= kPackedLimit)) return false;
            if (!packed && gr.base > kI32Max) return false;
            g.desc.push_back((int32_t)gr.ent.size());
            g.desc.push_back((int32_t)(uint32_t)word(gr.base));
            for (auto &e : gr.ent) {
                if (e.second % div) return false;
                if (packed ? e.second / div >= kPackedLimit : e.second > kI32Max) return false;
                g.desc.push_back(e.first);
                g.desc.push_back((int32_t)(uint32_t)word(e.second));
            }
            return true;
        };
        g.desc[base + 10] = (int32_t)groups.size();
        g.desc[base + 11] = (int32_t)g.desc.size() - base;
        for (auto &gr : groups)
            if (!emit(gr, 1, false)) return fail(err, SAME_ESIZE, "sweep table offset overflow");
        if (klass <= 1) {
            g.desc[base + 9] = (int32_t)g.desc.size() - base;
            bool ok = true;
            if (tab) {
                // one group over the blanket, last fastest, in threshold rows
                Group bg{0, {}};
                int64_t r = 1;
                for (int32_t t = (int32_t)b.size() - 1; t >= 0; --t) {
                    bg.ent.push_back({b[t], r * KT * 4});
                    r *= card[b[t]];
                }
                std::reverse(bg.ent.begin(), bg.ent.end());
                g.desc[base + 8] = 1;
                ok = emit(bg, unit, true);
            } else {
                g.desc[base + 8] = (int32_t)groups.size();
                for (size_t t = 0; t < groups.size(); ++t) {
                    const Group &gr = groups[t];
                    Group gb{gr.base * 4, {}};
                    for (auto &e : gr.ent) gb.ent.push_back({e.first, e.second * 4});
                    // staged groups count bytes into LDS, the rest k-vectors
                    ok = ok && emit(gb, (int32_t)t < n_staged ? 1 : unit, true);
                }
                if (ok) {
                    // the same list flat: per entry [node, mult, group base,
                    // flags: 1 first of its group, 2 last, 4 staged group];
                    // an empty group is one entry of the node itself with
                    // multiplier 0
                    std::vector<int32_t> flat;
                    int64_t pos = base + g.desc[base + 9];
                    for (size_t t = 0; t < groups.size(); ++t) {
                        const int32_t ne = g.desc[pos], gbase = g.desc[pos + 1];
                        const int32_t st = (int32_t)t < n_staged ? 4 : 0;
                        if (ne == 0) flat.insert(flat.end(), {i, 0, gbase, 1 | 2 | st});
                        for (int32_t q = 0; q < ne; ++q)
                            flat.insert(flat.end(), {g.desc[pos + 2 + 2 * q], g.desc[pos + 3 + 2 * q], gbase,
                                                     (q == 0 ? 1 : 0) | (q == ne - 1 ? 2 : 0) | st});
                        pos += 2 + 2 * ne;
                    }
                    g.desc[base + 15] = (int32_t)g.desc.size() - base;
                    g.desc.push_back((int32_t)(flat.size() / 4));
                    g.desc.insert(g.desc.end(), {0, 0, 0});
                    g.desc.insert(g.desc.end(), flat.begin(), flat.end());
                }
            }
            // the class test above bounds every index below 2^16 units
            if (!ok) return fail(err, SAME_ESIZE, "packed sweep index overflow");
        }

        if (g.rows[i] * K > kCountSplitBins) {
            g.cwork.push_back(i);
            g.cwork.push_back(-1);
        } else {
            for (int64_t lo = 0; lo == 0 || lo < g.rows[i] * K; lo += kCountLdsBins) {
                g.cwork.push_back(i);
                g.cwork.push_back((int32_t)lo);
            }
        }
        g.cdesc_off[i] = (int32_t)g.cdesc.size();
        g.cdesc.push_back(K);
        g.cdesc.push_back(pptr[i + 1] - pptr[i]);
        g.cdesc.push_back((int32_t)(g.rows[i] * K));
        g.cdesc.push_back((int32_t)g.off[i]);
        for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) {
            g.cdesc.push_back(g.pidx[a]);
            g.cdesc.push_back((int32_t)g.pstride[a]);
        }
    }

    // count work ordered by each family's smallest parent (a root by itself,
    // just before the families whose smallest parent it is): families that
    // share a parent run together, so its rows are re-read from L2 rather
    // than from memory.  The order changes no count (integer atomics).
    {
        const size_t nw = g.cwork.size() / 2;
        std::vector<std::pair<int64_t, size_t>> key(nw);
        for (size_t w = 0; w < nw; ++w) {
            const int32_t i = g.cwork[2 * w];
            int64_t k = 2 * (int64_t)i;
            for (int32_t a = pptr[i]; a < pptr[i + 1]; ++a) k = std::min(k, 2 * (int64_t)g.pidx[a] + 1);
            key[w] = {k, w};
        }
        std::stable_sort(key.begin(), key.end());
        std::vector<int32_t> cw;
        cw.reserve(g.cwork.size());
        for (const auto &kw : key) {
            cw.push_back(g.cwork[2 * kw.second]);
            cw.push_back(g.cwork[2 * kw.second + 1]);
        }
        g.cwork.swap(cw);
    }

    // launch order: per colour, the nodes of each launch class in turn, and
    // per (colour, class) the LDS bytes the launch needs
    g.launch.assign((size_t)g.n_colors * (kLaunchClasses + 1), 0);
    g.launch_lds.assign((size_t)g.n_colors * kLaunchClasses, 0);
    // a node's sweep cost per item, estimated from its fast list: the
    // entries' loads and, per group, the k-vector products or thresholds
    auto sweep_cost = [&](int32_t i) {
        const int32_t *d = g.desc.data() + g.desc_off[i];
        const int32_t *gl = d + d[9];
        const int32_t width = d[2] == kModeTable ? d[7] : d[1];
        int64_t cost = 0;
        for (int32_t t = 0; t < d[8]; ++t) {
            cost += gl[0] + width;
            gl += 2 + 2 * gl[0];
        }
        return cost;
    };
    for (int32_t c = 0; c < g.n_colors; ++c) {
        for (int32_t k = 0; k < kLaunchClasses; ++k) {
            g.launch[c * (kLaunchClasses + 1) + k] = (int32_t)g.order.size();
            std::vector<std::pair<int64_t, int32_t>> nodes;
            for (int32_t i : g.groups[c]) {
                if (g.klass[i] != k) continue;
                nodes.push_back({k <= 1 ? -sweep_cost(i) : 0, i});
                int32_t &lb = g.launch_lds[c * kLaunchClasses + k];
                lb = std::max(lb, g.lds_bytes[i]);
            }
            // the costliest nodes first: their blocks of every column slab
            // start before the cheap ones, which shortens the launch's tail
            std::stable_sort(nodes.begin(), nodes.end());
            for (const auto &ni : nodes) g.order.push_back(ni.second);
        }
        g.launch[c * (kLaunchClasses + 1) + kLaunchClasses] = (int32_t)g.order.size();
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
