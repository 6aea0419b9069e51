// Host planner: validates candidate trees and derives the shared tree descriptor
// consumed by every device entry point (LumoTree Sec. III-C), the spine-first slot
// map (Sec. V-B), the conv gather sources (Sec. V-C) and the verification schedule
// of each policy (path groups, Sec. IV-A and Alg. 2; cut states, Sec. IV-C).
#include <algorithm>
#include <cstring>
#include <vector>

#include "internal.h"

namespace {

struct Chain {
    int level;
    int req;
    int start;  // request-local first node
    int src;    // source cut (-1 = pre-tree state)
};

struct SegOut {
    int req, src;
    std::vector<int> rows, out, cut;
};

struct ReqTree {
    int n = 0;
    const int32_t* parent = nullptr;
    std::vector<int> depth, child_off, child;  // children CSR, ids increasing
    std::vector<int> leaves, spine, slot;
    std::vector<char> on_spine;
    std::vector<int> owner;  // smallest leaf id whose path contains the node
    std::vector<int> dfs, dfs_pos;  // preorder (children by increasing id) and its inverse

    int n_children(int x) const { return child_off[x + 1] - child_off[x]; }
    int first_child(int x) const { return n_children(x) ? child[child_off[x]] : -1; }
};

lumo_status build_tree(int r, int n, const int32_t* parent, ReqTree& t) {
    t.n = n;
    t.parent = parent;
    if (n == 0) return LUMO_OK;
    if (parent[0] != -1) return lumo::fail(LUMO_EDESC, "request %d: node 0 must be the root (parent -1)", r);
    for (int i = 1; i < n; ++i)
        if (parent[i] < 0 || parent[i] >= i)
            return lumo::fail(LUMO_EDESC, "request %d: node %d has parent %d (need 0 <= parent < id)", r, i,
                              parent[i]);
    t.depth.assign(n, 0);
    std::vector<int> cnt(n + 1, 0);
    for (int i = 1; i < n; ++i) {
        t.depth[i] = t.depth[parent[i]] + 1;
        ++cnt[parent[i] + 1];
    }
    t.child_off.assign(n + 1, 0);
    for (int i = 0; i < n; ++i) t.child_off[i + 1] = t.child_off[i] + cnt[i + 1];
    t.child.assign(std::max(n - 1, 0), 0);
    std::vector<int> fill(t.child_off.begin(), t.child_off.end() - 1);
    for (int i = 1; i < n; ++i) t.child[fill[parent[i]]++] = i;  // ids increase: lists sorted
    for (int i = 0; i < n; ++i)
        if (!t.n_children(i)) t.leaves.push_back(i);
    t.on_spine.assign(n, 0);
    for (int x = 0; x >= 0; x = t.first_child(x)) {
        t.spine.push_back(x);
        t.on_spine[x] = 1;
    }
    t.slot.assign(n, 0);
    int pos = 0;
    for (int x : t.spine) t.slot[x] = pos++;
    for (int i = 0; i < n; ++i)
        if (!t.on_spine[i]) t.slot[i] = pos++;
    // owner: the smallest leaf id in the node's subtree (children have larger ids, so a
    // reverse sweep sees every child before its parent)
    t.owner.assign(n, 0);
    for (int i = n - 1; i >= 0; --i) {
        int best = i;
        if (t.n_children(i)) {
            best = t.owner[t.child[t.child_off[i]]];
            for (int e = t.child_off[i] + 1; e < t.child_off[i + 1]; ++e) best = std::min(best, t.owner[t.child[e]]);
        }
        t.owner[i] = best;
    }
    t.dfs.reserve(n);
    std::vector<int> stack{0};
    while (!stack.empty()) {
        const int x = stack.back();
        stack.pop_back();
        t.dfs.push_back(x);
        for (int e = t.child_off[x + 1] - 1; e >= t.child_off[x]; --e) stack.push_back(t.child[e]);
    }
    t.dfs_pos.assign(n, 0);
    for (int p = 0; p < n; ++p) t.dfs_pos[t.dfs[p]] = p;
    return LUMO_OK;
}

}  // namespace

extern "C" lumo_status lumo_tree_plan(int32_t n_req, const int32_t* node_off, const int32_t* parent,
                                      const int32_t* n_rows, int32_t policy, int32_t* blob,
                                      int64_t blob_words, lumo_plan* out) {
    lumo::clear_error();
    if (!out) return lumo::fail(LUMO_EINVAL, "lumo_tree_plan: out is NULL");
    std::memset(out, 0, sizeof(*out));
    if (n_req < 0) return lumo::fail(LUMO_EINVAL, "lumo_tree_plan: n_req < 0");
    if (!node_off) return lumo::fail(LUMO_EINVAL, "lumo_tree_plan: node_off is NULL");
    if (n_req > 0 && !n_rows) return lumo::fail(LUMO_EINVAL, "lumo_tree_plan: n_rows is NULL");
    if (policy < LUMO_POLICY_PATHS || policy > LUMO_POLICY_WY)
        return lumo::fail(LUMO_EINVAL, "lumo_tree_plan: unknown policy %d", policy);
    if (node_off[0] != 0) return lumo::fail(LUMO_EDESC, "lumo_tree_plan: node_off[0] must be 0");
    int64_t total_nodes = 0, total_rows = 0;
    for (int r = 0; r < n_req; ++r) {
        const int64_t n = (int64_t)node_off[r + 1] - node_off[r];
        if (n < 0) return lumo::fail(LUMO_EDESC, "lumo_tree_plan: node_off decreases at request %d", r);
        if (n_rows[r] < n)
            return lumo::fail(LUMO_EDESC, "lumo_tree_plan: request %d has %d rows for %lld nodes", r, n_rows[r],
                              (long long)n);
        total_nodes += n;
        total_rows += n_rows[r];
    }
    if (total_nodes > (1 << 28) || total_rows > (1 << 28))
        return lumo::fail(LUMO_ESHAPE, "lumo_tree_plan: more than 2^28 nodes or rows");
    if (total_nodes > 0 && !parent) return lumo::fail(LUMO_EINVAL, "lumo_tree_plan: parent is NULL");

    std::vector<ReqTree> tr(n_req);
    for (int r = 0; r < n_req; ++r) {
        lumo_status st = build_tree(r, node_off[r + 1] - node_off[r], parent + node_off[r], tr[r]);
        if (st != LUMO_OK) return st;
    }

    // ---- verification schedule -------------------------------------------------------
    std::vector<std::vector<SegOut>> levels;
    int n_cuts = 0;
    auto seg_at = [&](int level) -> std::vector<SegOut>& {
        if ((int)levels.size() <= level) levels.resize(level + 1);
        return levels[level];
    };
    std::vector<int> row_base(n_req + 1, 0);
    for (int r = 0; r < n_req; ++r) row_base[r + 1] = row_base[r] + n_rows[r];

    if (policy == LUMO_POLICY_PATHS) {
        // Disjoint first-child chains; a node with >= 2 children exports its state once
        // and every non-first child starts a chain at the next level from that cut.
        for (int r = 0; r < n_req; ++r) {
            const ReqTree& t = tr[r];
            if (!t.n) continue;
            std::vector<Chain> todo{{0, r, 0, -1}};
            for (size_t c = 0; c < todo.size(); ++c) {
                Chain ch = todo[c];
                SegOut s;
                s.req = r;
                s.src = ch.src;
                for (int x = ch.start; x >= 0; x = t.first_child(x)) {
                    s.rows.push_back(row_base[r] + t.slot[x]);
                    s.out.push_back(1);
                    int cut = -1;
                    if (t.n_children(x) >= 2) {
                        cut = n_cuts++;
                        for (int e = t.child_off[x] + 1; e < t.child_off[x + 1]; ++e)
                            todo.push_back({ch.level + 1, r, t.child[e], cut});
                    }
                    s.cut.push_back(cut);
                }
                seg_at(ch.level).push_back(std::move(s));
            }
        }
    } else if (policy == LUMO_POLICY_TWO_LEVEL) {
        // Level 0: the spine, exporting the state of each spine node that has children
        // off the spine. Level 1: every other leaf's path from its spine branch point.
        for (int r = 0; r < n_req; ++r) {
            const ReqTree& t = tr[r];
            if (!t.n) continue;
            std::vector<int> spine_cut(t.n, -1);
            SegOut s;
            s.req = r;
            s.src = -1;
            for (int x : t.spine) {
                s.rows.push_back(row_base[r] + t.slot[x]);
                s.out.push_back(1);
                if (t.n_children(x) >= 2) spine_cut[x] = n_cuts++;
                s.cut.push_back(spine_cut[x]);
            }
            seg_at(0).push_back(std::move(s));
            for (int leaf : t.leaves) {
                if (t.on_spine[leaf]) continue;
                std::vector<int> path;
                int x = leaf;
                while (!t.on_spine[x]) {
                    path.push_back(x);
                    x = t.parent[x];
                }
                std::reverse(path.begin(), path.end());
                SegOut b;
                b.req = r;
                b.src = spine_cut[x];
                for (int y : path) {
                    b.rows.push_back(row_base[r] + t.slot[y]);
                    b.out.push_back(t.owner[y] == leaf ? 1 : 0);
                    b.cut.push_back(-1);
                }
                seg_at(1).push_back(std::move(b));
            }
        }
    } else if (policy == LUMO_POLICY_RECOMPUTE) {
        for (int r = 0; r < n_req; ++r) {
            const ReqTree& t = tr[r];
            for (int leaf : t.leaves) {
                std::vector<int> path;
                for (int x = leaf; x >= 0; x = t.parent[x]) path.push_back(x);
                std::reverse(path.begin(), path.end());
                SegOut s;
                s.req = r;
                s.src = -1;
                for (int y : path) {
                    s.rows.push_back(row_base[r] + t.slot[y]);
                    s.out.push_back(t.owner[y] == leaf ? 1 : 0);
                    s.cut.push_back(-1);
                }
                seg_at(0).push_back(std::move(s));
            }
        }
    }

    // ---- sizes ------------------------------------------------------------------------
    lumo_plan p;
    std::memset(&p, 0, sizeof p);
    p.n_req = n_req;
    p.total_nodes = (int32_t)total_nodes;
    p.total_rows = (int32_t)total_rows;
    p.policy = policy;
    for (int r = 0; r < n_req; ++r) {
        const ReqTree& t = tr[r];
        p.max_nodes = std::max(p.max_nodes, t.n);
        for (int d : t.depth) p.max_depth = std::max(p.max_depth, d + 1);
        p.n_paths += (int32_t)t.leaves.size();
        p.n_spine += (int32_t)t.spine.size();
    }
    p.n_levels = (int32_t)levels.size();
    p.n_cuts = n_cuts;
    int64_t seg_nodes = 0;
    for (auto& lv : levels) {
        p.n_seg += (int32_t)lv.size();
        p.max_level_seg = std::max(p.max_level_seg, (int32_t)lv.size());
        for (auto& s : lv) {
            seg_nodes += (int64_t)s.rows.size();
            p.max_seg_len = std::max(p.max_seg_len, (int32_t)s.rows.size());
        }
    }
    if (seg_nodes > (1 << 28)) return lumo::fail(LUMO_ESHAPE, "lumo_tree_plan: schedule too large");
    p.n_seg_nodes = (int32_t)seg_nodes;

    int64_t w = 0;
    auto take = [&](int64_t n) {
        int64_t o = w;
        w += n;
        return (int32_t)o;
    };
    const int64_t N = total_nodes;
    p.o_node_off = take(n_req + 1);
    p.o_row_off = take(n_req + 1);
    p.o_req = take(N);
    p.o_parent = take(N);
    p.o_depth = take(N);
    p.o_slot = take(N);
    p.o_row = take(N);
    p.o_conv_src = take(4 * N);
    p.o_path_off = take(n_req + 1);
    p.o_path_leaf = take(p.n_paths);
    p.o_spine_off = take(n_req + 1);
    p.o_spine = take(p.n_spine);
    p.o_level_off = take(p.n_levels + 1);
    p.o_seg = take((int64_t)lumo::kSegWords * p.n_seg);
    p.o_seg_nodes = take((int64_t)lumo::kSegNodeWords * p.n_seg_nodes);
    p.o_dfs = take(N);
    p.o_dfs_pos = take(N);
    for (int r = 0; r < n_req; ++r) p.n_chunks += (tr[r].n + lumo::kPreChunk - 1) / lumo::kPreChunk;
    p.o_pre_row = take(N);
    p.o_pre_depth = take(N);
    p.o_pre_ci = take((int64_t)lumo::kPreCiWords * N);
    p.o_chunk_off = take(n_req + 1);
    p.o_chunk_stack = take((int64_t)lumo::kPreStack * p.n_chunks);
    p.o_vis = take(2 * N);
    if (w > (int64_t(1) << 30)) return lumo::fail(LUMO_ESHAPE, "lumo_tree_plan: plan too large");
    p.n_words = (int32_t)w;
    *out = p;
    if (!blob || blob_words < w)
        return lumo::fail(LUMO_ESPACE, "lumo_tree_plan: plan needs %lld words", (long long)w);

    // ---- write --------------------------------------------------------------------------
    int32_t* b = blob;
    for (int r = 0; r <= n_req; ++r) {
        b[p.o_node_off + r] = node_off[r];
        b[p.o_row_off + r] = row_base[r];
    }
    int np = 0, ns = 0;
    for (int r = 0; r < n_req; ++r) {
        const ReqTree& t = tr[r];
        const int base = node_off[r];
        for (int i = 0; i < t.n; ++i) {
            b[p.o_req + base + i] = r;
            b[p.o_parent + base + i] = t.parent[i];
            b[p.o_depth + base + i] = t.depth[i];
            b[p.o_slot + base + i] = t.slot[i];
            b[p.o_row + base + i] = row_base[r] + t.slot[i];
            b[p.o_dfs + base + i] = t.dfs[i];
            b[p.o_dfs_pos + base + i] = t.dfs_pos[i];
            // window = last four of (hist0, hist1, hist2, ancestry root..i), oldest first
            int anc[4] = {-1, -1, -1, -1};  // anc[3] = i, anc[2] = parent, ...
            int x = i;
            for (int s = 3; s >= 0 && x >= 0; --s) {
                anc[s] = x;
                x = t.parent[x];
            }
            const int d = t.depth[i];
            for (int s = 0; s < 4; ++s) {
                const int pos = d + s;  // position in (hist ++ ancestry); ancestry starts at 3
                b[p.o_conv_src + 4 * (base + i) + s] =
                    pos >= 3 ? row_base[r] + t.slot[anc[s]] : -1 - pos;
            }
        }
        b[p.o_path_off + r] = np;
        for (int leaf : t.leaves) b[p.o_path_leaf + np++] = leaf;
        b[p.o_spine_off + r] = ns;
        for (int x : t.spine) b[p.o_spine + ns++] = x;
    }
    b[p.o_path_off + n_req] = np;
    b[p.o_spine_off + n_req] = ns;
    // attention visibility: per node (slot order) its preorder interval [pos, pos + subtree)
    for (int r = 0; r < n_req; ++r) {
        const ReqTree& t = tr[r];
        const int base = node_off[r];
        std::vector<int> size(t.n, 1);
        for (int pos = t.n - 1; pos > 0; --pos) {
            const int x = t.dfs[pos];
            size[t.parent[x]] += size[x];
        }
        for (int x = 0; x < t.n; ++x) {
            b[p.o_vis + 2 * (base + t.slot[x])] = t.dfs_pos[x];
            b[p.o_vis + 2 * (base + t.slot[x]) + 1] = t.dfs_pos[x] + size[x];
        }
    }
    // preorder tables: per position the node's row and depth, and the Gram candidate
    // slot of every ancestor in the position's chunk of kPreChunk (one byte per depth)
    int nc = 0;
    for (int r = 0; r < n_req; ++r) {
        const ReqTree& t = tr[r];
        const int base = node_off[r];
        b[p.o_chunk_off + r] = nc;
        std::vector<int> anc;
        for (int pos = 0; pos < t.n; ++pos) {
            const int x = t.dfs[pos];
            const int c0 = pos - pos % lumo::kPreChunk;
            b[p.o_pre_row + base + pos] = row_base[r] + t.slot[x];
            b[p.o_pre_depth + base + pos] = t.depth[x];
            anc.assign(t.depth[x], 0);
            for (int y = t.parent[x], m = t.depth[x] - 1; y >= 0; y = t.parent[y], --m) anc[m] = y;
            uint32_t ci[lumo::kPreCiWords] = {};
            for (int m = 0; m < 4 * lumo::kPreCiWords; ++m) {
                uint32_t slot = 0xffu;  // no ancestor at this depth (or deeper than the table)
                if (m < t.depth[x]) {
                    const int ap = t.dfs_pos[anc[m]];
                    slot = ap >= c0 ? (uint32_t)(lumo::kPreStack + (ap - c0)) : (uint32_t)m;
                }
                ci[m / 4] |= slot << (8 * (m % 4));
            }
            for (int w = 0; w < lumo::kPreCiWords; ++w) b[p.o_pre_ci + (int64_t)lumo::kPreCiWords * (base + pos) + w] = (int32_t)ci[w];
            if (pos == c0) {  // chunk start: the path stack is the first node's ancestry
                int32_t* cs = b + p.o_chunk_stack + (int64_t)lumo::kPreStack * nc;
                for (int m = 0; m < lumo::kPreStack; ++m)
                    cs[m] = m < t.depth[x] ? row_base[r] + t.slot[anc[m]] : -1;
                ++nc;
            }
        }
    }
    b[p.o_chunk_off + n_req] = nc;
    int si = 0, ei = 0;
    for (int lv = 0; lv < p.n_levels; ++lv) {
        b[p.o_level_off + lv] = si;
        for (auto& s : levels[lv]) {
            int32_t* sr = b + p.o_seg + lumo::kSegWords * si;
            sr[0] = s.req;
            sr[1] = s.src;
            sr[2] = ei;
            sr[3] = (int32_t)s.rows.size();
            for (size_t e = 0; e < s.rows.size(); ++e) {
                int32_t* en = b + p.o_seg_nodes + lumo::kSegNodeWords * ei++;
                en[0] = s.rows[e];
                en[1] = s.out[e];
                en[2] = s.cut[e];
            }
            ++si;
        }
    }
    b[p.o_level_off + p.n_levels] = si;
    return LUMO_OK;
}
