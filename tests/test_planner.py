"""The library's host planner (lumo_tree_plan) against the oracle's independent
derivations (bit-exact), and the verification schedules of every policy against the
ancestry contract: each segment starts from the state of its first node's parent,
consecutive entries are parent and child, every node's output is written exactly
once, every cut is exported once before any level that reads it."""
import numpy as np
import pytest

import paper_2609_23900_amd as L
from lumo_synth import configs, trees
from oracle import plan as oplan

POLICIES = [L.LUMO_POLICY_PATHS, L.LUMO_POLICY_TWO_LEVEL, L.LUMO_POLICY_RECOMPUTE,
            L.LUMO_POLICY_WY]


def _forest(seed, n_req=None):
    rng = np.random.default_rng(seed)
    n_req = n_req or int(rng.integers(1, 6))
    parents, rows = [], []
    for _ in range(n_req):
        kind = int(rng.integers(0, 4))
        if kind == 0:
            p = trees.chain(int(rng.integers(1, 20)))
        elif kind == 1:
            p = trees.random_tree(rng, int(rng.integers(2, 70)), int(rng.integers(2, 10)),
                                  trees.bmax_uniform(int(rng.integers(1, 5))))
        elif kind == 2:
            p = trees.random_tree(rng, int(rng.integers(2, 120)), 16, trees.bmax_root_skewed)
        else:
            p = np.array([-1], np.int32)
        parents.append(p)
        rows.append(len(p) + int(rng.integers(0, 4)))
    node_off = np.concatenate([[0], np.cumsum([len(p) for p in parents])]).astype(np.int32)
    return parents, np.array(rows, np.int32), node_off


def _check_against_oracle(parents, n_rows, node_off, policy):
    plan, blob = L.lumo_tree_plan(node_off, np.concatenate(parents), n_rows, policy)
    N = int(node_off[-1])
    row_off = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    sec = lambda name, n: blob[getattr(plan, "o_" + name):getattr(plan, "o_" + name) + n]
    assert plan.total_nodes == N and plan.total_rows == int(n_rows.sum())
    assert np.array_equal(sec("node_off", len(parents) + 1), node_off)
    assert np.array_equal(sec("row_off", len(parents) + 1), row_off)
    leaves, spines = [], []
    for r, par in enumerate(parents):
        b = int(node_off[r])
        n = len(par)
        rows = oplan.rows_of(par, int(row_off[r]))
        assert list(sec("req", N)[b:b + n]) == [r] * n
        assert list(sec("parent", N)[b:b + n]) == [int(x) for x in par]
        assert list(sec("depth", N)[b:b + n]) == oplan.depth(par)
        assert list(sec("slot", N)[b:b + n]) == oplan.slot_map(par)
        assert list(sec("row", N)[b:b + n]) == rows
        assert sec("conv_src", 4 * N).reshape(-1, 4)[b:b + n].tolist() == oplan.conv_sources(par, rows)
        leaves += oplan.leaves(par)
        spines += oplan.spine(par)
        # depth-first preorder: a permutation where every subtree is contiguous
        dfs = list(sec("dfs", N)[b:b + n])
        pos = list(sec("dfs_pos", N)[b:b + n])
        assert sorted(dfs) == list(range(n)) and all(pos[dfs[k]] == k for k in range(n))
        if n:
            assert dfs[0] == 0
            size = [1] * n
            for i in range(n - 1, 0, -1):
                size[par[i]] += size[i]
            for i in range(n):
                sub = set(dfs[pos[i]:pos[i] + size[i]])
                assert all(i in oplan.ancestry(par, x) for x in sub)
            ch = oplan.children(par)
            for i in range(n):   # children visited in increasing id
                cp = [pos[c] for c in ch[i]]
                assert cp == sorted(cp)
    # preorder tables used by the WY kernels (meaningful for paths of <= 17 nodes)
    if plan.max_depth <= 17:
        pre_ci = sec("pre_ci", 4 * N).astype(np.uint32).view(np.uint8).reshape(N, 16)
        chunk_off = sec("chunk_off", len(parents) + 1)
        stacks = sec("chunk_stack", 16 * plan.n_chunks).reshape(-1, 16)
        for r, par in enumerate(parents):
            b = int(node_off[r])
            rows = oplan.rows_of(par, int(row_off[r]))
            dfs = list(sec("dfs", N)[b:b + len(par)])
            dep = oplan.depth(par)
            assert int(chunk_off[r + 1] - chunk_off[r]) == (len(par) + 31) // 32
            for pos, x in enumerate(dfs):
                assert sec("pre_row", N)[b + pos] == rows[x]
                assert sec("pre_depth", N)[b + pos] == dep[x]
                anc = oplan.ancestry(par, x)[:-1]
                c0 = pos - pos % 32
                for m in range(16):
                    if m < len(anc):
                        ap = dfs.index(anc[m])
                        want = 16 + ap - c0 if ap >= c0 else m
                    else:
                        want = 0xFF
                    assert pre_ci[b + pos, m] == want
                if pos == c0:
                    st = stacks[chunk_off[r] + pos // 32]
                    fanc = oplan.ancestry(par, x)[:-1]
                    assert list(st) == [rows[fanc[m]] if m < len(fanc) else -1 for m in range(16)]
    assert list(sec("path_leaf", plan.n_paths)) == leaves
    assert list(sec("spine", plan.n_spine)) == spines
    assert plan.max_depth == max(max(oplan.depth(p)) + 1 for p in parents)
    return plan, blob


def _check_schedule(parents, n_rows, node_off, plan, blob):
    row_off = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    node_of_row = {}
    for r, par in enumerate(parents):
        for i, rw in enumerate(oplan.rows_of(par, int(row_off[r]))):
            node_of_row[rw] = (r, i)
    lvl = blob[plan.o_level_off:plan.o_level_off + plan.n_levels + 1]
    seg = blob[plan.o_seg:plan.o_seg + 4 * plan.n_seg].reshape(-1, 4)
    ent = blob[plan.o_seg_nodes:plan.o_seg_nodes + 3 * plan.n_seg_nodes].reshape(-1, 3)
    writes = {}
    cut_owner, cut_level = {}, {}
    for lv in range(plan.n_levels):
        for s in range(lvl[lv], lvl[lv + 1]):
            req, src, first, ln = seg[s]
            assert ln >= 1
            nodes = [node_of_row[int(ent[e, 0])] for e in range(first, first + ln)]
            assert all(rq == req for rq, _ in nodes)
            par = parents[req]
            ids = [i for _, i in nodes]
            for a, b in zip(ids, ids[1:]):
                assert par[b] == a
            if src < 0:
                assert ids[0] == 0
            else:
                assert cut_level[src] < lv, "cut read in the level that writes it"
                assert cut_owner[src] == (req, int(par[ids[0]]))
            for e, (rq, i) in zip(range(first, first + ln), nodes):
                if ent[e, 1]:
                    writes[(rq, i)] = writes.get((rq, i), 0) + 1
                if ent[e, 2] >= 0:
                    c = int(ent[e, 2])
                    assert c not in cut_owner, "cut exported twice"
                    cut_owner[c] = (rq, i)
                    cut_level[c] = lv
    all_nodes = {(r, i) for r, p in enumerate(parents) for i in range(len(p))}
    if plan.policy == L.LUMO_POLICY_WY:
        assert plan.n_seg == 0 and not writes
    else:
        assert set(writes) == all_nodes and set(writes.values()) <= {1}
    assert len(cut_owner) == plan.n_cuts


def test_fig1_plan():
    gd_parent = trees.FIG1_PARENT
    plan, blob = _check_against_oracle([gd_parent], np.array([7], np.int32),
                                       np.array([0, 7], np.int32), L.LUMO_POLICY_PATHS)
    assert plan.n_cuts == 2 and plan.n_levels == 2 and plan.n_seg == 3


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("seed", range(12))
def test_random_forests(policy, seed):
    parents, n_rows, node_off = _forest(seed)
    plan, blob = _check_against_oracle(parents, n_rows, node_off, policy)
    _check_schedule(parents, n_rows, node_off, plan, blob)


@pytest.mark.parametrize("name", ["tiny", "layer1", "batched", "widedeep", "chainmix", "paper28"])
@pytest.mark.parametrize("policy", POLICIES)
def test_config_plans(name, policy):
    wl, _ = configs.topology(name)
    plan, blob = _check_against_oracle(wl.parents, wl.n_rows, wl.node_off, policy)
    _check_schedule(wl.parents, wl.n_rows, wl.node_off, plan, blob)
    if policy == L.LUMO_POLICY_RECOMPUTE:
        assert plan.n_cuts == 0 and plan.n_levels == 1 and plan.n_seg == plan.n_paths
    if policy == L.LUMO_POLICY_PATHS:
        assert plan.n_seg_nodes == plan.total_nodes


def test_empty_and_single():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), 0)
    assert plan.n_req == 0 and plan.total_nodes == 0 and plan.n_seg == 0
    plan, blob = L.lumo_tree_plan(np.array([0, 0, 1], np.int32), np.array([-1], np.int32),
                                  np.array([2, 1], np.int32), 0)
    assert plan.total_nodes == 1 and plan.total_rows == 3 and plan.n_seg == 1


@pytest.mark.parametrize("parent,status", [
    ([0], L.LUMO_EDESC), ([-1, 1], L.LUMO_EDESC), ([-1, 2, 0], L.LUMO_EDESC),
    ([-1, -1], L.LUMO_EDESC), ([-1, 0, 5], L.LUMO_EDESC)])
def test_malformed_trees_rejected(parent, status):
    n = len(parent)
    with pytest.raises(L.LumoError) as e:
        L.lumo_tree_plan(np.array([0, n], np.int32), np.array(parent, np.int32),
                         np.array([n], np.int32), 0)
    assert e.value.status == status


def test_rows_fewer_than_nodes_rejected():
    with pytest.raises(L.LumoError) as e:
        L.lumo_tree_plan(np.array([0, 3], np.int32), np.array([-1, 0, 0], np.int32),
                         np.array([2], np.int32), 0)
    assert e.value.status == L.LUMO_EDESC


def test_bad_policy_rejected():
    with pytest.raises(L.LumoError) as e:
        L.lumo_tree_plan(np.array([0, 1], np.int32), np.array([-1], np.int32),
                         np.array([1], np.int32), 9)
    assert e.value.status == L.LUMO_EINVAL


def test_visibility_intervals_match_ancestry():
    """vis[slot] is the preorder interval of the node's subtree: a is an ancestor-or-self
    of i exactly when i's position falls in a's interval (checked by brute force)."""
    rng = np.random.default_rng(91)
    parents = [trees.random_tree(rng, n, 6, trees.bmax_uniform(4)) for n in (1, 9, 40)] + [trees.FIG1_PARENT]
    node_off = np.concatenate([[0], np.cumsum([len(p) for p in parents])]).astype(np.int32)
    plan, blob = L.lumo_tree_plan(node_off, np.concatenate(parents), np.array([len(p) for p in parents], np.int32))
    vis = blob[plan.o_vis:plan.o_vis + 2 * plan.total_nodes].reshape(-1, 2)
    for r, par in enumerate(parents):
        slot = oplan.slot_map(par)
        base = int(node_off[r])
        for i in range(len(par)):
            anc = set(oplan.ancestry(par, i))
            for a in range(len(par)):
                lo, hi = vis[base + slot[a]]
                assert (lo <= vis[base + slot[i]][0] < hi) == (a in anc), (r, a, i)
