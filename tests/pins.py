"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each pin raises AssertionError when the oracle disagrees. They are collected as
tests in test_oracle_pins.py and re-run against deliberately mutated copies of the
oracle in test_oracle_mutations.py (every plausible mistake must trip a pin).

Independent routes used here (none re-types the oracle's own loop):
  * hand-derived exact values of Eq. (2)-(3) (tests/golden/*.json)
  * closed forms: beta=0/alpha=1 keeps the state; beta=1, q=k, |k|=1 returns v;
    alpha=0 gives beta (k.q) v
  * the matrix form S <- alpha S (I - beta k k^T) + beta v k^T of a chain
  * the WY / triangular-solve closed form of the recurrence on a tree
    (delta from numpy.linalg.solve over the ancestor-masked Gram system)
  * numpy.convolve for the causal convolution along a chain
  * structural invariants: identical sibling subtrees, commit == node state,
    permutation equivariance over value rows, head independence, off-path poisoning
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import oracle
from lumo_synth import configs, trees
from lumo_synth import operands as ops
from lumo_synth.configs import Workload

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def make_wl(parents, *, d_k, d_v, h_k=1, h_v=1, n_layers=1, n_rows=None, channels=4,
            op_dtype=0, max_path=None):
    parents = [np.asarray(p, dtype=np.int32) for p in parents]
    n_rows = np.array([len(p) for p in parents] if n_rows is None else n_rows, dtype=np.int32)
    mp = max_path or max(int(trees.depths(p).max()) + 1 for p in parents)
    return Workload(name="custom", n_req=len(parents), n_layers=n_layers, h_k=h_k, h_v=h_v,
                    d_k=d_k, d_v=d_v, op_dtype=op_dtype, parents=parents, n_rows=n_rows,
                    accepted=np.full(len(parents), -1, np.int32), max_path=mp,
                    channels=channels)


def random_arrays(wl, rng, *, alpha_direct=False):
    """float32 operands in the boundary layouts (row = physical slot)."""
    L, R = wl.n_layers, wl.total_rows
    k = rng.standard_normal((L, R, wl.h_k, wl.d_k))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    a = dict(
        q=rng.standard_normal((L, R, wl.h_k, wl.d_k)).astype(np.float32),
        k=k.astype(np.float32),
        v=rng.standard_normal((L, R, wl.h_v, wl.d_v)).astype(np.float32),
        beta=(1 / (1 + np.exp(-rng.standard_normal((L, R, wl.h_v))))).astype(np.float32),
        state0=(0.1 * rng.standard_normal((wl.n_req, L, wl.h_v, wl.d_k, wl.d_v))).astype(np.float32),
    )
    z = rng.standard_normal((L, R, wl.h_v))
    a["g"] = (np.exp(-np.logaddexp(0, z)) if alpha_direct else -np.logaddexp(0, z)).astype(np.float32)
    return a


def _rows(wl, r):
    return oracle.plan.rows_of(wl.parents[r], int(wl.row_off[r]))


def _alpha(wl, a, l, row, h, alpha_direct):
    g = float(a["g"][l, row, h])
    return g if alpha_direct else float(np.exp(np.float64(g)))


# --------------------------------------------------------------------------- hand values

def pin_hand_scalar():
    gd = load_golden("hand_scalar.json")
    wl = make_wl([gd["parent"]], d_k=1, d_v=1)
    rows = _rows(wl, 0)
    a = dict(q=np.zeros((1, 3, 1, 1), np.float32), k=np.zeros((1, 3, 1, 1), np.float32),
             v=np.zeros((1, 3, 1, 1), np.float32), g=np.zeros((1, 3, 1), np.float32),
             beta=np.zeros((1, 3, 1), np.float32),
             state0=np.full((1, 1, 1, 1, 1), float(Fraction(gd["state0"])), np.float32))
    for i, nd in enumerate(gd["nodes"]):
        rw = rows[i]
        a["q"][0, rw, 0, 0] = float(Fraction(nd["q"]))
        a["k"][0, rw, 0, 0] = float(Fraction(nd["k"]))
        a["v"][0, rw, 0, 0] = float(Fraction(nd["v"]))
        a["g"][0, rw, 0] = float(Fraction(nd["alpha"]))
        a["beta"][0, rw, 0] = float(Fraction(nd["beta"]))
    wl.arrays = a
    o, st = oracle.verify_nodes(wl, 0, 0, 0, [0, 1, 2], gate_is_alpha=True, want_state=True)
    for i, nd in enumerate(gd["nodes"]):
        assert o[i, 0] == float(Fraction(nd["o"])), (nd["name"], o[i, 0])
        assert st[i, 0, 0] == float(Fraction(nd["state"])), (nd["name"], st[i, 0, 0])


def pin_hand_2x2():
    gd = load_golden("hand_2x2.json")
    wl = make_wl([[-1]], d_k=2, d_v=2)
    a = dict(q=np.array(gd["q"], np.float32).reshape(1, 1, 1, 2),
             k=np.array(gd["k"], np.float32).reshape(1, 1, 1, 2),
             v=np.array(gd["v"], np.float32).reshape(1, 1, 1, 2),
             g=np.full((1, 1, 1), gd["alpha"], np.float32),
             beta=np.full((1, 1, 1), gd["beta"], np.float32),
             state0=np.array(gd["state0_key_major"], np.float32).reshape(1, 1, 1, 2, 2))
    wl.arrays = a
    o, st = oracle.verify_nodes(wl, 0, 0, 0, [0], gate_is_alpha=True, want_state=True)
    assert np.array_equal(o[0], np.array(gd["o"], np.float64)), o
    assert np.array_equal(st[0], np.array(gd["state_key_major"], np.float64)), st


# --------------------------------------------------------------------------- closed forms

def pin_beta0_alpha1_identity():
    """beta = 0 and alpha = 1: the state is returned bit for bit, o = S0 q."""
    rng = np.random.default_rng(11)
    wl = make_wl([trees.FIG1_PARENT], d_k=8, d_v=6)
    a = random_arrays(wl, rng, alpha_direct=True)
    a["beta"][:] = 0.0
    a["g"][:] = 1.0
    wl.arrays = a
    nodes = list(range(7))
    o, st = oracle.verify_nodes(wl, 0, 0, 0, nodes, gate_is_alpha=True, want_state=True)
    S0 = a["state0"][0, 0, 0].astype(np.float64)
    rows = _rows(wl, 0)
    for i in nodes:
        assert np.array_equal(st[i], S0)
        want = S0.T @ a["q"][0, rows[i], 0].astype(np.float64)
        np.testing.assert_allclose(o[i], want, rtol=0, atol=1e-14)


def pin_delta_rule_writes_v():
    """beta = 1, q = k with |k| = 1 exactly: o = v whatever alpha and the parent state."""
    rng = np.random.default_rng(12)
    wl = make_wl([trees.FIG1_PARENT], d_k=4, d_v=5)
    a = random_arrays(wl, rng)
    signs = rng.choice([-0.5, 0.5], size=a["k"].shape).astype(np.float32)
    a["k"] = signs                      # (+-1/2, ..., +-1/2) has norm exactly 1 at d_k = 4
    a["q"] = signs.copy()
    a["beta"][:] = 1.0
    wl.arrays = a
    o = oracle.verify_nodes(wl, 0, 0, 0, list(range(7)))
    rows = _rows(wl, 0)
    for i in range(7):
        np.testing.assert_allclose(o[i], a["v"][0, rows[i], 0], rtol=0, atol=1e-13)


def pin_alpha0_forgets():
    """alpha = 0: R = beta v k^T, o = beta (k . q) v, independent of the ancestry."""
    rng = np.random.default_rng(13)
    wl = make_wl([trees.FIG1_PARENT], d_k=6, d_v=3)
    a = random_arrays(wl, rng, alpha_direct=True)
    a["g"][:] = 0.0
    wl.arrays = a
    o = oracle.verify_nodes(wl, 0, 0, 0, list(range(7)), gate_is_alpha=True)
    rows = _rows(wl, 0)
    for i in range(7):
        rw = rows[i]
        k = a["k"][0, rw, 0].astype(np.float64)
        q = a["q"][0, rw, 0].astype(np.float64)
        want = float(a["beta"][0, rw, 0]) * float(k @ q) * a["v"][0, rw, 0].astype(np.float64)
        np.testing.assert_allclose(o[i], want, rtol=1e-13, atol=1e-15)


# --------------------------------------------------------------------------- independent forms

def chain_matrix_form(S0_key_major, alphas, betas, ks, vs, qs):
    """Sequential scan in the form S <- alpha S (I - beta k k^T) + beta v k^T, o = S q."""
    R = S0_key_major.T.astype(np.float64).copy()
    dk = R.shape[1]
    outs, states = [], []
    for a, b, k, v, q in zip(alphas, betas, ks, vs, qs):
        R = a * R @ (np.eye(dk) - b * np.outer(k, k)) + b * np.outer(v, k)
        outs.append(R @ q)
        states.append(R.T.copy())
    return np.array(outs), np.array(states)


def tree_wy_form(parent, S0_key_major, alphas, betas, K, V, Q):
    """Closed form R_t = gamma_t R0 + sum_{s anc-or-self t} Gamma(s->t) delta_s k_s^T.

    delta solves the ancestor-masked unit-triangular system
      delta_t + beta_t sum_{s strict anc t} Gamma(s->t) (k_s.k_t) delta_s
          = beta_t (v_t - gamma_t R0 k_t)
    with gamma_t the product of alpha along root..t and Gamma(s->t) the product over
    the nodes after s up to t. Solved with numpy.linalg.solve; outputs
      o_t = gamma_t R0 q_t + sum_{s anc-or-self t} Gamma(s->t) (k_s.q_t) delta_s.
    """
    n = len(parent)
    R0 = S0_key_major.T.astype(np.float64)
    anc = [oracle.plan.ancestry(parent, t) for t in range(n)]

    def Gam(s, t):
        path = anc[t]
        return float(np.prod([alphas[x] for x in path[path.index(s) + 1:]]))

    gamma = np.array([float(np.prod([alphas[x] for x in anc[t]])) for t in range(n)])
    A = np.eye(n)
    for t in range(n):
        for s in anc[t][:-1]:
            A[t, s] = betas[t] * Gam(s, t) * float(K[s] @ K[t])
    rhs = np.stack([betas[t] * (V[t] - gamma[t] * (R0 @ K[t])) for t in range(n)])
    delta = np.linalg.solve(A, rhs)
    O = np.stack([gamma[t] * (R0 @ Q[t]) + sum(Gam(s, t) * float(K[s] @ Q[t]) * delta[s]
                                               for s in anc[t]) for t in range(n)])
    return O


def _node_operands(wl, a, r, l, h, alpha_direct=False):
    rows = _rows(wl, r)
    hk = h // (wl.h_v // wl.h_k)
    n = len(wl.parents[r])
    al = [_alpha(wl, a, l, rows[i], h, alpha_direct) for i in range(n)]
    be = [float(a["beta"][l, rows[i], h]) for i in range(n)]
    K = np.stack([a["k"][l, rows[i], hk].astype(np.float64) for i in range(n)])
    Q = np.stack([a["q"][l, rows[i], hk].astype(np.float64) for i in range(n)])
    V = np.stack([a["v"][l, rows[i], h].astype(np.float64) for i in range(n)])
    return al, be, K, Q, V


def pin_chain_equals_matrix_scan():
    rng = np.random.default_rng(21)
    wl = make_wl([trees.chain(9)], d_k=7, d_v=5, h_k=1, h_v=2)
    a = random_arrays(wl, rng)
    wl.arrays = a
    for h in range(2):
        al, be, K, Q, V = _node_operands(wl, a, 0, 0, h)
        want_o, want_s = chain_matrix_form(a["state0"][0, 0, h], al, be, K, V, Q)
        o, st = oracle.verify_nodes(wl, 0, 0, h, list(range(9)), want_state=True)
        np.testing.assert_allclose(o, want_o, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(st, want_s, rtol=1e-12, atol=1e-13)


def pin_tree_equals_wy_closed_form():
    rng = np.random.default_rng(22)
    par = trees.random_tree(rng, 20, 6, trees.bmax_uniform(3))
    wl = make_wl([par, trees.FIG1_PARENT], d_k=6, d_v=5, h_k=2, h_v=4, n_layers=2,
                 n_rows=[22, 8])
    a = random_arrays(wl, rng)
    wl.arrays = a
    for (r, l, h) in [(0, 0, 0), (0, 1, 3), (1, 1, 1), (1, 0, 2)]:
        al, be, K, Q, V = _node_operands(wl, a, r, l, h)
        want = tree_wy_form(wl.parents[r], a["state0"][r, l, h], al, be, K, V, Q)
        o = oracle.verify_nodes(wl, r, l, h, list(range(len(wl.parents[r]))))
        np.testing.assert_allclose(o, want, rtol=1e-11, atol=1e-12)


def pin_paths_equal_chain_scans():
    """Every node's output equals the chain scan of its own root-to-node path."""
    rng = np.random.default_rng(23)
    par = trees.random_tree(rng, 16, 5, trees.bmax_uniform(4))
    wl = make_wl([par], d_k=5, d_v=4)
    a = random_arrays(wl, rng)
    wl.arrays = a
    al, be, K, Q, V = _node_operands(wl, a, 0, 0, 0)
    o = oracle.verify_nodes(wl, 0, 0, 0, list(range(16)))
    for path in oracle.plan.paths(par):
        ch_o, _ = chain_matrix_form(a["state0"][0, 0, 0], [al[x] for x in path],
                                    [be[x] for x in path], K[path], V[path], Q[path])
        for pos, node in enumerate(path):
            np.testing.assert_allclose(o[node], ch_o[pos], rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------------------- invariants

def pin_identical_sibling_subtrees():
    """Two sibling subtrees carrying identical operands give bit-identical outputs."""
    par = [-1, 0, 0, 1, 2, 3, 4, 1, 2]   # subtrees of 1 and 2 mirror each other: 1->{3,7}, 3->5; 2->{4,8}, 4->6
    rng = np.random.default_rng(31)
    wl = make_wl([par], d_k=6, d_v=6, h_k=1, h_v=2)
    a = random_arrays(wl, rng)
    rows = _rows(wl, 0)
    for x, y in ((1, 2), (3, 4), (5, 6), (7, 8)):
        for key in ("q", "k", "v", "g", "beta"):
            a[key][:, rows[y]] = a[key][:, rows[x]]
    wl.arrays = a
    for h in range(2):
        o = oracle.verify_nodes(wl, 0, 0, h, list(range(9)))
        for x, y in ((1, 2), (3, 4), (5, 6), (7, 8)):
            assert np.array_equal(o[x], o[y])


def pin_commit_equals_node_state():
    """Replaying the accepted path reproduces that node's verified state bit for bit."""
    rng = np.random.default_rng(32)
    par = trees.random_tree(rng, 12, 5, trees.bmax_uniform(3))
    wl = make_wl([par], d_k=5, d_v=7, h_k=1, h_v=2, n_layers=2, max_path=5)
    a = random_arrays(wl, rng)
    wl.arrays = a
    for node in range(12):
        st_c, po, pl = oracle.commit(wl, accepted=[node])
        assert list(po[0][:pl[0]]) == oracle.plan.ancestry(par, node)
        for l in range(2):
            for h in range(2):
                _, st = oracle.verify_nodes(wl, 0, l, h, [node], want_state=True)
                assert np.array_equal(st_c[0, l, h], st[0])
    st_c, po, pl = oracle.commit(wl, accepted=[-1])
    assert pl[0] == 0 and np.all(po == -1)
    assert np.array_equal(st_c, a["state0"].astype(np.float64))


def pin_value_row_permutation():
    rng = np.random.default_rng(33)
    wl = make_wl([trees.FIG1_PARENT], d_k=5, d_v=6)
    a = random_arrays(wl, rng)
    wl.arrays = a
    o = oracle.verify_nodes(wl, 0, 0, 0, list(range(7)))
    perm = rng.permutation(6)
    b = {k: v.copy() for k, v in a.items()}
    b["v"] = a["v"][..., perm]
    b["state0"] = a["state0"][..., perm]
    o2 = oracle.verify_nodes(wl, 0, 0, 0, list(range(7)), arrays=b)
    assert np.array_equal(o2, o[:, perm])


def pin_head_independence():
    rng = np.random.default_rng(34)
    wl = make_wl([trees.FIG1_PARENT], d_k=4, d_v=4, h_k=2, h_v=4)
    a = random_arrays(wl, rng)
    wl.arrays = a
    base = [oracle.verify_nodes(wl, 0, 0, h, list(range(7))) for h in range(4)]
    b = {k: v.copy() for k, v in a.items()}
    b["v"][:, :, 3] += 1.0
    b["state0"][:, :, 3] *= 2
    b["k"][:, :, 1] = b["k"][:, :, 1][..., ::-1].copy()   # key head 1 feeds value heads 2, 3
    for h in range(2):
        assert np.array_equal(oracle.verify_nodes(wl, 0, 0, h, list(range(7)), arrays=b), base[h])
    assert not np.array_equal(oracle.verify_nodes(wl, 0, 0, 2, list(range(7)), arrays=b), base[2])


def pin_head_grouping():
    """Value head h reads key head h // (h_v / h_k) (contiguous groups)."""
    rng = np.random.default_rng(35)
    wl = make_wl([[-1, 0]], d_k=3, d_v=3, h_k=2, h_v=4)
    a = random_arrays(wl, rng)
    wl.arrays = a
    for h in range(4):
        al, be, K, Q, V = _node_operands(wl, a, 0, 0, h)
        want, _ = chain_matrix_form(a["state0"][0, 0, h], al, be, K, V, Q)
        np.testing.assert_allclose(oracle.verify_nodes(wl, 0, 0, h, [0, 1]), want, rtol=1e-12)


def pin_off_path_poison():
    """NaN operands on rows off the accepted path leave the published state unchanged."""
    rng = np.random.default_rng(36)
    wl = make_wl([trees.FIG1_PARENT], d_k=4, d_v=4, max_path=4)
    a = random_arrays(wl, rng)
    wl.arrays = a
    st, po, pl = oracle.commit(wl, accepted=[4])
    b = {k: v.copy() for k, v in a.items()}
    rows = _rows(wl, 0)
    for node in (2, 3, 5, 6):
        for key in ("k", "v", "g", "beta", "q"):
            b[key][:, rows[node]] = np.nan
    st2, _, _ = oracle.commit(wl, accepted=[4], arrays=b)
    assert np.array_equal(st, st2)


def pin_fig1_worked_commit():
    """Fig. 1: accepting d publishes S(m a d): the replay of m, a, d from S0."""
    wl = configs.build("tiny", with_conv=False)
    st, po, pl = oracle.commit(wl)
    gd = load_golden("fig1_descriptor.json")
    assert list(po[0][:pl[0]]) == gd["accepted_path"] and pl[0] == gd["accepted_len"]
    al, be, K, Q, V = _node_operands(wl, wl.arrays, 0, 0, 0)
    p = gd["accepted_path"]
    _, states = chain_matrix_form(wl.arrays["state0"][0, 0, 0], [al[x] for x in p],
                                  [be[x] for x in p], K[p], V[p], Q[p])
    np.testing.assert_allclose(st[0, 0, 0], states[-1], rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------------------- batch drivers

def _batch_wl(rng, n_layers=2, h_k=2, h_v=4, d_k=5, d_v=3, channels=3):
    """Three requests laid out as the boundary lays them out: a random tree with two pad
    rows, a request without nodes (two pad rows), and the Fig. 1 tree with two pad
    rows, so that a node's physical row differs from its id and from its position in
    the flat node list, and each request's rows start at its own offset."""
    parents = [trees.random_tree(rng, 11, 5, trees.bmax_uniform(3)), np.zeros(0, np.int32),
               trees.FIG1_PARENT.copy()]
    wl = make_wl(parents, d_k=d_k, d_v=d_v, h_k=h_k, h_v=h_v, n_layers=n_layers,
                 n_rows=[13, 2, 9], channels=channels, max_path=6)
    return wl


def _hand_rows(parents, n_rows):
    """Physical rows written out from the layout rule (spine first by depth, then the
    other nodes in id order) and the per-request row offsets, without the planner."""
    out, base = [], 0
    for par, nr in zip(parents, n_rows):
        n = len(par)
        spine = []
        if n:
            spine = [0]
            while True:
                kids = [i for i in range(n) if par[i] == spine[-1]]
                if not kids:
                    break
                spine.append(min(kids))
        order = spine + [i for i in range(n) if i not in spine]
        slot = [0] * n
        for pos, node in enumerate(order):
            slot[node] = pos
        out.append([base + slot[i] for i in range(n)])
        base += nr
    return out


def pin_verify_all_batch_layout():
    """Every (request, layer, value head) instance of a padded three-request batch, one
    request without nodes: each node's output sits at its own physical row and equals
    the WY closed form of its request's tree; pad rows stay unwritten."""
    rng = np.random.default_rng(51)
    wl = _batch_wl(rng)
    a = random_arrays(wl, rng)
    wl.arrays = a
    o = oracle.verify_all(wl, n_threads=2)
    rows = _hand_rows(wl.parents, wl.n_rows)
    written = np.zeros((wl.n_layers, wl.total_rows, wl.h_v), bool)
    for r in (0, 2):
        for l in range(wl.n_layers):
            for h in range(wl.h_v):
                al, be, K, Q, V = _node_operands(wl, a, r, l, h)
                want = tree_wy_form(wl.parents[r], a["state0"][r, l, h], al, be, K, V, Q)
                for i, rw in enumerate(rows[r]):
                    np.testing.assert_allclose(o[l, rw, h], want[i], rtol=1e-11, atol=1e-12)
                    written[l, rw, h] = True
    assert np.all(np.isnan(o[~written])), "pad rows or the empty request were written"


def pin_commit_batch_layout():
    """Per request of the padded batch, the published state of every (layer, head) is
    the chain scan of that request's own accepted path; the request without nodes and an
    invalid selection publish the state unchanged; path_out / path_len are the
    hand-derived ancestries (-1 for a selection outside the tree)."""
    rng = np.random.default_rng(52)
    wl = _batch_wl(rng)
    a = random_arrays(wl, rng)
    wl.arrays = a
    par0 = wl.parents[0]
    deep = int(np.argmax(trees.depths(par0)))
    want_path0 = []
    x = deep
    while x != -1:
        want_path0.insert(0, x)
        x = int(par0[x])
    for acc, want2, want_len2 in (([deep, -1, 6], [0, 1, 3, 6], 4), ([deep, -1, 7], [], -1),
                                  ([deep, -1, -2], [], -1), ([deep, -1, 2], [0, 2], 2)):
        st, po, pl = oracle.commit(wl, accepted=np.array(acc, np.int32), max_path=6, n_threads=2)
        assert pl.tolist() == [len(want_path0), 0, want_len2]
        assert po[0].tolist() == want_path0 + [-1] * (6 - len(want_path0))
        assert po[1].tolist() == [-1] * 6
        assert po[2].tolist() == want2 + [-1] * (6 - len(want2))
        for l in range(wl.n_layers):
            for h in range(wl.h_v):
                assert np.array_equal(st[1, l, h], a["state0"][1, l, h].astype(np.float64))
                for r, path in ((0, want_path0), (2, want2)):
                    if not path:
                        assert np.array_equal(st[r, l, h], a["state0"][r, l, h].astype(np.float64))
                        continue
                    al, be, K, Q, V = _node_operands(wl, a, r, l, h)
                    _, states = chain_matrix_form(a["state0"][r, l, h], [al[x] for x in path],
                                                  [be[x] for x in path], K[path], V[path], Q[path])
                    np.testing.assert_allclose(st[r, l, h], states[-1], rtol=1e-12, atol=1e-13)


def _batch_conv_arrays(wl, rng):
    return dict(x=rng.standard_normal((wl.n_layers, wl.total_rows, wl.channels)).astype(np.float32),
                hist=rng.standard_normal((wl.n_req, wl.n_layers, 3, wl.channels)).astype(np.float32),
                w=rng.uniform(-0.5, 0.5, (wl.n_layers, wl.channels, 4)).astype(np.float32))


def pin_conv_batch_layout():
    """Tree conv over the padded batch: each node's output at its physical row equals
    numpy.convolve over its own request's history followed by its ancestry's x rows;
    pad rows stay unwritten."""
    rng = np.random.default_rng(53)
    wl = _batch_wl(rng)
    wl.arrays = _batch_conv_arrays(wl, rng)
    bias = rng.standard_normal((wl.n_layers, wl.channels)).astype(np.float32)
    y = oracle.conv_all(wl, bias=bias, act=0)
    rows = _hand_rows(wl.parents, wl.n_rows)
    written = np.zeros((wl.n_layers, wl.total_rows), bool)
    x, hist, w = wl.arrays["x"], wl.arrays["hist"], wl.arrays["w"]
    for r in (0, 2):
        par = wl.parents[r]
        for i, rw in enumerate(rows[r]):
            anc = []
            n_ = i
            while n_ != -1:
                anc.insert(0, n_)
                n_ = int(par[n_])
            for l in range(wl.n_layers):
                for c in range(wl.channels):
                    seq = np.concatenate([hist[r, l, :, c], x[l, [rows[r][m] for m in anc], c]]).astype(np.float64)
                    full = np.convolve(seq, w[l, c].astype(np.float64)[::-1], mode="full")
                    np.testing.assert_allclose(y[l, rw, c], full[len(seq) - 1] + bias[l, c],
                                               rtol=1e-13, atol=1e-14)
                written[l, rw] = True
    assert np.all(np.isnan(y[~written]))


def pin_conv_hist_publish_batch_layout():
    """History publication over the padded batch: request r's new history is the last
    three of (its own old history, the x rows of its own path); a request with an empty
    or invalid path keeps its history."""
    rng = np.random.default_rng(54)
    wl = _batch_wl(rng)
    wl.arrays = _batch_conv_arrays(wl, rng)
    rows = _hand_rows(wl.parents, wl.n_rows)
    x, hist = wl.arrays["x"], wl.arrays["hist"]
    for paths in (([0, 2], [], [0, 1, 3, 6]), ([0], [], [0, 2, 5]), ([], [], [0])):
        po = np.full((3, 6), -1, np.int32)
        pl = np.array([len(p) for p in paths], np.int32)
        for r, p in enumerate(paths):
            po[r, :len(p)] = p
        out = oracle.conv_hist_publish(wl, po, pl)
        for r, p in enumerate(paths):
            for l in range(wl.n_layers):
                seq = list(hist[r, l]) + [x[l, rows[r][m]] for m in p]
                assert np.array_equal(out[r, l], np.array(seq[-3:], np.float64)), (r, l, p)


# --------------------------------------------------------------------------- convolution

def _conv_wl(par, C=5, n_layers=1):
    wl = make_wl([par], d_k=1, d_v=1, channels=C, n_layers=n_layers)
    rng = np.random.default_rng(41)
    wl.arrays = dict(x=rng.standard_normal((n_layers, wl.total_rows, C)).astype(np.float32),
                     hist=rng.standard_normal((1, n_layers, 3, C)).astype(np.float32),
                     w=rng.uniform(-0.5, 0.5, (n_layers, C, 4)).astype(np.float32))
    return wl


def pin_conv_identity_tap():
    wl = _conv_wl(trees.FIG1_PARENT)
    wl.arrays["w"][:] = np.array([0, 0, 0, 1], np.float32)
    y = oracle.conv_all(wl, act=0)
    rows = _rows(wl, 0)
    for i in range(7):
        assert np.array_equal(y[0, rows[i]], wl.arrays["x"][0, rows[i]].astype(np.float64))


def pin_conv_oldest_tap_indexing():
    """Tap 0 sees the third ancestor, or committed history entry `depth` when shallower."""
    wl = _conv_wl(trees.FIG1_PARENT)
    wl.arrays["w"][:] = np.array([1, 0, 0, 0], np.float32)
    y = oracle.conv_all(wl, act=0)
    rows = _rows(wl, 0)
    d = trees.depths(trees.FIG1_PARENT)
    for i in range(7):
        if d[i] >= 3:
            want = wl.arrays["x"][0, rows[oracle.plan.ancestry(trees.FIG1_PARENT, i)[-4]]]
        else:
            want = wl.arrays["hist"][0, 0, d[i]]
        assert np.array_equal(y[0, rows[i]], want.astype(np.float64))


def pin_conv_chain_equals_numpy_convolve():
    n = 9
    wl = _conv_wl(trees.chain(n), C=3, n_layers=2)
    bias = np.random.default_rng(42).standard_normal((2, 3)).astype(np.float32)
    y = oracle.conv_all(wl, act=0, bias=bias)
    rows = _rows(wl, 0)
    for l in range(2):
        for c in range(3):
            seq = np.concatenate([wl.arrays["hist"][0, l, :, c],
                                  wl.arrays["x"][l, rows, c]]).astype(np.float64)
            taps = wl.arrays["w"][l, c].astype(np.float64)
            full = np.convolve(seq, taps[::-1], mode="full")[3:3 + n] + bias[l, c]
            np.testing.assert_allclose(y[l, rows, c], full, rtol=1e-13, atol=1e-14)


def pin_conv_silu():
    wl = _conv_wl(trees.chain(3), C=4)
    y0 = oracle.conv_all(wl, act=0)
    y1 = oracle.conv_all(wl, act=1)
    rows = _rows(wl, 0)
    z = y0[0, rows]
    np.testing.assert_allclose(y1[0, rows], z * 0.5 * (1 + np.tanh(z / 2)), rtol=1e-13, atol=1e-15)


def pin_conv_hist_publish():
    wl = _conv_wl(trees.FIG1_PARENT, C=3)
    rows = _rows(wl, 0)
    for acc, L in ((-1, 0), (0, 1), (1, 2), (4, 3), (6, 4)):
        path, plen = oracle.plan.accepted_path(trees.FIG1_PARENT, acc, 4)
        out = oracle.conv_hist_publish(wl, np.array([path]), np.array([plen]))
        seq = list(wl.arrays["hist"][0, 0]) + [wl.arrays["x"][0, rows[x]] for x in path[:plen]]
        assert plen == L
        assert np.array_equal(out[0, 0], np.array(seq[-3:], np.float64))


# --------------------------------------------------------------------------- operand preparation

def _prep_params(rng, wl, eps):
    a_log = (0.5 * rng.standard_normal((wl.n_layers, wl.h_v))).astype(np.float32)
    dt_bias = rng.standard_normal((wl.n_layers, wl.h_v)).astype(np.float32)
    return oracle.Prep(oracle.PREP_QK_NORM | oracle.PREP_RAW_GATES, eps, a_log, dt_bias)


def _prepared_operands(wl, a, r, l, h, prep):
    """Sec. IV-B preparation written out with numpy: x / sqrt(|x|^2 + eps) for q and k,
    alpha = exp(-exp(A_log) log(1 + e^(a + dt_bias))), beta = 1 / (1 + e^-b)."""
    rows = _rows(wl, r)
    hk = h // (wl.h_v // wl.h_k)
    n = len(wl.parents[r])
    K = np.stack([a["k"][l, rows[i], hk].astype(np.float64) for i in range(n)])
    Q = np.stack([a["q"][l, rows[i], hk].astype(np.float64) for i in range(n)])
    V = np.stack([a["v"][l, rows[i], h].astype(np.float64) for i in range(n)])
    if prep.flags & oracle.PREP_QK_NORM:
        K = K / np.sqrt((K * K).sum(1, keepdims=True) + prep.eps)
        Q = Q / np.sqrt((Q * Q).sum(1, keepdims=True) + prep.eps)
    graw = np.array([float(a["g"][l, rows[i], h]) for i in range(n)])
    braw = np.array([float(a["beta"][l, rows[i], h]) for i in range(n)])
    x = graw + float(prep.dt_bias[l, h])
    al = np.exp(-np.exp(np.float64(prep.a_log[l, h])) * np.logaddexp(0.0, x))
    be = 1.0 / (1.0 + np.exp(-braw))
    return list(al), list(be), K, Q, V


def pin_prep_half_gates():
    """a = -dt_bias, A_log = 0 and b = 0 give alpha = exp(-log 2) = 1/2 and beta = 1/2:
    the prepared run equals the run with alpha = beta = 1/2 given directly."""
    rng = np.random.default_rng(61)
    wl = make_wl([trees.FIG1_PARENT], d_k=4, d_v=3, h_k=1, h_v=2, n_layers=2)
    a = random_arrays(wl, rng)
    wl.arrays = a
    dt = rng.standard_normal((2, 2)).astype(np.float32)
    prep = oracle.Prep(oracle.PREP_RAW_GATES, 0.0, np.zeros((2, 2), np.float32), dt)
    raw = dict(a)
    raw["g"] = np.broadcast_to(-dt[:, None, :], a["g"].shape).astype(np.float32).copy()
    raw["beta"] = np.zeros_like(a["beta"])
    half = dict(a)
    half["g"] = np.full_like(a["g"], 0.5)
    half["beta"] = np.full_like(a["beta"], 0.5)
    for (l, h) in [(0, 0), (1, 1)]:
        o1, s1 = oracle.verify_nodes(wl, 0, l, h, list(range(7)), arrays=raw, prep=prep, want_state=True)
        o2, s2 = oracle.verify_nodes(wl, 0, l, h, list(range(7)), arrays=half, gate_is_alpha=True,
                                     want_state=True)
        np.testing.assert_allclose(o1, o2, rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(s1, s2, rtol=1e-14, atol=1e-15)


def pin_prep_chain_equals_matrix_scan():
    """Normalised q, k and raw gates on a chain: the matrix-form scan of the operands
    prepared with numpy (eps = 0.3, so its placement matters)."""
    rng = np.random.default_rng(62)
    wl = make_wl([trees.chain(9)], d_k=7, d_v=5, h_k=1, h_v=2, n_layers=2)
    a = random_arrays(wl, rng)
    a["k"] = (a["k"] * rng.uniform(0.2, 3.0, size=a["k"].shape[:-1] + (1,))).astype(np.float32)
    wl.arrays = a
    prep = _prep_params(rng, wl, 0.3)
    for (l, h) in [(0, 1), (1, 0)]:
        al, be, K, Q, V = _prepared_operands(wl, a, 0, l, h, prep)
        want_o, want_s = chain_matrix_form(a["state0"][0, l, h], al, be, K, V, Q)
        o, st = oracle.verify_nodes(wl, 0, l, h, list(range(9)), want_state=True, prep=prep)
        np.testing.assert_allclose(o, want_o, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(st, want_s, rtol=1e-12, atol=1e-13)


def pin_prep_tree_equals_wy_closed_form():
    rng = np.random.default_rng(63)
    par = trees.random_tree(rng, 18, 6, trees.bmax_uniform(3))
    wl = make_wl([par, trees.FIG1_PARENT], d_k=6, d_v=5, h_k=2, h_v=4, n_layers=2, n_rows=[20, 8])
    a = random_arrays(wl, rng)
    a["q"] = (3.0 * a["q"]).astype(np.float32)
    wl.arrays = a
    prep = _prep_params(rng, wl, 1e-6)
    for (r, l, h) in [(0, 0, 1), (0, 1, 2), (1, 1, 3)]:
        al, be, K, Q, V = _prepared_operands(wl, a, r, l, h, prep)
        want = tree_wy_form(wl.parents[r], a["state0"][r, l, h], al, be, K, V, Q)
        o = oracle.verify_nodes(wl, r, l, h, list(range(len(wl.parents[r]))), prep=prep)
        np.testing.assert_allclose(o, want, rtol=1e-11, atol=1e-12)


def pin_prep_qk_scale_invariance():
    """With eps = 0 the normalisation removes any positive scale of a query or key row."""
    rng = np.random.default_rng(64)
    par = trees.random_tree(rng, 12, 5, trees.bmax_uniform(3))
    wl = make_wl([par], d_k=5, d_v=4, h_k=1, h_v=2)
    a = random_arrays(wl, rng)
    wl.arrays = a
    prep = oracle.Prep(oracle.PREP_QK_NORM, 0.0)
    b = dict(a)
    b["k"] = (a["k"] * rng.uniform(0.1, 10.0, size=a["k"].shape[:-1] + (1,))).astype(np.float64)
    b["q"] = (a["q"] * rng.uniform(0.1, 10.0, size=a["q"].shape[:-1] + (1,))).astype(np.float64)
    # the scaled rows are rounded to fp32 by the oracle's loader; compare at that precision
    for h in range(2):
        o1 = oracle.verify_nodes(wl, 0, 0, h, list(range(12)), prep=prep)
        o2 = oracle.verify_nodes(wl, 0, 0, h, list(range(12)), arrays=b, prep=prep)
        np.testing.assert_allclose(o2, o1, rtol=2e-6, atol=2e-7)
        o3 = oracle.verify_nodes(wl, 0, 0, h, list(range(12)), arrays=b)
        assert not np.allclose(o3, o1, rtol=1e-3)


def pin_prep_commit_equals_node_state():
    """The replay of a path with prepared operands publishes the verified state of its last node."""
    rng = np.random.default_rng(65)
    par = trees.random_tree(rng, 14, 6, trees.bmax_uniform(3))
    wl = make_wl([par], d_k=6, d_v=4, h_k=1, h_v=2, max_path=14)
    a = random_arrays(wl, rng)
    wl.arrays = a
    prep = _prep_params(rng, wl, 1e-3)
    node = int(np.argmax(trees.depths(par)))
    _, st = oracle.verify_nodes(wl, 0, 0, 1, [node], want_state=True, prep=prep)
    pub, _, _ = oracle.commit(wl, accepted=np.array([node], np.int32), prep=prep)
    np.testing.assert_array_equal(pub[0, 0, 1], st[0])


# --------------------------------------------------------------------------- tree attention

def _attn_case(rng, parents, n_ctx, h_q, h_kv, d, n_rows=None, scale_q=1.0):
    n_rows = [len(p) for p in parents] if n_rows is None else n_rows
    row_off = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    total = int(row_off[-1])
    ctx_off = np.concatenate([[0], np.cumsum(n_ctx)]).astype(np.int32)
    a = dict(q=(scale_q * rng.standard_normal((total, h_q, d))).astype(np.float32),
             k_tree=rng.standard_normal((total, h_kv, d)).astype(np.float32),
             v_tree=rng.standard_normal((total, h_kv, d)).astype(np.float32),
             k_ctx=rng.standard_normal((int(ctx_off[-1]), h_kv, d)).astype(np.float32),
             v_ctx=rng.standard_normal((int(ctx_off[-1]), h_kv, d)).astype(np.float32))
    return row_off, total, ctx_off, a


def _attn(parents, row_off, total, ctx_off, a, h_q, h_kv, d, scale=None):
    return oracle.tree_attention(parents, row_off, total, ctx_off, a["q"], a["k_ctx"], a["v_ctx"],
                                 a["k_tree"], a["v_tree"], h_q=h_q, h_kv=h_kv, d=d, op_dtype=0,
                                 scale=scale)


def pin_attention_root_only():
    """A root with no context sees only itself: o = v_root, lse = scale q.k."""
    rng = np.random.default_rng(81)
    row_off, total, ctx_off, a = _attn_case(rng, [np.array([-1], np.int32)], [0], 2, 1, 8)
    o, lse = _attn([np.array([-1], np.int32)], row_off, total, ctx_off, a, 2, 1, 8, scale=0.7)
    for h in range(2):
        np.testing.assert_allclose(o[0, h], a["v_tree"][0, 0], rtol=1e-15)
        want = 0.7 * float(a["q"][0, h].astype(np.float64) @ a["k_tree"][0, 0].astype(np.float64))
        np.testing.assert_allclose(lse[0, h], want, rtol=1e-14)


def pin_attention_uniform_scores():
    """q = 0: every visible key weighs the same, so o is the mean of the visible values
    (the context and the node's own path) and lse = log(number of visible keys)."""
    rng = np.random.default_rng(82)
    par = trees.FIG1_PARENT
    row_off, total, ctx_off, a = _attn_case(rng, [par], [5], 2, 2, 4, scale_q=0.0)
    rows = oracle.plan.rows_of(par, 0)
    o, lse = _attn([par], row_off, total, ctx_off, a, 2, 2, 4)
    for i in range(len(par)):
        path = oracle.plan.ancestry(par, i)
        for h in range(2):
            vis = [a["v_ctx"][t, h] for t in range(5)] + [a["v_tree"][rows[x], h] for x in path]
            np.testing.assert_allclose(o[rows[i], h], np.mean(np.array(vis, np.float64), 0), rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(lse[rows[i], h], np.log(5 + len(path)), rtol=1e-14)


def pin_attention_dense_masked_softmax():
    """Against a dense formulation: visibility from boolean reachability powers of the
    parent matrix, scores by matrix product, masked softmax; two requests, grouped heads."""
    rng = np.random.default_rng(83)
    parents = [trees.random_tree(rng, 13, 5, trees.bmax_uniform(3)), trees.FIG1_PARENT]
    n_ctx = [6, 3]
    h_q, h_kv, d = 4, 2, 8
    row_off, total, ctx_off, a = _attn_case(rng, parents, n_ctx, h_q, h_kv, d, n_rows=[15, 7])
    o, lse = _attn(parents, row_off, total, ctx_off, a, h_q, h_kv, d, scale=0.35)
    for r, par in enumerate(parents):
        n = len(par)
        A = np.zeros((n, n), bool)
        for i, p_ in enumerate(par):
            if p_ >= 0:
                A[i, p_] = True
        vis = np.eye(n, dtype=bool)
        step = np.eye(n, dtype=bool)
        for _ in range(n):
            step = (step.astype(int) @ A.astype(int)) > 0
            vis |= step
        rows = np.array(oracle.plan.rows_of(par, int(row_off[r])))
        ctx = slice(int(ctx_off[r]), int(ctx_off[r + 1]))
        for h in range(h_q):
            g = h // (h_q // h_kv)
            Q = a["q"][rows, h].astype(np.float64)
            K = np.concatenate([a["k_ctx"][ctx, g], a["k_tree"][rows, g]]).astype(np.float64)
            V = np.concatenate([a["v_ctx"][ctx, g], a["v_tree"][rows, g]]).astype(np.float64)
            S = 0.35 * Q @ K.T
            mask = np.concatenate([np.ones((n, n_ctx[r]), bool), vis], axis=1)
            S = np.where(mask, S, -np.inf)
            m = S.max(1, keepdims=True)
            P = np.exp(S - m)
            want_l = np.log(P.sum(1)) + m[:, 0]
            want_o = (P / P.sum(1, keepdims=True)) @ V
            np.testing.assert_allclose(o[rows, h], want_o, rtol=1e-11, atol=1e-13)
            np.testing.assert_allclose(lse[rows, h], want_l, rtol=1e-12)


def pin_attention_context_order_and_padding():
    """Permuting the context tokens changes nothing; NaN in pad rows of the tree keys
    and values is never read."""
    rng = np.random.default_rng(84)
    par = trees.random_tree(rng, 10, 4, trees.bmax_uniform(3))
    row_off, total, ctx_off, a = _attn_case(rng, [par], [9], 2, 1, 6, n_rows=[12])
    o1, l1 = _attn([par], row_off, total, ctx_off, a, 2, 1, 6)
    perm = rng.permutation(9)
    b = dict(a)
    b["k_ctx"], b["v_ctx"] = a["k_ctx"][perm], a["v_ctx"][perm]
    rows = oracle.plan.rows_of(par, 0)
    pad = [x for x in range(12) if x not in rows]
    for key in ("k_tree", "v_tree", "q"):
        b[key] = b[key].copy()
        b[key][pad] = np.nan
    o2, l2 = _attn([par], row_off, total, ctx_off, b, 2, 1, 6)
    np.testing.assert_allclose(o2[rows], o1[rows], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l2[rows], l1[rows], rtol=1e-13)
    assert np.all(np.isfinite(o2[rows]))


def _tied_logits(rng, rows, vocab, levels):
    """Logits drawn from a few levels, so that ties are common; some -inf entries."""
    x = rng.integers(0, levels, size=(rows, vocab)).astype(np.float32) * 0.25 - 1.0
    x[rng.random((rows, vocab)) < 0.05] = -np.inf
    return x


def pin_select_spine_is_numpy_argmax():
    """The spine is numpy's argmax (first occurrence of the maximum; a NaN, if any, is
    the maximum), also with ties, -inf, -0 against +0, and NaN entries."""
    rng = np.random.default_rng(91)
    x = _tied_logits(rng, 40, 300, 6)
    x[3, 17] = np.nan
    x[3, 5] = np.nan
    x[4] = -np.inf
    x[5] = 0.0
    x[5, 2] = -0.0
    x[6, :] = -0.0
    x[6, 9] = 0.0
    spine, _ = oracle.draft_select(x, k=3, op_dtype=0)
    assert spine.tolist() == np.argmax(x.astype(np.float64), axis=1).tolist()


def pin_select_distinct_is_argsort():
    """With distinct logits the candidates are numpy's descending argsort, for both tie
    conventions, and the spine is the first candidate."""
    rng = np.random.default_rng(92)
    x = np.stack([rng.permutation(500).astype(np.float32) - 250.0 for _ in range(12)])
    for ties in (0, 1):
        spine, cand = oracle.draft_select(x, k=5, op_dtype=0, ties=ties)
        assert cand.tolist() == np.argsort(-x, axis=1)[:, :5].tolist()
        assert spine.tolist() == cand[:, 0].tolist()


def pin_select_brute_force():
    """Tiny rows with heavy ties, NaN and infinities: the candidates are the first k of
    all indices sorted by (NaN first, then value descending, then index in the tie
    direction)."""
    rng = np.random.default_rng(93)
    vals = np.array([np.nan, np.inf, -np.inf, 1.5, 1.5, -0.0, 0.0, 2.0], np.float32)
    for case in range(60):
        vocab = int(rng.integers(3, 12))
        row = vals[rng.integers(0, len(vals), size=vocab)][None, :]
        k = int(rng.integers(1, vocab + 1))
        for ties in (0, 1):
            spine, cand = oracle.draft_select(row, k=k, op_dtype=0, ties=ties)

            def key(i):
                v = float(row[0, i])
                tie = -i if ties == 0 else i
                return (1, 0.0, tie) if np.isnan(v) else (0, v, tie)
            want = sorted(range(vocab), key=key, reverse=True)[:k]
            assert cand[0].tolist() == want, (case, ties, row, cand)
            top = [i for i in range(vocab) if key(i)[:2] == key(want[0])[:2]]
            assert spine[0] == min(top)


def pin_select_all_equal():
    """A row of equal logits: spine 0; candidates 0, 1, 2 (ties ascending) or the last
    three indices, last first (descending)."""
    x = np.full((2, 1000), 0.5, np.float32)
    s0, c0 = oracle.draft_select(x, k=3, op_dtype=0, ties=0)
    s1, c1 = oracle.draft_select(x, k=3, op_dtype=0, ties=1)
    assert s0.tolist() == [0, 0] and s1.tolist() == [0, 0]
    assert c0.tolist() == [[0, 1, 2]] * 2 and c1.tolist() == [[999, 998, 997]] * 2


def pin_select_tie_conventions_differ():
    """The maximum at indices 3 and 7: the spine is 3 under either tie convention,
    while the first candidate is 3 (ascending) or 7 (descending); the spine token is
    duplicated among the candidates."""
    x = np.array([[0.1, 0.2, 0.0, 0.9, 0.5, 0.9 - 0.4, 0.3, 0.9, 0.7]], np.float32)
    s0, c0 = oracle.draft_select(x, k=3, op_dtype=0, ties=0)
    s1, c1 = oracle.draft_select(x, k=3, op_dtype=0, ties=1)
    assert s0[0] == 3 and s1[0] == 3
    assert c0[0].tolist() == [3, 7, 8] and c1[0].tolist() == [7, 3, 8]


def pin_select_bf16_equals_decoded_f32():
    """bf16 bit patterns give the same selection as their exact fp32 values."""
    rng = np.random.default_rng(94)
    bits = ops.to_bf16_bits((rng.standard_normal((8, 777)) * 3).astype(np.float32))
    f = ops.bf16_bits_to_f32(bits)
    for ties in (0, 1):
        a = oracle.draft_select(bits, k=4, op_dtype=1, ties=ties)
        b = oracle.draft_select(f, k=4, op_dtype=0, ties=ties)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_") and callable(v)]
