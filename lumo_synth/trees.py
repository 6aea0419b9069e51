"""Seeded synthetic speculative-tree topologies.

Only topology is produced here (parent arrays with parent[i] < i); nothing of the
gated delta rule's arithmetic lives in this module. Both the GPU path's tests and the
CPU oracle consume the arrays generated here.

Shapes follow the paper's workloads: a candidate tree rooted at the pending token
(Sec. III-C, Fig. 1), the evaluated geometry of 27 drafts plus the root padded to
32 rows with maximum draft depth eleven (Sec. VI), and the random trees of the
benchmark configurations (64-node depth-8 trees with branching 1-4, 256-node
depth-16 trees that are wide near the root, chains of 16 plus 128-node trees).
"""
from __future__ import annotations

import numpy as np

# Fig. 1 tree: m -> {a, b}, a -> {c, d}, b -> e, c -> f with ids m,a,b,c,d,e,f = 0..6.
FIG1_PARENT = np.array([-1, 0, 0, 1, 1, 2, 3], dtype=np.int32)
FIG1_NAMES = ("m", "a", "b", "c", "d", "e", "f")


def chain(n: int) -> np.ndarray:
    """Linear chain of n nodes (plain multi-token proposal)."""
    p = np.arange(-1, n - 1, dtype=np.int32)
    return p


def random_tree(rng: np.random.Generator, n_nodes: int, max_depth: int, bmax) -> np.ndarray:
    """Random-frontier growth of an n_nodes tree.

    max_depth counts nodes on a root-to-leaf path (depth index <= max_depth - 1).
    bmax(depth) gives the largest branching factor for a node at that depth.
    A uniformly random frontier node is expanded with b ~ U{1..bmax(depth)}
    children, ids assigned in creation order so that parent[i] < i. When the
    frontier empties before n_nodes are placed, a random non-capped node is
    re-opened.
    """
    if n_nodes < 1:
        raise ValueError("n_nodes must be >= 1")
    if max_depth < 1:
        raise ValueError("max_depth must be >= 1")
    if max_depth == 1 and n_nodes > 1:
        raise ValueError("a depth-1 tree holds one node")
    parent = [-1]
    depth = [0]
    frontier = [0] if max_depth > 1 else []
    while len(parent) < n_nodes:
        if not frontier:
            cands = [i for i in range(len(parent)) if depth[i] < max_depth - 1]
            frontier.append(cands[int(rng.integers(len(cands)))])
        p = frontier.pop(int(rng.integers(len(frontier))))
        b = int(rng.integers(1, int(bmax(depth[p])) + 1))
        for _ in range(min(b, n_nodes - len(parent))):
            parent.append(p)
            depth.append(depth[p] + 1)
            if depth[-1] < max_depth - 1:
                frontier.append(len(parent) - 1)
    return np.asarray(parent, dtype=np.int32)


def bmax_uniform(b: int):
    return lambda d: b


def bmax_root_skewed(d: int) -> int:
    """Wide near the root, narrowing with depth: 6,6,6,5,5,5,4,... down to 1."""
    return max(1, 6 - d // 3)


def paper_geometry_tree() -> np.ndarray:
    """A 28-node tree with the evaluated draft geometry (Sec. VI).

    Root (pending token) plus a five-deep multi-token-prediction head giving 15
    candidates (a principal chain of 5 plus two runner-up siblings at each depth),
    a six-token principal suffix tail (max draft depth 11) and rescue branches of
    four and two tokens hanging off the principal chain. The exact attachment
    points of the rescue branches are not given in the paper; they are placed on
    the principal chain at depths 2 and 4 here.
    """
    parent = [-1]
    spine = [0]
    # MTP head: principal chain of 5 with two runner-up siblings at each depth.
    for _depth in range(5):
        p = spine[-1]
        parent.append(p)
        principal = len(parent) - 1
        parent.append(p)
        parent.append(p)
        spine.append(principal)
    # six-token principal tail continuing the MTP principal chain
    for _ in range(6):
        parent.append(spine[-1])
        spine.append(len(parent) - 1)
    # rescue branches of four and two tokens
    for attach, length in ((spine[2], 4), (spine[4], 2)):
        p = attach
        for _ in range(length):
            parent.append(p)
            p = len(parent) - 1
    arr = np.asarray(parent, dtype=np.int32)
    assert arr.shape[0] == 28
    return arr


def depths(parent: np.ndarray) -> np.ndarray:
    """Depth of each node (root depth 0); parent[i] < i is required."""
    d = np.zeros(parent.shape[0], dtype=np.int32)
    for i in range(1, parent.shape[0]):
        d[i] = d[parent[i]] + 1
    return d
