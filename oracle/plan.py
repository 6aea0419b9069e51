"""Plain derivation of the tree descriptor products (integer, bit-exact).

TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the benchmark's
CPU-baseline leg, never by the GPU library.

Each function restates what the paper specifies for the shared tree descriptor:
  - parent indices with the ancestry contract (Sec. III-A/B): node i consumes the
    state of its root-to-parent path; depth is the distance from the root.
  - root-to-leaf paths, leaves taken in increasing logical id (the unit the
    path-parallel verifier scans, Sec. IV-A).
  - the principal spine and the physical slot map (Sec. III-C, Sec. V-B): the
    spine is placed first and contiguously, the remaining nodes keep logical order.
    The spine is read as the first-child chain from the root, children ordered by
    logical id.
  - convolution gather sources (Sec. V-C): window of the last four entries of the
    committed history followed by the node's ancestry.
  - the accepted path (Sec. V-A): root-first node list of the accepted node, padded
    to a fixed length; an accepted node of -1 gives the empty path.
"""
from __future__ import annotations

import numpy as np


def validate(parent) -> None:
    parent = [int(p) for p in parent]
    if not parent:
        raise ValueError("empty tree")
    if parent[0] != -1:
        raise ValueError("node 0 must be the root")
    for i, p in enumerate(parent[1:], start=1):
        if not (0 <= p < i):
            raise ValueError(f"node {i}: parent {p} must satisfy 0 <= parent < id")


def depth(parent) -> list:
    out = []
    for i in range(len(parent)):
        d, x = 0, int(parent[i])
        while x != -1:
            d += 1
            x = int(parent[x])
        out.append(d)
    return out


def children(parent) -> list:
    ch = [[] for _ in parent]
    for i in range(len(parent)):
        if parent[i] >= 0:
            ch[int(parent[i])].append(i)
    for c in ch:
        c.sort()
    return ch


def ancestry(parent, i) -> list:
    """Root-first list of nodes from the root to i inclusive."""
    out = []
    x = int(i)
    while x != -1:
        out.append(x)
        x = int(parent[x])
    return out[::-1]


def leaves(parent) -> list:
    ch = children(parent)
    return [i for i in range(len(parent)) if not ch[i]]


def paths(parent) -> list:
    return [ancestry(parent, leaf) for leaf in leaves(parent)]


def spine(parent) -> list:
    if len(parent) == 0:  # a request without nodes has an empty spine
        return []
    ch = children(parent)
    s = [0]
    while ch[s[-1]]:
        s.append(ch[s[-1]][0])
    return s


def slot_map(parent) -> list:
    """slot[i] = physical row (request-local) of logical node i."""
    sp = spine(parent)
    on = set(sp)
    order = sp + [i for i in range(len(parent)) if i not in on]
    slot = [0] * len(parent)
    for pos, node in enumerate(order):
        slot[node] = pos
    return slot


def owner_leaf(parent) -> list:
    """Smallest leaf id among the root-to-leaf paths that contain each node."""
    own = [None] * len(parent)
    for leaf in leaves(parent):
        for x in ancestry(parent, leaf):
            if own[x] is None or leaf < own[x]:
                own[x] = leaf
    return own


def conv_sources(parent, row) -> list:
    """Per node, 4 window sources oldest first: absolute row (>= 0) or -1-h for history h."""
    out = []
    for i in range(len(parent)):
        anc = ancestry(parent, i)
        seq = [("h", 0), ("h", 1), ("h", 2)] + [("x", a) for a in anc]
        src = []
        for kind, val in seq[-4:]:
            src.append(int(row[val]) if kind == "x" else -1 - val)
        out.append(src)
    return out


def accepted_path(parent, accepted, max_path) -> tuple:
    """(root-first path padded with -1 to max_path, length).

    -1 accepts nothing (length 0). A node outside the tree, or a path longer than
    max_path, names no publishable path: all -1 with length -1."""
    if accepted == -1:
        return [-1] * max_path, 0
    if not 0 <= accepted < len(parent):
        return [-1] * max_path, -1
    p = ancestry(parent, accepted)
    if len(p) > max_path:
        return [-1] * max_path, -1
    return p + [-1] * (max_path - len(p)), len(p)


def rows_of(parent, row_base) -> list:
    """Absolute physical row of every node of one request (row_base + slot)."""
    return [row_base + s for s in slot_map(parent)]


def flat_rows(parents, row_off) -> np.ndarray:
    return np.concatenate([np.asarray(rows_of(p, int(row_off[r])), dtype=np.int32)
                           for r, p in enumerate(parents)]).astype(np.int32)
