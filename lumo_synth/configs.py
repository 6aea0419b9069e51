"""Workload configurations for tree GDN verification (seeded, synthetic).

  tiny       1 request, 1 head, d=16, fp32 operands, the Fig. 1 tree (7 nodes)
  layer1     1 request, one GDN layer, 16 key heads / 32 value heads, d=128, bf16
             operands, one 64-node random tree (depth <= 8, branching 1-4)
  batched    8 requests x 48 stacked GDN layers of the layer1 shape, each request
             with its own 64-node tree and initial state (the headline workload)
  widedeep   32 requests x 256-node trees, depth <= 16, branching wide near the root
  chainmix   64 requests: 32 chains of 16 draft nodes + 32 trees of 128 nodes
             (branching 1-4, depth <= 16); accepted lengths 0..16
  paper28    the evaluated draft geometry of Sec. VI: 28 nodes padded to 32 rows,
             depth 12 (root + 11 drafts), 48 layers x 48 value heads is the paper's
             count; one layer with 16/32 heads is used here

Every config is generated from numpy's PCG64 seeded with the config index.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import operands as ops
from . import trees


@dataclass
class Workload:
    name: str
    n_req: int
    n_layers: int
    h_k: int
    h_v: int
    d_k: int
    d_v: int
    op_dtype: int
    parents: list            # per request: int32 parent array (request-local ids)
    n_rows: np.ndarray       # per request: physical rows (>= nodes)
    accepted: np.ndarray     # per request: accepted node (-1 = none)
    max_path: int            # fixed commit shape (max accepted path length)
    channels: int
    arrays: dict = field(default_factory=dict)

    @property
    def node_off(self) -> np.ndarray:
        n = np.array([len(p) for p in self.parents], dtype=np.int32)
        return np.concatenate([[0], np.cumsum(n)]).astype(np.int32)

    @property
    def row_off(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.n_rows)]).astype(np.int32)

    @property
    def total_nodes(self) -> int:
        return int(sum(len(p) for p in self.parents))

    @property
    def total_rows(self) -> int:
        return int(self.n_rows.sum())

    @property
    def parent_flat(self) -> np.ndarray:
        return np.concatenate(self.parents).astype(np.int32)

    @property
    def head_node_updates(self) -> int:
        """Tree nodes x layers x value heads (each node counted once)."""
        return self.total_nodes * self.n_layers * self.h_v


def _pick_accepted(rng, parent, lo, hi):
    """Accepted length L ~ U{lo..hi} clipped to the deepest path; node uniform at depth L-1."""
    d = trees.depths(parent)
    L = int(rng.integers(lo, hi + 1))
    L = min(L, int(d.max()) + 1)
    if L <= 0:
        return -1
    cands = np.nonzero(d == L - 1)[0]
    return int(cands[int(rng.integers(len(cands)))])


CONFIG_NAMES = ("tiny", "layer1", "batched", "widedeep", "chainmix", "paper28")


def _shape(name):
    if name == "tiny":
        return dict(n_req=1, n_layers=1, h_k=1, h_v=1, d_k=16, d_v=16, op_dtype=ops.F32)
    if name == "batched":
        return dict(n_req=8, n_layers=48, h_k=16, h_v=32, d_k=128, d_v=128, op_dtype=ops.BF16)
    if name == "widedeep":
        return dict(n_req=32, n_layers=1, h_k=16, h_v=32, d_k=128, d_v=128, op_dtype=ops.BF16)
    if name == "chainmix":
        return dict(n_req=64, n_layers=1, h_k=16, h_v=32, d_k=128, d_v=128, op_dtype=ops.BF16)
    return dict(n_req=1, n_layers=1, h_k=16, h_v=32, d_k=128, d_v=128, op_dtype=ops.BF16)


def topology(name: str, seed: int | None = None, **over):
    """Trees, rows, accepted nodes and commit shape of a config (no operand arrays)."""
    idx = CONFIG_NAMES.index(name)
    rng = np.random.default_rng(idx if seed is None else seed)
    shp = _shape(name)
    shp.update({k: v for k, v in over.items() if k in shp})
    n_req = shp["n_req"]
    if name == "tiny":
        parents = [trees.FIG1_PARENT.copy()]
        accepted = np.array([4], dtype=np.int32)  # node d: path m, a, d
        max_path = 4
    elif name in ("layer1", "batched"):
        parents = [trees.random_tree(rng, 64, 8, trees.bmax_uniform(4)) for _ in range(n_req)]
        accepted = np.array([_pick_accepted(rng, p, 1, 8) for p in parents], dtype=np.int32)
        max_path = 8
    elif name == "widedeep":
        parents = [trees.random_tree(rng, 256, 16, trees.bmax_root_skewed) for _ in range(n_req)]
        accepted = np.array([_pick_accepted(rng, p, 1, 16) for p in parents], dtype=np.int32)
        max_path = 16
    elif name == "chainmix":
        half = n_req // 2
        parents = [trees.chain(16) for _ in range(half)]
        parents += [trees.random_tree(rng, 128, 16, trees.bmax_uniform(4))
                    for _ in range(n_req - half)]
        accepted = np.array([_pick_accepted(rng, p, 0, 16) for p in parents], dtype=np.int32)
        max_path = 16
    elif name == "paper28":
        parents = [trees.paper_geometry_tree() for _ in range(n_req)]
        accepted = np.array([_pick_accepted(rng, p, 1, 12) for p in parents], dtype=np.int32)
        max_path = 12
    else:
        raise KeyError(name)
    n_rows = np.array([32 if name == "paper28" else len(p) for p in parents], dtype=np.int32)
    channels = 2 * shp["h_k"] * shp["d_k"] + shp["h_v"] * shp["d_v"]
    return Workload(name=name, parents=parents, n_rows=n_rows, accepted=accepted,
                    max_path=max_path, channels=channels, **shp), rng


def build(name: str, seed: int | None = None, with_conv: bool = True, **over) -> Workload:
    """Topology plus all operand arrays of a config."""
    wl, _ = topology(name, seed, **over)
    s = CONFIG_NAMES.index(name) if seed is None else seed
    wl.arrays.update(ops.make_gdn_operands(
        s, n_req=wl.n_req, n_layers=wl.n_layers, total_rows=wl.total_rows, h_k=wl.h_k,
        h_v=wl.h_v, d_k=wl.d_k, d_v=wl.d_v, op_dtype=wl.op_dtype))
    if with_conv:
        wl.arrays.update(ops.make_conv_operands(
            s, n_req=wl.n_req, n_layers=wl.n_layers, total_rows=wl.total_rows,
            channels=wl.channels, op_dtype=wl.op_dtype))
    return wl
