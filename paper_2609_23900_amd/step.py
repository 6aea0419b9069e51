"""One speculative verification step on device buffers: conv gather, verify, commit.

A convenience layer over the binding: it owns the device tensors of a batch (operands,
state, outputs, workspace, plan) and calls the C ABI in the order of one serving
iteration (Alg. 1): tree convolution, path verification, then publication of the
accepted path. Marshalling only; all arithmetic runs in the HIP kernels.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (LUMO_BF16, LumoError, TreeDesc, dims, lumo_gdn_commit_graph_create,
               lumo_gdn_commit_prep, lumo_tree_conv_gather, lumo_tree_conv_gather_pending,
               lumo_tree_gdn_verify, lumo_tree_gdn_verify_conv_pending,
               lumo_tree_gdn_verify_pending, lumo_tree_gdn_verify_prep,
               lumo_tree_gdn_workspace_bytes)


def to_device(a: np.ndarray, device="cuda", bf16=False) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(a))
    if bf16:
        t = t.view(torch.bfloat16) if t.dtype == torch.uint16 else t
    return t.to(device)


class GdnTreeStep:
    """Device-resident batch for one verification step.

    arrays: q, k, v, g, beta, state0 (and optionally x, hist, w for the conv step) in the
    boundary layouts; operands as float32 or uint16 bf16 bit patterns.
    """

    def __init__(self, *, n_req, n_layers, h_k, h_v, d_k, d_v, op_dtype, node_off, parent,
                 n_rows, arrays, policy=0, max_path=16, accepted=None, channels=0, act=1,
                 device="cuda", with_node_states=False, keep_state0=True, prep=None):
        self.dims = dims(n_req, n_layers, h_k, h_v, d_k, d_v, op_dtype)
        self.prep = prep  # a Prep (operand preparation inside the kernels) or None
        self.desc = TreeDesc.build(node_off, parent, n_rows, policy, device)
        self.plan = self.desc.plan
        self.max_path = int(max_path)
        self.channels = int(channels)
        self.act = int(act)
        self.device = device
        bf = op_dtype == LUMO_BF16
        self.t = {}
        for key in ("q", "k", "v"):
            self.t[key] = to_device(arrays[key], device, bf)
        for key in ("g", "beta"):
            self.t[key] = to_device(np.asarray(arrays[key], np.float32), device)
        self.state0 = to_device(np.asarray(arrays["state0"], np.float32), device)
        # state is the native running state that commit updates in place
        self.state = self.state0.clone() if keep_state0 else self.state0
        odt = torch.bfloat16 if bf else torch.float32
        rows = self.plan.total_rows
        self.o = torch.zeros((n_layers, rows, h_v, d_v), dtype=odt, device=device)
        self.node_states = (torch.zeros((n_layers, rows, h_v, d_k, d_v), dtype=torch.float32,
                                        device=device) if with_node_states else None)
        wsb = lumo_tree_gdn_workspace_bytes(self.dims, self.plan)
        self.ws = torch.empty((max(wsb // 4, 1),), dtype=torch.float32, device=device) if wsb else None
        acc = np.full((n_req,), -1, np.int32) if accepted is None else np.asarray(accepted, np.int32)
        self.accepted = torch.from_numpy(acc).to(device)
        self.path_out = torch.full((max(n_req, 1), self.max_path), -7, dtype=torch.int32, device=device)
        self.path_len = torch.full((max(n_req, 1),), -7, dtype=torch.int32, device=device)
        self.has_conv = "x" in arrays and channels > 0
        if self.has_conv:
            self.x = to_device(arrays["x"], device, bf)
            self.hist = to_device(arrays["hist"], device, bf)
            self.w = to_device(np.asarray(arrays["w"], np.float32), device)
            self.bias = (to_device(np.asarray(arrays["bias"], np.float32), device)
                         if arrays.get("bias") is not None else None)
            self.y = torch.zeros((n_layers, rows, channels), dtype=odt, device=device)

    # ---------------------------------------------------------------- steps
    def conv(self, stream=None):
        if not self.has_conv:
            raise LumoError(1, "no conv operands")
        lumo_tree_conv_gather(self.dims, self.desc, self.channels, self.x, self.hist, self.w,
                              self.bias, self.act, self.y, stream)

    def conv_pending(self, prev: "GdnTreeStep", stream=None):
        """Publish prev's accepted path (written by prev.commit(defer=True, with_conv=False))
        into the conv history, then the tree conv of this step from it, in one launch."""
        if not self.has_conv:
            raise LumoError(1, "no conv operands")
        lumo_tree_conv_gather_pending(self.dims, self.desc, self.channels, self.x, self.hist, self.w,
                                      self.bias, self.act, self.y, prev.desc, prev.max_path,
                                      prev.path_out, prev.path_len, prev.x if prev.has_conv else None,
                                      stream)

    def verify(self, stream=None, state0=None):
        s0 = self.state if state0 is None else state0
        if self.prep is not None:
            lumo_tree_gdn_verify_prep(self.dims, self.desc, self.prep, self.t["q"], self.t["k"],
                                      self.t["v"], self.t["g"], self.t["beta"], s0, self.o, stream)
            return
        lumo_tree_gdn_verify(self.dims, self.desc, self.t["q"], self.t["k"], self.t["v"],
                             self.t["g"], self.t["beta"], s0, self.o, self.node_states, self.ws, 0,
                             stream)

    def verify_pending(self, prev: "GdnTreeStep", stream=None, state=None):
        """Publish prev's accepted path (written by prev.commit(defer=True)) into the
        state bank and verify this step's tree from it, in one launch. The state bank is
        self.state unless given."""
        lumo_tree_gdn_verify_pending(self.dims, self.desc, self.t["q"], self.t["k"], self.t["v"],
                                     self.t["g"], self.t["beta"],
                                     self.state if state is None else state, self.o, prev.desc,
                                     prev.max_path, prev.path_out, prev.path_len, prev.t["k"],
                                     prev.t["v"], prev.t["g"], prev.t["beta"], stream, self.prep)

    def verify_conv_pending(self, prev: "GdnTreeStep", stream=None, state=None):
        """conv_pending and verify_pending in one pass: the queries, keys and values are
        this step's conv outputs of x (channels q | k | v), never stored; prev's accepted
        path (prev.commit(defer=True, with_conv=False)) is published into the history and
        the state bank first. self.t["q"], ["k"], ["v"] and self.y are not used."""
        if not self.has_conv:
            raise LumoError(1, "no conv operands")
        lumo_tree_gdn_verify_conv_pending(self.dims, self.desc, self.channels, self.x, self.hist, self.w,
                                          self.bias, self.act, self.t["g"], self.t["beta"],
                                          self.state if state is None else state, self.o, prev.desc,
                                          prev.max_path, prev.path_out, prev.path_len, prev.x, prev.t["g"],
                                          prev.t["beta"], stream, self.prep)

    def commit(self, stream=None, with_conv=True, defer=False):
        """Accepted path, conv history (unless with_conv is False: then the next
        conv_pending publishes it) and (unless defer) the replay into self.state."""
        use_conv = with_conv and self.has_conv
        lumo_gdn_commit_prep(self.dims, self.desc, self.prep, self.max_path, self.accepted,
                             self.path_out, self.path_len, self.t["k"], self.t["v"], self.t["g"],
                             self.t["beta"], None if defer else self.state,
                             self.channels if use_conv else 0, self.x if use_conv else None,
                             self.hist if use_conv else None, stream)

    def commit_graph(self, with_conv=True):
        use_conv = with_conv and self.has_conv
        return lumo_gdn_commit_graph_create(
            self.dims, self.desc, self.max_path, self.accepted, self.path_out, self.path_len,
            self.t["k"], self.t["v"], self.t["g"], self.t["beta"], self.state,
            self.channels if use_conv else 0, self.x if use_conv else None,
            self.hist if use_conv else None, self.prep)

    def reset_state(self):
        self.state.copy_(self.state0)

    @classmethod
    def from_workload(cls, wl, *, policy=0, with_conv=True, **kw):
        a = dict(wl.arrays)
        if not with_conv:
            for key in ("x", "hist", "w"):
                a.pop(key, None)
        return cls(n_req=wl.n_req, n_layers=wl.n_layers, h_k=wl.h_k, h_v=wl.h_v, d_k=wl.d_k,
                   d_v=wl.d_v, op_dtype=wl.op_dtype, node_off=wl.node_off, parent=wl.parent_flat,
                   n_rows=wl.n_rows, arrays=a, policy=policy, max_path=wl.max_path,
                   accepted=wl.accepted, channels=wl.channels if with_conv else 0, **kw)
