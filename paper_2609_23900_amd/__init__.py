"""Python binding of liblumo_tree.so (tree verification of the Gated DeltaNet recurrence
on MI355X / gfx950). Argument marshalling only: every step runs in the library's HIP
kernels; torch tensors only provide device memory and the current HIP stream.

The functions keep the names of the C ABI (include/lumo_tree.h):
  lumo_tree_plan, lumo_tree_gdn_workspace_bytes, lumo_tree_conv_gather,
  lumo_tree_conv_gather_pending, lumo_tree_gdn_verify, lumo_tree_gdn_verify_prep, lumo_tree_gdn_verify_pending,
  lumo_tree_gdn_verify_conv_pending, lumo_gdn_commit,
  lumo_gdn_commit_prep, lumo_tree_attention, lumo_tree_attention_noalloc,
  lumo_tree_attention_workspace_bytes,
  lumo_tree_attention_splits, lumo_draft_select, lumo_draft_select_workspace_bytes,
  lumo_draft_select_splits, lumo_gdn_commit_graph_create,
  lumo_gdn_commit_graph_launch, lumo_gdn_commit_graph_destroy, lumo_last_error,
  lumo_version.
Device arguments are torch tensors on the GPU (or None where the ABI allows NULL);
host arguments are numpy int32 arrays. A non-OK status raises LumoError.

Importing this module loads the library and fails if it has not been built
(python -m paper_2609_23900_amd.build); there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # loads the process's HIP runtime before the library binds to it

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblumo_tree.so")

LUMO_OK, LUMO_EINVAL, LUMO_EDESC, LUMO_ESHAPE, LUMO_EUNSUPPORTED, LUMO_EHIP, LUMO_ESPACE = range(7)
LUMO_F32, LUMO_BF16 = 0, 1
LUMO_POLICY_PATHS, LUMO_POLICY_TWO_LEVEL, LUMO_POLICY_RECOMPUTE, LUMO_POLICY_WY = range(4)
POLICIES = {"paths": 0, "two_level": 1, "recompute": 2, "wy": 3}
STATUS_NAMES = ("LUMO_OK", "LUMO_EINVAL", "LUMO_EDESC", "LUMO_ESHAPE", "LUMO_EUNSUPPORTED",
                "LUMO_EHIP", "LUMO_ESPACE")


class LumoError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES[status] if 0 <= status < 7 else status}: {msg}")
        self.status = status


class lumo_gdn_dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_req", "n_layers", "h_k", "h_v", "d_k", "d_v", "op_dtype")]


_PLAN_FIELDS = ("n_req", "total_nodes", "total_rows", "max_nodes", "max_depth", "policy",
                "n_paths", "n_spine", "n_seg", "n_seg_nodes", "n_levels", "n_cuts",
                "max_level_seg", "max_seg_len", "n_words", "o_node_off", "o_row_off", "o_req",
                "o_parent", "o_depth", "o_slot", "o_row", "o_conv_src", "o_path_off",
                "o_path_leaf", "o_spine_off", "o_spine", "o_level_off", "o_seg", "o_seg_nodes",
                "o_dfs", "o_dfs_pos", "n_chunks", "o_pre_row", "o_pre_depth",
                "o_pre_ci", "o_chunk_off", "o_chunk_stack", "o_vis")


class lumo_plan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in _PLAN_FIELDS]


class lumo_tree_desc(ctypes.Structure):
    _fields_ = [("blob", ctypes.c_void_p), ("host_blob", ctypes.c_void_p), ("plan", lumo_plan)]


class lumo_attn_dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_req", "h_q", "h_kv", "d", "op_dtype")]


LUMO_PREP_QK_NORM, LUMO_PREP_RAW_GATES = 1, 2


class lumo_gdn_prep(ctypes.Structure):
    _fields_ = [("flags", ctypes.c_int32), ("qk_eps", ctypes.c_float), ("a_log", ctypes.c_void_p),
                ("dt_bias", ctypes.c_void_p)]


class lumo_gdn_pending_call(ctypes.Structure):
    _fields_ = [("dims", ctypes.POINTER(lumo_gdn_dims)), ("desc", ctypes.POINTER(lumo_tree_desc)),
                ("prep", ctypes.POINTER(lumo_gdn_prep)), ("q", ctypes.c_void_p), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("g", ctypes.c_void_p), ("beta", ctypes.c_void_p),
                ("state", ctypes.c_void_p), ("o", ctypes.c_void_p), ("pend_desc", ctypes.POINTER(lumo_tree_desc)),
                ("max_path", ctypes.c_int32), ("path_out", ctypes.c_void_p), ("path_len", ctypes.c_void_p),
                ("pend_k", ctypes.c_void_p), ("pend_v", ctypes.c_void_p), ("pend_g", ctypes.c_void_p),
                ("pend_beta", ctypes.c_void_p)]


class Prep:
    """Operand preparation (lumo_gdn_prep): flags, qk_eps and, for raw gates, the device
    tensors a_log and dt_bias [n_layers][h_v] fp32 (kept alive here)."""

    def __init__(self, flags, qk_eps=1e-6, a_log=None, dt_bias=None):
        self.a_log, self.dt_bias = a_log, dt_bias
        self.c = lumo_gdn_prep(int(flags), float(qk_eps), _dptr(a_log), _dptr(dt_bias))


def _prep_ptr(prep):
    return None if prep is None else ctypes.byref(prep.c)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run `python paper_2609_23900_amd/build.py` "
                          "(hipcc, gfx950); there is no fallback implementation")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    PD = ctypes.POINTER(lumo_gdn_dims)
    PT = ctypes.POINTER(lumo_tree_desc)
    L.lumo_tree_plan.argtypes = [I32, P, P, P, I32, P, I64, ctypes.POINTER(lumo_plan)]
    L.lumo_tree_gdn_workspace_bytes.argtypes = [PD, ctypes.POINTER(lumo_plan)]
    L.lumo_tree_gdn_workspace_bytes.restype = SZ
    L.lumo_tree_conv_gather.argtypes = [PD, PT, I32, P, P, P, P, I32, P, P]
    L.lumo_tree_conv_gather_pending.argtypes = [PD, PT, I32, P, P, P, P, I32, P, PT, I32, P, P, P, P]
    L.lumo_tree_gdn_verify.argtypes = [PD, PT, P, P, P, P, P, P, P, P, P, SZ, I32, P]
    PP = ctypes.POINTER(lumo_gdn_prep)
    PA = ctypes.POINTER(lumo_attn_dims)
    L.lumo_tree_attention_workspace_bytes.argtypes = [PA, ctypes.POINTER(lumo_plan), I32]
    L.lumo_tree_attention_workspace_bytes.restype = SZ
    L.lumo_tree_attention_splits.argtypes = [PA, ctypes.POINTER(lumo_plan), I32]
    L.lumo_tree_attention_splits.restype = I32
    L.lumo_tree_attention.argtypes = [PA, PT, P, I32, ctypes.c_float, P, P, P, P, P, P, P, I32, P, SZ, P]
    L.lumo_tree_attention_noalloc.argtypes = [PA, PT, P, I32, ctypes.c_float, P, P, P, P, P, P, P, I32, P]
    L.lumo_draft_select_workspace_bytes.argtypes = [I32, I32, I32]
    L.lumo_draft_select_workspace_bytes.restype = SZ
    L.lumo_draft_select_splits.argtypes = [I32, I32, I32]
    L.lumo_draft_select_splits.restype = I32
    L.lumo_draft_select.argtypes = [I32, I32, I64, I32, I32, I32, P, P, P, I32, P, SZ, P]
    L.lumo_tree_gdn_verify_prep.argtypes = [PD, PT, PP, P, P, P, P, P, P, P, P]
    L.lumo_tree_gdn_verify_pending.argtypes = [PD, PT, PP, P, P, P, P, P, P, P, PT, I32, P, P, P, P, P, P,
                                               P]
    L.lumo_tree_gdn_verify_pending_pair.argtypes = [ctypes.POINTER(lumo_gdn_pending_call),
                                                    ctypes.POINTER(lumo_gdn_pending_call), P]
    L.lumo_tree_gdn_verify_conv_pending.argtypes = [PD, PT, PP, I32, P, P, P, P, I32, P, P, P, P, PT, I32, P, P,
                                                    P, P, P, P]
    L.lumo_gdn_commit_prep.argtypes = [PD, PT, PP, I32, P, P, P, P, P, P, P, P, I32, P, P, P]
    L.lumo_gdn_commit.argtypes = [PD, PT, I32, P, P, P, P, P, P, P, P, I32, P, P, P]
    L.lumo_gdn_commit_hist_layers.argtypes = [PD, PT, I32, P, P, P, I32, P, P, P]
    L.lumo_gdn_commit_graph_create.argtypes = [PD, PT, PP, I32, P, P, P, P, P, P, P, P, I32, P, P,
                                               ctypes.POINTER(ctypes.c_void_p)]
    L.lumo_gdn_commit_graph_launch.argtypes = [P, P]
    L.lumo_gdn_commit_graph_destroy.argtypes = [P]
    L.lumo_gdn_commit_graph_destroy.restype = None
    L.lumo_last_error.restype = ctypes.c_char_p
    L.lumo_version.restype = ctypes.c_char_p
    for f in ("lumo_tree_plan", "lumo_tree_conv_gather", "lumo_tree_conv_gather_pending", "lumo_tree_gdn_verify",
              "lumo_tree_gdn_verify_prep", "lumo_tree_gdn_verify_pending", "lumo_tree_gdn_verify_conv_pending", "lumo_gdn_commit",
              "lumo_gdn_commit_prep", "lumo_gdn_commit_hist_layers", "lumo_tree_gdn_verify_pending_pair", "lumo_tree_attention", "lumo_tree_attention_noalloc", "lumo_draft_select", "lumo_gdn_commit_graph_create", "lumo_gdn_commit_graph_launch"):
        getattr(L, f).restype = ctypes.c_int
    return L


_lib = _load()


def lumo_last_error() -> str:
    return _lib.lumo_last_error().decode()


def lumo_version() -> str:
    return _lib.lumo_version().decode()


def _check(st: int):
    if st != LUMO_OK:
        raise LumoError(st, lumo_last_error())


def _dptr(t):
    """Device pointer of a tensor (None -> NULL)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("device arguments must be torch tensors")
    if not t.is_cuda:
        raise ValueError("device argument is not on the GPU")
    if not t.is_contiguous():
        raise ValueError("device argument must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _hptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def dims(n_req, n_layers, h_k, h_v, d_k, d_v, op_dtype) -> lumo_gdn_dims:
    return lumo_gdn_dims(n_req, n_layers, h_k, h_v, d_k, d_v, op_dtype)


def lumo_tree_plan(node_off, parent, n_rows, policy=LUMO_POLICY_PATHS):
    """Host planner. Returns (plan summary, int32 numpy blob)."""
    node_off = np.ascontiguousarray(node_off, dtype=np.int32)
    parent = np.ascontiguousarray(parent, dtype=np.int32)
    n_rows = np.ascontiguousarray(n_rows, dtype=np.int32)
    n_req = int(node_off.shape[0]) - 1
    plan = lumo_plan()
    st = _lib.lumo_tree_plan(n_req, _hptr(node_off), _hptr(parent) if parent.size else None,
                             _hptr(n_rows) if n_rows.size else None, int(policy), None, 0,
                             ctypes.byref(plan))
    if st != LUMO_ESPACE:
        _check(st)
    blob = np.zeros(max(plan.n_words, 1), dtype=np.int32)
    _check(_lib.lumo_tree_plan(n_req, _hptr(node_off), _hptr(parent) if parent.size else None,
                               _hptr(n_rows) if n_rows.size else None, int(policy), _hptr(blob),
                               blob.shape[0], ctypes.byref(plan)))
    return plan, blob


class TreeDesc:
    """A plan plus its device copy (keeps both buffers alive)."""

    def __init__(self, plan: lumo_plan, blob: np.ndarray, device="cuda"):
        self.plan = plan
        self.host = np.ascontiguousarray(blob, dtype=np.int32)
        self.dev = torch.from_numpy(self.host).to(device)
        self.desc = lumo_tree_desc(ctypes.c_void_p(self.dev.data_ptr()), _hptr(self.host), plan)

    @classmethod
    def build(cls, node_off, parent, n_rows, policy=LUMO_POLICY_PATHS, device="cuda"):
        plan, blob = lumo_tree_plan(node_off, parent, n_rows, policy)
        return cls(plan, blob, device)

    def section(self, name, count):
        off = getattr(self.plan, "o_" + name)
        return self.host[off:off + count]


def lumo_tree_gdn_workspace_bytes(d: lumo_gdn_dims, plan: lumo_plan) -> int:
    return int(_lib.lumo_tree_gdn_workspace_bytes(ctypes.byref(d), ctypes.byref(plan)))


def lumo_tree_conv_gather(d, desc: TreeDesc, channels, x, conv_hist, w, bias, act, y, stream=None):
    _check(_lib.lumo_tree_conv_gather(ctypes.byref(d), ctypes.byref(desc.desc), int(channels),
                                      _dptr(x), _dptr(conv_hist), _dptr(w), _dptr(bias), int(act),
                                      _dptr(y), _stream(stream)))


def lumo_tree_conv_gather_pending(d, desc: TreeDesc, channels, x, conv_hist, w, bias, act, y,
                                  pend_desc: TreeDesc, max_path, path_out, path_len, x_prev,
                                  stream=None):
    _check(_lib.lumo_tree_conv_gather_pending(
        ctypes.byref(d), ctypes.byref(desc.desc), int(channels), _dptr(x), _dptr(conv_hist), _dptr(w),
        _dptr(bias), int(act), _dptr(y), ctypes.byref(pend_desc.desc), int(max_path), _dptr(path_out),
        _dptr(path_len), _dptr(x_prev), _stream(stream)))


def lumo_tree_gdn_verify(d, desc: TreeDesc, q, k, v, g, beta, state0, o, node_states=None,
                         workspace=None, flags=0, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.lumo_tree_gdn_verify(ctypes.byref(d), ctypes.byref(desc.desc), _dptr(q), _dptr(k),
                                     _dptr(v), _dptr(g), _dptr(beta), _dptr(state0), _dptr(o),
                                     _dptr(node_states), _dptr(workspace), ws_bytes, int(flags),
                                     _stream(stream)))


def lumo_tree_gdn_verify_prep(d, desc: TreeDesc, prep: Prep | None, q, k, v, g, beta, state0, o,
                              stream=None):
    _check(_lib.lumo_tree_gdn_verify_prep(ctypes.byref(d), ctypes.byref(desc.desc), _prep_ptr(prep),
                                          _dptr(q), _dptr(k), _dptr(v), _dptr(g), _dptr(beta),
                                          _dptr(state0), _dptr(o), _stream(stream)))


def pending_call(d, desc: TreeDesc, q, k, v, g, beta, state, o, pend_desc: TreeDesc, max_path, path_out,
                 path_len, pend_k, pend_v, pend_g, pend_beta, prep: Prep | None = None):
    """The arguments of lumo_tree_gdn_verify_pending as one lumo_gdn_pending_call (the
    struct keeps the objects it points to alive)."""
    c = lumo_gdn_pending_call(ctypes.pointer(d), ctypes.pointer(desc.desc),
                              None if prep is None else ctypes.pointer(prep.c), _dptr(q), _dptr(k), _dptr(v),
                              _dptr(g), _dptr(beta), _dptr(state), _dptr(o), ctypes.pointer(pend_desc.desc),
                              int(max_path), _dptr(path_out), _dptr(path_len), _dptr(pend_k), _dptr(pend_v),
                              _dptr(pend_g), _dptr(pend_beta))
    c._refs = (d, desc, pend_desc, prep)
    return c


def lumo_tree_gdn_verify_pending_pair(a, b=None, stream=None):
    """a, b: pending_call(...) structs; b may be None."""
    _check(_lib.lumo_tree_gdn_verify_pending_pair(ctypes.byref(a), None if b is None else ctypes.byref(b),
                                                  _stream(stream)))


def lumo_tree_gdn_verify_pending(d, desc: TreeDesc, q, k, v, g, beta, state, o, pend_desc: TreeDesc,
                                 max_path, path_out, path_len, pend_k, pend_v, pend_g, pend_beta,
                                 stream=None, prep: Prep | None = None):
    _check(_lib.lumo_tree_gdn_verify_pending(
        ctypes.byref(d), ctypes.byref(desc.desc), _prep_ptr(prep), _dptr(q), _dptr(k), _dptr(v), _dptr(g),
        _dptr(beta), _dptr(state), _dptr(o), ctypes.byref(pend_desc.desc), int(max_path),
        _dptr(path_out), _dptr(path_len), _dptr(pend_k), _dptr(pend_v), _dptr(pend_g),
        _dptr(pend_beta), _stream(stream)))


def lumo_tree_gdn_verify_conv_pending(d, desc: TreeDesc, channels, x, conv_hist, w, bias, act, g, beta, state, o,
                                      pend_desc: TreeDesc, max_path, path_out, path_len, x_prev, pend_g,
                                      pend_beta, stream=None, prep: Prep | None = None):
    _check(_lib.lumo_tree_gdn_verify_conv_pending(
        ctypes.byref(d), ctypes.byref(desc.desc), _prep_ptr(prep), int(channels), _dptr(x), _dptr(conv_hist),
        _dptr(w), _dptr(bias), int(act), _dptr(g), _dptr(beta), _dptr(state), _dptr(o),
        ctypes.byref(pend_desc.desc), int(max_path), _dptr(path_out), _dptr(path_len), _dptr(x_prev),
        _dptr(pend_g), _dptr(pend_beta), _stream(stream)))


def lumo_gdn_commit(d, desc: TreeDesc, max_path, accepted_node, path_out, path_len, k, v, g, beta,
                    state, channels=0, x=None, conv_hist=None, stream=None):
    _check(_lib.lumo_gdn_commit(ctypes.byref(d), ctypes.byref(desc.desc), int(max_path),
                                _dptr(accepted_node), _dptr(path_out), _dptr(path_len), _dptr(k),
                                _dptr(v), _dptr(g), _dptr(beta), _dptr(state), int(channels),
                                _dptr(x), _dptr(conv_hist), _stream(stream)))


def lumo_gdn_commit_hist_layers(d, desc: TreeDesc, max_path, accepted_node, path_out, path_len, channels,
                                x_layers, conv_hist_layers, stream=None):
    """x_layers, conv_hist_layers: one device tensor per layer (None allowed in x_layers
    when the tree has no nodes); the pointer tables are built here, on the host."""
    n = len(conv_hist_layers)
    if len(x_layers) != n:
        raise ValueError("x_layers and conv_hist_layers need one entry per layer")
    xt = (ctypes.c_void_p * max(n, 1))(*[_dptr(t) for t in x_layers])
    ht = (ctypes.c_void_p * max(n, 1))(*[_dptr(t) for t in conv_hist_layers])
    _check(_lib.lumo_gdn_commit_hist_layers(ctypes.byref(d), ctypes.byref(desc.desc), int(max_path),
                                            _dptr(accepted_node), _dptr(path_out), _dptr(path_len),
                                            int(channels), xt, ht, _stream(stream)))


def lumo_gdn_commit_prep(d, desc: TreeDesc, prep: Prep | None, max_path, accepted_node, path_out,
                         path_len, k, v, g, beta, state, channels=0, x=None, conv_hist=None,
                         stream=None):
    _check(_lib.lumo_gdn_commit_prep(ctypes.byref(d), ctypes.byref(desc.desc), _prep_ptr(prep),
                                     int(max_path), _dptr(accepted_node), _dptr(path_out),
                                     _dptr(path_len), _dptr(k), _dptr(v), _dptr(g), _dptr(beta),
                                     _dptr(state), int(channels), _dptr(x), _dptr(conv_hist),
                                     _stream(stream)))


def attn_dims(n_req, h_q, h_kv, d=128, op_dtype=LUMO_BF16) -> lumo_attn_dims:
    return lumo_attn_dims(n_req, h_q, h_kv, d, op_dtype)


def lumo_tree_attention_workspace_bytes(d: lumo_attn_dims, plan: lumo_plan, n_split) -> int:
    return int(_lib.lumo_tree_attention_workspace_bytes(ctypes.byref(d), ctypes.byref(plan), int(n_split)))


def lumo_tree_attention_splits(d: lumo_attn_dims, plan: lumo_plan, max_ctx) -> int:
    return int(_lib.lumo_tree_attention_splits(ctypes.byref(d), ctypes.byref(plan), int(max_ctx)))


def lumo_tree_attention(d, desc: TreeDesc, ctx_off, max_ctx, scale, q, k_ctx, v_ctx, k_tree, v_tree,
                        o, lse, n_split, workspace, stream=None):
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.lumo_tree_attention(ctypes.byref(d), ctypes.byref(desc.desc), _dptr(ctx_off),
                                    int(max_ctx), float(scale), _dptr(q), _dptr(k_ctx), _dptr(v_ctx),
                                    _dptr(k_tree), _dptr(v_tree), _dptr(o), _dptr(lse), int(n_split),
                                    _dptr(workspace), ws_bytes, _stream(stream)))


# Bytes of the fixed per-device scratch array behind lumo_tree_attention_noalloc.
LUMO_TREE_ATTENTION_SCRATCH_BYTES = 32 << 20


def lumo_tree_attention_noalloc(d, desc: TreeDesc, ctx_off, max_ctx, scale, q, k_ctx, v_ctx, k_tree,
                                v_tree, o, lse, n_split, stream=None):
    _check(_lib.lumo_tree_attention_noalloc(ctypes.byref(d), ctypes.byref(desc.desc), _dptr(ctx_off),
                                            int(max_ctx), float(scale), _dptr(q), _dptr(k_ctx),
                                            _dptr(v_ctx), _dptr(k_tree), _dptr(v_tree), _dptr(o),
                                            _dptr(lse), int(n_split), _stream(stream)))


def _logits_dtype(t):
    if t.dtype == torch.float32:
        return LUMO_F32
    if t.dtype == torch.bfloat16:
        return LUMO_BF16
    raise TypeError("logits must be float32 or bfloat16")


def lumo_draft_select_workspace_bytes(rows, k, n_split) -> int:
    return int(_lib.lumo_draft_select_workspace_bytes(int(rows), int(k), int(n_split)))


def lumo_draft_select_splits(rows, vocab, dtype) -> int:
    return int(_lib.lumo_draft_select_splits(int(rows), int(vocab), int(dtype)))


def lumo_draft_select(logits, k, ties, spine, cand, n_split, workspace, stream=None, vocab=None):
    """logits: contiguous [rows][ld] float32 or bfloat16 tensor; the first `vocab`
    (default ld) entries of each row are ranked. spine int32 [rows], cand int32 [rows][k]."""
    if logits.dim() != 2:
        raise ValueError("logits must be [rows][ld]")
    rows, ld = logits.shape
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.lumo_draft_select(int(rows), int(ld if vocab is None else vocab), int(ld), _logits_dtype(logits),
                                  int(k), int(ties), _dptr(logits), _dptr(spine), _dptr(cand), int(n_split),
                                  _dptr(workspace), ws_bytes, _stream(stream)))


class CommitGraph:
    """Captured fixed-shape commit (lumo_gdn_commit_graph_*)."""

    def __init__(self, handle, keep):
        self.handle = handle
        self._keep = keep

    def launch(self, stream=None):
        lumo_gdn_commit_graph_launch(self, stream)

    def close(self):
        if self.handle:
            lumo_gdn_commit_graph_destroy(self)

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def lumo_gdn_commit_graph_create(d, desc: TreeDesc, max_path, accepted_node, path_out, path_len,
                                 k, v, g, beta, state, channels=0, x=None, conv_hist=None, prep=None):
    h = ctypes.c_void_p()
    _check(_lib.lumo_gdn_commit_graph_create(ctypes.byref(d), ctypes.byref(desc.desc), _prep_ptr(prep),
                                             int(max_path), _dptr(accepted_node), _dptr(path_out),
                                             _dptr(path_len), _dptr(k), _dptr(v), _dptr(g),
                                             _dptr(beta), _dptr(state), int(channels), _dptr(x),
                                             _dptr(conv_hist), ctypes.byref(h)))
    return CommitGraph(h, (desc, accepted_node, path_out, path_len, k, v, g, beta, state, x,
                           conv_hist, prep))


def lumo_gdn_commit_graph_launch(graph: CommitGraph, stream=None):
    _check(_lib.lumo_gdn_commit_graph_launch(graph.handle, _stream(stream)))


def lumo_gdn_commit_graph_destroy(graph: CommitGraph):
    _lib.lumo_gdn_commit_graph_destroy(graph.handle)
    graph.handle = None
