"""fp64 CPU oracle for tree GDN verification, commit and tree convolution.

TEST INFRASTRUCTURE ONLY. Imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg; the GPU library and its Python binding never import it.

The arithmetic lives in lumo_oracle.c (plain C, fp64); the integer descriptor
products are derived in plan.py. build() compiles the C file with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import plan  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lumo_oracle.c")
_LIB = os.path.join(_HERE, "liblumo_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP over independent instances)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class Dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in (
        "n_req", "n_layers", "h_k", "h_v", "d_k", "d_v", "op_dtype", "total_rows",
        "gate_is_alpha", "prep_flags")] + [
        ("qk_eps", ctypes.c_double), ("a_log", ctypes.c_void_p), ("dt_bias", ctypes.c_void_p)]


PREP_QK_NORM, PREP_RAW_GATES = 1, 2


class Prep:
    """Sec. IV-B operand preparation: flags (PREP_QK_NORM | PREP_RAW_GATES), the
    normalisation constant, and the per-(layer, value head) gate parameters."""

    def __init__(self, flags, eps=1e-6, a_log=None, dt_bias=None):
        self.flags = int(flags)
        self.eps = float(eps)
        self.a_log = _c(a_log, np.float32)
        self.dt_bias = _c(dt_bias, np.float32)
        if self.flags & PREP_RAW_GATES and (self.a_log is None or self.dt_bias is None):
            raise ValueError("raw gates need a_log and dt_bias")


def use_library(path=None):
    """Point the wrappers at another build of lumo_oracle.c (None: the default build).

    Used by the mutation tests, which compile deliberately broken copies of the
    oracle and check that the pins reject them."""
    global _lib
    _lib = None if path is None else _load(path)


def _load(path):
    L = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I = ctypes.c_int
    L.orc_verify_nodes.argtypes = [ctypes.POINTER(Dims), I, P, P, I, I, I, I, P, P, P, P, P,
                                   P, P, P, P]
    L.orc_verify_all.argtypes = [ctypes.POINTER(Dims), P, P, P, P, P, P, P, P, P, P, I]
    L.orc_commit.argtypes = [ctypes.POINTER(Dims), P, P, P, P, I, P, P, P, P, P, P, P, P, I]
    L.orc_conv_all.argtypes = [I, I, I, I, I, P, P, P, P, P, P, P, I, P]
    L.orc_conv_hist_publish.argtypes = [I, I, I, I, I, P, P, P, P, I, P, P, P]
    L.orc_tree_attention.argtypes = [I, I, I, I, I, P, P, P, P, ctypes.c_double, P, P, P, P, P, P, P, I]
    L.orc_draft_select.argtypes = [I, I, I, I, I, P, P, P, I]
    for f in ("orc_verify_nodes", "orc_verify_all", "orc_commit", "orc_conv_all",
              "orc_conv_hist_publish", "orc_tree_attention", "orc_draft_select", "orc_max_threads"):
        getattr(L, f).restype = I
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        _lib = _load(_LIB)
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def _op(a, op_dtype):
    return np.ascontiguousarray(a, dtype=np.float32 if op_dtype == 0 else np.uint16)


def dims(wl, gate_is_alpha=False, prep: Prep | None = None) -> Dims:
    """The oracle's dimensions; `prep` must stay alive while the result is used."""
    if prep is None:
        return Dims(wl.n_req, wl.n_layers, wl.h_k, wl.h_v, wl.d_k, wl.d_v, wl.op_dtype,
                    wl.total_rows, int(gate_is_alpha), 0, 0.0, None, None)
    return Dims(wl.n_req, wl.n_layers, wl.h_k, wl.h_v, wl.d_k, wl.d_v, wl.op_dtype,
                wl.total_rows, int(gate_is_alpha), prep.flags, prep.eps, _p(prep.a_log),
                _p(prep.dt_bias))


class _Ops:
    def __init__(self, wl, arrays=None):
        a = wl.arrays if arrays is None else arrays
        self.q = _op(a["q"], wl.op_dtype)
        self.k = _op(a["k"], wl.op_dtype)
        self.v = _op(a["v"], wl.op_dtype)
        self.g = _c(a["g"], np.float32)
        self.beta = _c(a["beta"], np.float32)
        self.state0 = _c(a["state0"], np.float32)


def verify_nodes(wl, r, l, h, targets, *, arrays=None, gate_is_alpha=False, want_state=False,
                 prep=None):
    """o (and state) of the given request-local nodes of instance (r, l, h), fp64."""
    d = dims(wl, gate_is_alpha, prep)
    par = _c(wl.parents[r], np.int32)
    rows = _c(plan.rows_of(wl.parents[r], int(wl.row_off[r])), np.int32)
    tg = _c(targets, np.int32)
    o = np.zeros((len(tg), wl.d_v), np.float64)
    st = np.zeros((len(tg), wl.d_k, wl.d_v), np.float64) if want_state else None
    x = _Ops(wl, arrays)
    rc = lib().orc_verify_nodes(ctypes.byref(d), len(par), _p(par), _p(rows), r, l, h, len(tg),
                                _p(tg), _p(x.q), _p(x.k), _p(x.v), _p(x.g), _p(x.beta),
                                _p(x.state0), _p(o), _p(st))
    if rc:
        raise ValueError("oracle: malformed tree")
    return (o, st) if want_state else o


def verify_all(wl, *, arrays=None, gate_is_alpha=False, n_threads=None, prep=None):
    """All outputs [layers][rows][h_v][d_v] in fp64 (pad rows NaN)."""
    d = dims(wl, gate_is_alpha, prep)
    rows = plan.flat_rows(wl.parents, wl.row_off)
    o = np.full((wl.n_layers, wl.total_rows, wl.h_v, wl.d_v), np.nan, np.float64)
    x = _Ops(wl, arrays)
    nt = n_threads or lib().orc_max_threads()
    rc = lib().orc_verify_all(ctypes.byref(d), _p(_c(wl.node_off, np.int32)),
                              _p(_c(wl.parent_flat, np.int32)), _p(rows), _p(x.q), _p(x.k),
                              _p(x.v), _p(x.g), _p(x.beta), _p(x.state0), _p(o), int(nt))
    if rc:
        raise ValueError("oracle: malformed tree")
    return o


def commit(wl, accepted=None, *, arrays=None, state_in=None, gate_is_alpha=False,
           max_path=None, n_threads=None, prep=None):
    """(published state fp64, path_out int32, path_len int32)."""
    d = dims(wl, gate_is_alpha, prep)
    a = wl.arrays if arrays is None else arrays
    acc = _c(wl.accepted if accepted is None else accepted, np.int32)
    mp = int(wl.max_path if max_path is None else max_path)
    rows = plan.flat_rows(wl.parents, wl.row_off)
    x = _Ops(wl, arrays)
    s_in = x.state0 if state_in is None else _c(state_in, np.float32)
    out = np.zeros(s_in.shape, np.float64)
    po = np.zeros((wl.n_req, mp), np.int32)
    pl = np.zeros((wl.n_req,), np.int32)
    nt = n_threads or lib().orc_max_threads()
    rc = lib().orc_commit(ctypes.byref(d), _p(_c(wl.node_off, np.int32)),
                          _p(_c(wl.parent_flat, np.int32)), _p(rows), _p(acc), mp, _p(x.k),
                          _p(x.v), _p(x.g), _p(x.beta), _p(s_in), _p(out), _p(po), _p(pl),
                          int(nt))
    if rc:
        raise ValueError("oracle: malformed accepted path")
    del a
    return out, po, pl


def conv_all(wl, *, arrays=None, bias=None, act=1):
    a = wl.arrays if arrays is None else arrays
    rows = plan.flat_rows(wl.parents, wl.row_off)
    y = np.full((wl.n_layers, wl.total_rows, wl.channels), np.nan, np.float64)
    rc = lib().orc_conv_all(wl.n_req, wl.n_layers, wl.total_rows, wl.channels, wl.op_dtype,
                            _p(_c(wl.node_off, np.int32)), _p(_c(wl.parent_flat, np.int32)),
                            _p(rows), _p(_op(a["x"], wl.op_dtype)),
                            _p(_op(a["hist"], wl.op_dtype)), _p(_c(a["w"], np.float32)),
                            _p(_c(bias, np.float32)), int(act), _p(y))
    if rc:
        raise ValueError("oracle: malformed tree")
    return y


def conv_hist_publish(wl, path_out, path_len, *, arrays=None):
    a = wl.arrays if arrays is None else arrays
    rows = plan.flat_rows(wl.parents, wl.row_off)
    po = _c(path_out, np.int32)
    out = np.zeros((wl.n_req, wl.n_layers, 3, wl.channels), np.float64)
    lib().orc_conv_hist_publish(wl.n_req, wl.n_layers, wl.total_rows, wl.channels, wl.op_dtype,
                                _p(_c(wl.node_off, np.int32)), _p(rows), _p(po),
                                _p(_c(path_len, np.int32)), po.shape[1],
                                _p(_op(a["x"], wl.op_dtype)), _p(_op(a["hist"], wl.op_dtype)),
                                _p(out))
    return out


def tree_attention(parents, row_off, total_rows, ctx_off, q, k_ctx, v_ctx, k_tree, v_tree, *,
                   h_q, h_kv, d, op_dtype, scale=None, n_threads=None):
    """(o [rows][h_q][d], lse [rows][h_q]) in fp64; rows without a node are NaN.

    Row i of request r attends to its context tokens ctx_off[r] .. ctx_off[r+1]-1 and to
    the tree nodes of its own root-to-node path (Sec. V-B)."""
    node_off = np.zeros(len(parents) + 1, np.int32)
    node_off[1:] = np.cumsum([len(p) for p in parents])
    parent_flat = np.concatenate([np.asarray(p, np.int32) for p in parents]) if len(parents) else np.zeros(0, np.int32)
    rows = plan.flat_rows(parents, row_off) if len(parents) else np.zeros(0, np.int32)
    o = np.full((total_rows, h_q, d), np.nan, np.float64)
    lse = np.full((total_rows, h_q), np.nan, np.float64)
    sc = 1.0 / np.sqrt(d) if scale is None else float(scale)
    nt = n_threads or lib().orc_max_threads()
    rc = lib().orc_tree_attention(len(parents), h_q, h_kv, d, op_dtype, _p(node_off),
                                  _p(_c(parent_flat, np.int32)), _p(_c(rows, np.int32)),
                                  _p(_c(ctx_off, np.int32)), sc, _p(_op(q, op_dtype)),
                                  _p(_op(k_ctx, op_dtype)), _p(_op(v_ctx, op_dtype)),
                                  _p(_op(k_tree, op_dtype)), _p(_op(v_tree, op_dtype)), _p(o), _p(lse),
                                  int(nt))
    if rc:
        raise ValueError("oracle: malformed tree")
    return o, lse


def draft_select(logits, *, k, op_dtype, ties=0, n_threads=None):
    """(spine [rows], cand [rows][k]) int32 of a logits array [rows][vocab] (Sec. V-D):
    spine = lowest index among each row's maximal logits; cand = the k indices ranked
    first by logit, descending, ties by index ascending (ties=0) or descending (ties=1).
    NaN ranks above every number."""
    x = _op(logits, op_dtype)
    if x.ndim != 2:
        raise ValueError("logits must be [rows][vocab]")
    rows, vocab = x.shape
    spine = np.empty(rows, np.int32)
    cand = np.empty((rows, k), np.int32)
    nt = n_threads if n_threads is not None else lib().orc_max_threads()
    if lib().orc_draft_select(rows, vocab, int(k), int(op_dtype), int(ties), _p(x), _p(spine), _p(cand), int(nt)):
        raise ValueError("oracle: k must be in 1..vocab and ties 0 or 1")
    return spine, cand
