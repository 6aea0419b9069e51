"""The C ABI without a GPU: the library loads, exports every function that
include/lumo_tree.h declares, and rejects bad arguments on the host (documented
status codes) before anything would be launched. No compute call is made here."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2609_23900_amd as L
from lumo_synth import trees

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lumo_tree.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lumo_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ("lumo_tree_plan", "lumo_tree_conv_gather", "lumo_tree_gdn_verify", "lumo_gdn_commit",
              "lumo_gdn_commit_graph_create", "lumo_gdn_commit_graph_launch",
              "lumo_gdn_commit_graph_destroy", "lumo_tree_gdn_workspace_bytes", "lumo_last_error"):
        assert f in names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", L.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (lumo_\w+)", out))
    missing = [f for f in declared_functions() if f not in exported]
    assert not missing, missing
    for f in declared_functions():
        assert hasattr(L._lib, f)


def test_binding_names_match_abi():
    for f in declared_functions():
        assert callable(getattr(L, f)), f


def test_version():
    assert "gfx950" in L.lumo_version()


# ---------------------------------------------------------------- host-side rejection
FAKE = 0x10000  # an aligned address that is never dereferenced (validation fails first)


def _desc(n_req=1, policy=0):
    par = trees.FIG1_PARENT
    plan, blob = L.lumo_tree_plan(np.array([0, 7] if n_req == 1 else [0, 7, 14], np.int32),
                                  np.concatenate([par] * n_req),
                                  np.array([7] * n_req, np.int32), policy)
    d = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    return d, blob


def _verify(d, desc, ptrs=None, ws=0, flags=0):
    p = [ctypes.c_void_p(FAKE)] * 7 if ptrs is None else ptrs
    return L._lib.lumo_tree_gdn_verify(ctypes.byref(d), ctypes.byref(desc), *p, None,
                                       ctypes.c_void_p(FAKE), ws, flags, None)


def _dims(**kw):
    base = dict(n_req=1, n_layers=1, h_k=1, h_v=1, d_k=16, d_v=16, op_dtype=0)
    base.update(kw)
    return L.lumo_gdn_dims(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(d_k=48), L.LUMO_EUNSUPPORTED), (dict(d_v=256), L.LUMO_EUNSUPPORTED),
    (dict(h_k=2, h_v=3), L.LUMO_ESHAPE), (dict(n_layers=0), L.LUMO_ESHAPE),
    (dict(op_dtype=7), L.LUMO_EUNSUPPORTED), (dict(n_req=2), L.LUMO_EDESC)])
def test_verify_rejects_bad_dims(kw, status):
    desc, _blob = _desc()
    assert _verify(_dims(**kw), desc) == status
    assert L.lumo_last_error()


def test_verify_rejects_null_and_misaligned():
    desc, _blob = _desc()
    ptrs = [ctypes.c_void_p(FAKE)] * 7
    ptrs[2] = None
    assert _verify(_dims(), desc, ptrs) == L.LUMO_EINVAL
    ptrs = [ctypes.c_void_p(FAKE)] * 7
    ptrs[0] = ctypes.c_void_p(FAKE + 4)
    assert _verify(_dims(), desc, ptrs) == L.LUMO_EINVAL
    assert "aligned" in L.lumo_last_error()


def test_verify_rejects_flags_and_small_workspace():
    desc, _blob = _desc()
    assert _verify(_dims(), desc, flags=1) == L.LUMO_EINVAL
    need = L.lumo_tree_gdn_workspace_bytes(_dims(), desc.plan)
    assert need == 2 * 16 * 16 * 4
    assert _verify(_dims(), desc, ws=need - 4) == L.LUMO_ESPACE


def test_verify_rejects_null_desc_blob():
    desc, _blob = _desc()
    desc.blob = None
    assert _verify(_dims(), desc) == L.LUMO_EINVAL


def test_wy_node_states_refused():
    """The WY form keeps no per-node states: a debug dump is refused before any launch."""
    desc, _blob = _desc(policy=L.LUMO_POLICY_WY)
    P = ctypes.c_void_p
    st = L._lib.lumo_tree_gdn_verify(ctypes.byref(_dims()), ctypes.byref(desc), *([P(FAKE)] * 7), P(FAKE),
                                     P(FAKE), 0, 0, None)
    assert st == L.LUMO_EUNSUPPORTED and "node states" in L.lumo_last_error()


def _commit(d, desc, max_path=4, x=True, hist=True, channels=8, accepted=FAKE):
    P = ctypes.c_void_p
    return L._lib.lumo_gdn_commit(ctypes.byref(d), ctypes.byref(desc), max_path,
                                  P(accepted) if accepted else None, P(FAKE), P(FAKE), P(FAKE),
                                  P(FAKE), P(FAKE), P(FAKE), P(FAKE), channels,
                                  P(FAKE) if x else None, P(FAKE) if hist else None, None)


def test_commit_rejects_bad_arguments():
    desc, _blob = _desc()
    assert _commit(_dims(), desc, max_path=0) == L.LUMO_EINVAL
    assert _commit(_dims(), desc, max_path=5000) == L.LUMO_EINVAL
    assert _commit(_dims(), desc, x=True, hist=False) == L.LUMO_EINVAL
    assert _commit(_dims(), desc, channels=12) == L.LUMO_ESHAPE
    assert _commit(_dims(), desc, accepted=0) == L.LUMO_EINVAL
    assert _commit(_dims(d_k=24), desc) == L.LUMO_EUNSUPPORTED


def _commit_layers(d, desc, max_path=4, accepted=FAKE, channels=16, x=None, hist=None, n=None):
    P = ctypes.c_void_p
    n = d.n_layers if n is None else n
    xt = (P * max(n, 1))(*([P(FAKE)] * n if x is None else x))
    ht = (P * max(n, 1))(*([P(FAKE)] * n if hist is None else hist))
    return L._lib.lumo_gdn_commit_hist_layers(ctypes.byref(d), ctypes.byref(desc), max_path, P(accepted),
                                              P(FAKE), P(FAKE), channels, xt, ht, None)


def test_commit_hist_layers_rejects_bad_arguments():
    desc, _blob = _desc()
    P = ctypes.c_void_p
    assert _commit_layers(_dims(), desc, max_path=0) == L.LUMO_EINVAL
    assert _commit_layers(_dims(), desc, channels=12) == L.LUMO_ESHAPE
    assert _commit_layers(_dims(), desc, channels=0) == L.LUMO_ESHAPE
    assert _commit_layers(_dims(n_layers=129), desc) == L.LUMO_EUNSUPPORTED
    assert "128" in L.lumo_last_error()
    assert _commit_layers(_dims(), desc, accepted=0) == L.LUMO_EINVAL
    assert _commit_layers(_dims(n_layers=2), desc, hist=[P(FAKE), None]) == L.LUMO_EINVAL
    assert "conv_hist_layers[1]" in L.lumo_last_error()
    assert _commit_layers(_dims(n_layers=2), desc, hist=[P(FAKE), P(FAKE + 8)]) == L.LUMO_EINVAL
    assert _commit_layers(_dims(n_layers=3), desc, x=[P(FAKE), P(FAKE), None]) == L.LUMO_EINVAL
    assert "x_layers[2]" in L.lumo_last_error()
    d = _dims()
    assert L._lib.lumo_gdn_commit_hist_layers(ctypes.byref(d), ctypes.byref(desc), 4, P(FAKE), P(FAKE),
                                              P(FAKE), 16, None, (P * 1)(P(FAKE)), None) == L.LUMO_EINVAL
    assert L._lib.lumo_gdn_commit_hist_layers(ctypes.byref(d), ctypes.byref(desc), 4, P(FAKE), P(FAKE),
                                              P(FAKE), 16, (P * 1)(P(FAKE)), None, None) == L.LUMO_EINVAL


def test_commit_hist_layers_empty_batch_is_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), 0)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    assert _commit_layers(_dims(n_req=0, n_layers=2), desc, accepted=0, x=[None, None]) == L.LUMO_OK


def test_conv_rejects_bad_arguments():
    desc, _blob = _desc()
    P = ctypes.c_void_p
    f = L._lib.lumo_tree_conv_gather
    assert f(ctypes.byref(_dims()), ctypes.byref(desc), 12, P(FAKE), P(FAKE), P(FAKE), None, 1,
             P(FAKE), None) == L.LUMO_ESHAPE
    assert f(ctypes.byref(_dims()), ctypes.byref(desc), 16, P(FAKE), P(FAKE), P(FAKE), None, 3,
             P(FAKE), None) == L.LUMO_EINVAL
    assert f(ctypes.byref(_dims()), ctypes.byref(desc), 16, P(FAKE), None, P(FAKE), None, 1,
             P(FAKE), None) == L.LUMO_EINVAL


def _conv_pending(d, desc, pdesc, *, channels=16, act=1, max_path=4, hist=FAKE, x_prev=FAKE, path=FAKE,
                  pend_desc=True):
    P = ctypes.c_void_p
    return L._lib.lumo_tree_conv_gather_pending(
        ctypes.byref(d), ctypes.byref(desc), channels, P(FAKE), P(hist) if hist else None, P(FAKE), None, act,
        P(FAKE), ctypes.byref(pdesc) if pend_desc else None, max_path, P(path) if path else None, P(FAKE),
        P(x_prev) if x_prev else None, None)


def test_conv_pending_rejects_bad_arguments():
    desc, _b1 = _desc()
    two, _b2 = _desc(n_req=2)
    d = _dims()
    assert _conv_pending(d, desc, desc, channels=12) == L.LUMO_ESHAPE
    assert _conv_pending(d, desc, desc, act=2) == L.LUMO_EINVAL
    assert _conv_pending(d, desc, desc, max_path=0) == L.LUMO_EINVAL
    assert _conv_pending(d, desc, two) == L.LUMO_EDESC            # request counts differ
    assert _conv_pending(d, desc, desc, pend_desc=False) == L.LUMO_EINVAL
    assert _conv_pending(d, desc, desc, hist=0) == L.LUMO_EINVAL
    assert "conv_hist" in L.lumo_last_error()
    assert _conv_pending(d, desc, desc, path=0) == L.LUMO_EINVAL
    assert _conv_pending(d, desc, desc, x_prev=0) == L.LUMO_EINVAL  # the previous tree has nodes
    assert "x_prev" in L.lumo_last_error()
    assert _conv_pending(d, desc, desc, x_prev=FAKE + 2) == L.LUMO_EINVAL


def test_conv_pending_empty_batch_is_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32), np.zeros(0, np.int32), 0)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    assert _conv_pending(_dims(n_req=0), desc, desc, hist=0, path=0, x_prev=0) == L.LUMO_OK


def test_graph_create_rejects_and_null_launch():
    desc, _blob = _desc()
    h = ctypes.c_void_p()
    P = ctypes.c_void_p
    st = L._lib.lumo_gdn_commit_graph_create(ctypes.byref(_dims()), ctypes.byref(desc), None, 0, P(FAKE),
                                             P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                             P(FAKE), 0, None, None, ctypes.byref(h))
    assert st == L.LUMO_EINVAL and not h.value
    # a malformed preparation is refused before anything is captured
    bad = L.lumo_gdn_prep(8, 0.0, None, None)
    st = L._lib.lumo_gdn_commit_graph_create(ctypes.byref(_dims()), ctypes.byref(desc), ctypes.byref(bad), 4,
                                             P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                             P(FAKE), 0, None, None, ctypes.byref(h))
    assert st == L.LUMO_EINVAL and not h.value and "prep" in L.lumo_last_error()
    assert L._lib.lumo_gdn_commit_graph_launch(None, None) == L.LUMO_EINVAL
    L._lib.lumo_gdn_commit_graph_destroy(None)


def test_empty_batch_is_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), 0)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    d = _dims(n_req=0)
    assert _verify(d, desc, [None] * 7) == L.LUMO_OK
    assert _commit(d, desc, accepted=0) == L.LUMO_OK


def test_wy_rejects_paths_longer_than_32():
    """The WY policy's verification takes paths of up to 32 nodes (the matrix-core kernel
    17, the vector-ALU kernel the rest); the deferred publication keeps the 17-node
    limit of the matrix-core kernel."""
    par = trees.chain(33)
    plan, blob = L.lumo_tree_plan(np.array([0, 33], np.int32), par, np.array([33], np.int32),
                                  L.LUMO_POLICY_WY)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    for d in (_dims(h_k=1, h_v=1, d_k=128, d_v=128, op_dtype=1), _dims()):
        assert _verify(d, desc, ws=L.lumo_tree_gdn_workspace_bytes(d, plan)) == L.LUMO_EUNSUPPORTED
        assert "32" in L.lumo_last_error()
    par = trees.chain(18)
    plan, blob = L.lumo_tree_plan(np.array([0, 18], np.int32), par, np.array([18], np.int32),
                                  L.LUMO_POLICY_WY)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    dw = _dims(h_k=1, h_v=1, d_k=128, d_v=128, op_dtype=1)
    assert _pending(dw, desc, desc) == L.LUMO_EUNSUPPORTED and "17" in L.lumo_last_error()


def test_wy_needs_no_workspace():
    par = trees.FIG1_PARENT
    plan, blob = L.lumo_tree_plan(np.array([0, 7], np.int32), par, np.array([7], np.int32),
                                  L.LUMO_POLICY_WY)
    d = _dims(h_k=2, h_v=4, d_k=128, d_v=128, op_dtype=1, n_layers=3)
    assert L.lumo_tree_gdn_workspace_bytes(d, plan) == 0


def _pending(d, desc, pdesc, max_path=4, state=FAKE, pend_desc=True):
    P = ctypes.c_void_p
    return L._lib.lumo_tree_gdn_verify_pending(
        ctypes.byref(d), ctypes.byref(desc), None, P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
        P(state) if state else None, P(FAKE), ctypes.byref(pdesc) if pend_desc else None,
        max_path, P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), None)


def test_verify_pending_rejects_bad_arguments():
    dw = _dims(h_k=2, h_v=4, d_k=128, d_v=128, op_dtype=1)
    wy, _b1 = _desc(policy=L.LUMO_POLICY_WY)
    paths, _b2 = _desc(policy=L.LUMO_POLICY_PATHS)
    two, _b3 = _desc(n_req=2)
    assert _pending(dw, paths, paths) == L.LUMO_EUNSUPPORTED      # needs a WY plan
    assert _pending(_dims(), wy, paths) == L.LUMO_EUNSUPPORTED    # fp32, d = 16
    assert _pending(dw, wy, paths, max_path=0) == L.LUMO_EINVAL
    assert _pending(dw, wy, paths, max_path=5000) == L.LUMO_EINVAL
    assert _pending(dw, wy, two) == L.LUMO_EDESC                  # request counts differ
    assert _pending(dw, wy, paths, pend_desc=False) == L.LUMO_EINVAL
    assert _pending(dw, wy, paths, state=0) == L.LUMO_EINVAL
    assert "state" in L.lumo_last_error()
    assert _pending(dw, wy, paths, state=FAKE + 4) == L.LUMO_EINVAL


def test_verify_pending_empty_batch_is_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), L.LUMO_POLICY_WY)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    d = _dims(n_req=0, h_k=1, h_v=1, d_k=128, d_v=128, op_dtype=1)
    assert _pending(d, desc, desc) == L.LUMO_OK


def _pcall(d, desc, pdesc, state=FAKE, prep=None, max_path=4):
    P = ctypes.c_void_p
    return L.lumo_gdn_pending_call(ctypes.pointer(d), ctypes.pointer(desc),
                                   None if prep is None else ctypes.pointer(prep), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                   P(FAKE), P(state) if state else None, P(FAKE), ctypes.pointer(pdesc), max_path,
                                   P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE))


def _pair(a, b):
    return L._lib.lumo_tree_gdn_verify_pending_pair(None if a is None else ctypes.byref(a),
                                                    None if b is None else ctypes.byref(b), None)


def test_pending_call_layout_matches_header():
    src = os.path.join(ROOT, "_build_abi_layout.c")
    exe = os.path.join(ROOT, "_build_abi_layout")
    fields = [f for f, _ in L.lumo_gdn_pending_call._fields_]
    body = "".join(f'printf("%zu ", offsetof(lumo_gdn_pending_call, {f}));' for f in fields)
    with open(src, "w") as fh:
        fh.write("#include <stddef.h>\n#include <stdio.h>\n#include \"lumo_tree.h\"\n"
                 f"int main(void) {{ {body} printf(\"%zu\\n\", sizeof(lumo_gdn_pending_call)); return 0; }}\n")
    try:
        subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), src, "-o", exe], check=True)
        got = [int(x) for x in subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split()]
    finally:
        for f in (src, exe):
            if os.path.exists(f):
                os.remove(f)
    want = [getattr(L.lumo_gdn_pending_call, f).offset for f in fields] + [ctypes.sizeof(L.lumo_gdn_pending_call)]
    assert got == want


def test_verify_pending_pair_rejects_bad_arguments():
    dw = _dims(h_k=2, h_v=4, d_k=128, d_v=128, op_dtype=1)
    wy, _b1 = _desc(policy=L.LUMO_POLICY_WY)
    paths, _b2 = _desc(policy=L.LUMO_POLICY_PATHS)
    assert _pair(None, None) == L.LUMO_EINVAL
    assert _pair(_pcall(dw, paths, paths), None) == L.LUMO_EUNSUPPORTED  # needs a WY plan
    assert _pair(_pcall(dw, wy, paths), _pcall(dw, wy, paths, state=0)) == L.LUMO_EINVAL
    assert "state" in L.lumo_last_error()
    assert _pair(_pcall(dw, wy, paths), _pcall(dw, wy, paths, max_path=0)) == L.LUMO_EINVAL
    norm = L.lumo_gdn_prep(L.LUMO_PREP_QK_NORM, 1e-6, None, None)
    assert _pair(_pcall(dw, wy, paths), _pcall(dw, wy, paths, prep=norm)) == L.LUMO_EUNSUPPORTED
    assert "normalisation" in L.lumo_last_error()


def test_verify_pending_pair_empty_calls_are_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), L.LUMO_POLICY_WY)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    d = _dims(n_req=0, h_k=1, h_v=1, d_k=128, d_v=128, op_dtype=1)
    assert _pair(_pcall(d, desc, desc), None) == L.LUMO_OK
    assert _pair(_pcall(d, desc, desc), _pcall(d, desc, desc)) == L.LUMO_OK


def _verify_prep(d, desc, prep):
    P = ctypes.c_void_p
    return L._lib.lumo_tree_gdn_verify_prep(ctypes.byref(d), ctypes.byref(desc),
                                            ctypes.byref(prep) if prep is not None else None,
                                            *([P(FAKE)] * 7), None)


def test_prep_rejects_bad_arguments():
    dw = _dims(h_k=2, h_v=4, d_k=128, d_v=128, op_dtype=1)
    wy, _b1 = _desc(policy=L.LUMO_POLICY_WY)
    paths, _b2 = _desc(policy=L.LUMO_POLICY_PATHS)
    ok = L.lumo_gdn_prep(L.LUMO_PREP_QK_NORM, 1e-6, None, None)
    assert _verify_prep(dw, paths, ok) == L.LUMO_EUNSUPPORTED          # needs a WY plan
    assert _verify_prep(dw, wy, L.lumo_gdn_prep(4, 0.0, None, None)) == L.LUMO_EINVAL
    assert _verify_prep(dw, wy, L.lumo_gdn_prep(L.LUMO_PREP_QK_NORM, -1.0, None, None)) == L.LUMO_EINVAL
    assert _verify_prep(dw, wy, L.lumo_gdn_prep(L.LUMO_PREP_QK_NORM, float("nan"), None, None)) == L.LUMO_EINVAL
    assert _verify_prep(dw, wy, L.lumo_gdn_prep(L.LUMO_PREP_RAW_GATES, 0.0, FAKE, None)) == L.LUMO_EINVAL
    assert "a_log" in L.lumo_last_error()
    assert _verify_prep(dw, wy, L.lumo_gdn_prep(L.LUMO_PREP_RAW_GATES, 0.0, FAKE + 2, FAKE)) == L.LUMO_EINVAL
    P = ctypes.c_void_p
    bad = L.lumo_gdn_prep(8, 0.0, None, None)
    st = L._lib.lumo_gdn_commit_prep(ctypes.byref(_dims()), ctypes.byref(paths), ctypes.byref(bad), 4,
                                     P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                     P(FAKE), 0, None, None, None)
    assert st == L.LUMO_EINVAL


def test_prep_empty_batch_is_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), L.LUMO_POLICY_WY)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    d = _dims(n_req=0, h_k=1, h_v=1, d_k=128, d_v=128, op_dtype=1)
    prep = L.lumo_gdn_prep(L.LUMO_PREP_QK_NORM | L.LUMO_PREP_RAW_GATES, 1e-6, FAKE, FAKE)
    assert _verify_prep(d, desc, prep) == L.LUMO_OK


def _attn(d, desc, n_split=2, max_ctx=100, scale=0.1, ws=1 << 30, ptrs=True):
    P = ctypes.c_void_p
    f = P(FAKE) if ptrs else None
    return L._lib.lumo_tree_attention(ctypes.byref(d), ctypes.byref(desc), P(FAKE), max_ctx, scale,
                                      f, P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                      n_split, P(FAKE), ws, None)


def test_attention_rejects_bad_arguments():
    desc, _blob = _desc()
    ok = L.attn_dims(1, 4, 2)
    assert _attn(L.attn_dims(1, 6, 2), desc) == L.LUMO_EUNSUPPORTED     # group of 3
    assert _attn(L.attn_dims(1, 32, 2), desc) == L.LUMO_EUNSUPPORTED    # group of 16
    assert _attn(L.attn_dims(1, 4, 3), desc) == L.LUMO_ESHAPE           # not a multiple
    assert _attn(L.attn_dims(1, 4, 2, d=64), desc) == L.LUMO_EUNSUPPORTED
    assert _attn(L.attn_dims(2, 4, 2), desc) == L.LUMO_EDESC
    assert _attn(ok, desc, n_split=0) == L.LUMO_EINVAL
    assert _attn(ok, desc, max_ctx=-1) == L.LUMO_EINVAL
    assert _attn(ok, desc, scale=0.0) == L.LUMO_EINVAL
    assert _attn(ok, desc, scale=float("inf")) == L.LUMO_EINVAL
    assert _attn(ok, desc, ptrs=False) == L.LUMO_EINVAL
    need = L.lumo_tree_attention_workspace_bytes(ok, desc.plan, 2)
    assert need == 3 * 7 * 4 * 129 * 4
    assert _attn(ok, desc, ws=need - 4) == L.LUMO_ESPACE
    assert 1 <= L.lumo_tree_attention_splits(ok, desc.plan, 131072) <= 512


def test_attention_noalloc_refuses_on_the_host():
    """The no-allocation form refuses partial results beyond its fixed array before any
    device call (so this runs without a GPU), and validates like the workspace form."""
    desc, _blob = _desc()
    P = ctypes.c_void_p

    def call(d, n_split, scale=0.1):
        return L._lib.lumo_tree_attention_noalloc(ctypes.byref(d), ctypes.byref(desc), P(FAKE), 16, scale,
                                                  P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE), P(FAKE),
                                                  P(FAKE), n_split, None)
    big = L.attn_dims(1, 8, 8)
    assert L.lumo_tree_attention_workspace_bytes(big, desc.plan, 4096) > L.LUMO_TREE_ATTENTION_SCRATCH_BYTES
    assert call(big, 4096) == L.LUMO_ESPACE
    assert "scratch" in L.lumo_last_error()
    assert call(L.attn_dims(1, 6, 2), 2) == L.LUMO_EUNSUPPORTED
    assert call(L.attn_dims(1, 4, 2), 0) == L.LUMO_EINVAL
    assert call(L.attn_dims(1, 4, 2), 2, scale=0.0) == L.LUMO_EINVAL


def test_attention_empty_batch_is_a_no_op():
    plan, blob = L.lumo_tree_plan(np.array([0], np.int32), np.zeros(0, np.int32),
                                  np.zeros(0, np.int32), 0)
    desc = L.lumo_tree_desc(ctypes.c_void_p(FAKE), blob.ctypes.data_as(ctypes.c_void_p), plan)
    assert _attn(L.attn_dims(0, 4, 2), desc, ptrs=False) == L.LUMO_OK


def _select(rows=2, vocab=100, ld=None, dtype=0, k=3, ties=0, logits=FAKE, spine=FAKE, cand=FAKE,
            n_split=2, ws=FAKE, ws_bytes=None):
    P = ctypes.c_void_p
    if ws_bytes is None:
        ws_bytes = L.lumo_draft_select_workspace_bytes(rows, k, n_split)
    return L._lib.lumo_draft_select(rows, vocab, vocab if ld is None else ld, dtype, k, ties,
                                    P(logits) if logits else None, P(spine) if spine else None,
                                    P(cand) if cand else None, n_split, P(ws) if ws else None, ws_bytes, None)


def test_draft_select_rejects_bad_arguments():
    assert _select(rows=-1) == L.LUMO_EINVAL
    assert _select(vocab=0) == L.LUMO_EINVAL
    assert _select(ld=99) == L.LUMO_EINVAL
    assert _select(dtype=2) == L.LUMO_EUNSUPPORTED
    assert _select(ties=2) == L.LUMO_EINVAL
    assert _select(k=0) == L.LUMO_EINVAL
    assert _select(vocab=2, k=3) == L.LUMO_EINVAL
    assert _select(k=9) == L.LUMO_EUNSUPPORTED
    assert _select(n_split=0) == L.LUMO_EINVAL
    assert _select(n_split=4097) == L.LUMO_EINVAL
    assert _select(logits=None) == L.LUMO_EINVAL
    assert _select(logits=FAKE + 4) == L.LUMO_EINVAL
    assert _select(spine=None) == L.LUMO_EINVAL
    assert _select(cand=FAKE + 8) == L.LUMO_EINVAL
    assert _select(ws=None) == L.LUMO_EINVAL
    need = L.lumo_draft_select_workspace_bytes(2, 3, 2)
    assert need == 2 * 2 * 4 * 4 * 8
    assert _select(ws_bytes=need - 8) == L.LUMO_ESPACE
    assert "workspace" in L.lumo_last_error()


def test_draft_select_empty_and_single_part_need_no_workspace():
    assert _select(rows=0, logits=None, spine=None, cand=None, ws=None) == L.LUMO_OK
    assert L.lumo_draft_select_workspace_bytes(8, 3, 1) == 0
    assert L.lumo_draft_select_splits(8, 248320, 0) == 30
    assert L.lumo_draft_select_splits(64, 248320, 1) == 15
    assert L.lumo_draft_select_splits(1, 10, 1) == 1


def _fused(d, desc, pdesc=None, channels=None, act=1, ptrs=True, max_path=4):
    P = ctypes.c_void_p
    f = P(FAKE) if ptrs else None
    ch = 2 * d.h_k * d.d_k + d.h_v * d.d_v if channels is None else channels
    return L._lib.lumo_tree_gdn_verify_conv_pending(
        ctypes.byref(d), ctypes.byref(desc), None, ch, f, f, f, None, act, f, f, f, f,
        ctypes.byref(pdesc if pdesc is not None else desc), max_path, f, f, f, f, f, None)


def test_fused_conv_rejects_bad_arguments():
    wy, _b1 = _desc(policy=L.LUMO_POLICY_WY)
    paths, _b2 = _desc(policy=L.LUMO_POLICY_PATHS)
    ok = _dims(h_k=2, h_v=4, d_k=128, d_v=128, op_dtype=L.LUMO_BF16)
    # the fused conv serves two value heads per key head (one block per key-head slice of
    # the history); groups of 1, 3 and 4 are refused with a status, nothing launched
    for h_k, h_v in ((2, 2), (2, 6), (1, 4)):
        assert _fused(_dims(h_k=h_k, h_v=h_v, d_k=128, d_v=128, op_dtype=L.LUMO_BF16), wy) == L.LUMO_EUNSUPPORTED
        assert "h_v / h_k = 2 only" in L.lumo_last_error()
    assert _fused(ok, wy, channels=1000) == L.LUMO_ESHAPE
    assert _fused(ok, wy, act=2) == L.LUMO_EINVAL
    assert _fused(ok, wy, max_path=0) == L.LUMO_EINVAL
    assert _fused(ok, paths) == L.LUMO_EUNSUPPORTED  # the WY plan only
    assert _fused(ok, wy, ptrs=False) == L.LUMO_EINVAL
    assert L._lib.lumo_tree_gdn_verify_conv_pending(
        ctypes.byref(ok), ctypes.byref(wy), None, 1024, *([ctypes.c_void_p(FAKE)] * 3), None, 1,
        *([ctypes.c_void_p(FAKE)] * 4), None, 4, *([ctypes.c_void_p(FAKE)] * 5), None) == L.LUMO_EINVAL
