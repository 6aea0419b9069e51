"""The per-layer serving flow against the stacked one.

A model calls the step one layer at a time: for every layer its own conv and its own
verification (n_layers = 1, the layer's own state bank and conv history), and after
the step one commit for all layers, which derives the accepted paths and publishes
them into every layer's conv history (lumo_gdn_commit_hist_layers); each layer's state
is published by that layer's next verification. Two iterations of it must equal, bit
for bit, the same two iterations with the calls for all layers at once (the conv
publishing the pending history, the verification the pending state): the conv
outputs, the verification outputs, the state banks and, once the stacked side has
published the last paths too, the histories. Cases: the deferred-publication edge
cases (a 20-node pending path, a path into a request without nodes in the next tree,
an empty and an invalid path) on two layers, and four layers of the batched workload,
where the stacked verification runs 64-column pair blocks and the layer calls
32-column blocks.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_23900_amd as L  # noqa: E402
from paper_2609_23900_amd.step import GdnTreeStep  # noqa: E402
from lumo_synth import configs, trees  # noqa: E402
from lumo_synth import operands as ops  # noqa: E402
import pins  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _step(wl):
    return GdnTreeStep(n_req=wl.n_req, n_layers=wl.n_layers, h_k=wl.h_k, h_v=wl.h_v, d_k=wl.d_k,
                       d_v=wl.d_v, op_dtype=wl.op_dtype, node_off=wl.node_off, parent=wl.parent_flat,
                       n_rows=wl.n_rows, arrays=dict(wl.arrays), policy=L.LUMO_POLICY_WY,
                       max_path=wl.max_path, accepted=wl.accepted, channels=wl.channels)


def _split(y, hk, hv, d):
    """A conv output [..., rows, q | k | v] as contiguous q, k, v tensors."""
    lead = y.shape[:-1]
    q = y[..., :hk * d].reshape(*lead, hk, d).contiguous()
    k = y[..., hk * d:2 * hk * d].reshape(*lead, hk, d).contiguous()
    v = y[..., 2 * hk * d:].reshape(*lead, hv, d).contiguous()
    return q, k, v


def _edge_workloads():
    """Two iterations over five requests: the first one's accepted paths are a 20-node
    chain, a path into a request that has no nodes in the second tree, none, an invalid
    node, and a deep path of a random tree."""
    rng = np.random.default_rng(61)
    prev_par = [trees.chain(20), np.array([-1, 0, 0, 1], np.int32), np.array([-1], np.int32),
                trees.FIG1_PARENT, trees.random_tree(rng, 40, 8, trees.bmax_uniform(3))]
    cur_par = [trees.random_tree(rng, 30, 8, trees.bmax_uniform(3)), np.zeros(0, np.int32),
               trees.chain(5), np.zeros(0, np.int32), trees.random_tree(rng, 50, 9, trees.bmax_uniform(4))]
    h_k, h_v = 2, 4
    C = 2 * h_k * 128 + h_v * 128
    wls = []
    for par, n_rows, s in ((prev_par, [20, 5, 1, 9, 40], 71), (cur_par, [31, 2, 5, 0, 50], 72)):
        wl = pins.make_wl(par, d_k=128, d_v=128, h_k=h_k, h_v=h_v, op_dtype=ops.BF16, n_rows=n_rows,
                          n_layers=2, max_path=24)
        wl.channels = C
        wl.arrays = ops.make_gdn_operands(s, n_req=5, n_layers=2, total_rows=wl.total_rows, h_k=h_k, h_v=h_v,
                                          d_k=128, d_v=128, op_dtype=ops.BF16)
        wl.arrays.update(ops.make_conv_operands(s, n_req=5, n_layers=2, total_rows=wl.total_rows, channels=C,
                                                op_dtype=ops.BF16))
        wls.append(wl)
    prev, cur = wls
    cur.arrays["w"] = prev.arrays["w"]  # the layers' conv taps
    cur.arrays["hist"] = prev.arrays["hist"]
    cur.arrays["state0"] = prev.arrays["state0"]
    deep = int(np.argmax(trees.depths(prev_par[4])))
    prev.accepted = np.array([19, 3, -1, 99, deep], np.int32)
    cur.accepted = np.array([25, -1, 4, -1, 49], np.int32)
    return [prev, cur]


def _stacked(wls):
    """The first iteration's conv and commit (its tree is only convolved: the 20-node
    chain of the edge cases is beyond the WY form), then the second iteration with the
    calls for all layers; then the last paths' history publication, so that the
    histories compare at the same point."""
    sp, sc = (_step(w) for w in wls)
    d = sp.dims
    sc.hist = sp.hist
    state = sp.state
    sp.conv()
    sp.t["q"], sp.t["k"], sp.t["v"] = _split(sp.y, d.h_k, d.h_v, d.d_k)  # the pending keys and values
    sp.commit(defer=True, with_conv=False)  # the accepted paths only
    sc.conv_pending(sp)
    q, k, v = _split(sc.y, d.h_k, d.h_v, d.d_k)
    L.lumo_tree_gdn_verify_pending(d, sc.desc, q, k, v, sc.t["g"], sc.t["beta"], state, sc.o, sp.desc,
                                   sp.max_path, sp.path_out, sp.path_len, sp.t["k"], sp.t["v"], sp.t["g"],
                                   sp.t["beta"])
    sc.commit(defer=True, with_conv=False)
    L.lumo_gdn_commit(sc.dims, sc.desc, sc.max_path, sc.accepted, sc.path_out, sc.path_len,
                      None, None, None, None, None, sc.channels, sc.x, sc.hist)
    torch.cuda.synchronize()
    return dict(y=[sp.y, sc.y], o=sc.o, state=state, hist=sc.hist, path_len=[sp.path_len, sc.path_len])


def _layers(wls):
    """The same two iterations with one conv and one verification call per layer, each
    layer's state bank and history its own buffer, and one commit for all layers after
    each iteration."""
    sp, sc = (_step(w) for w in wls)
    d = sp.dims
    nl = d.n_layers
    d1 = L.dims(d.n_req, 1, d.h_k, d.h_v, d.d_k, d.d_v, d.op_dtype)
    states = [sp.state[:, l:l + 1].contiguous() for l in range(nl)]
    hists = [sp.hist[:, l:l + 1].contiguous() for l in range(nl)]
    for l in range(nl):
        L.lumo_tree_conv_gather(d1, sp.desc, sp.channels, sp.x[l], hists[l], sp.w[l], None, sp.act, sp.y[l])
    sp.t["q"], sp.t["k"], sp.t["v"] = _split(sp.y, d.h_k, d.h_v, d.d_k)
    L.lumo_gdn_commit_hist_layers(d, sp.desc, sp.max_path, sp.accepted, sp.path_out, sp.path_len, sp.channels,
                                  [sp.x[l] for l in range(nl)], hists)
    for l in range(nl):
        L.lumo_tree_conv_gather(d1, sc.desc, sc.channels, sc.x[l], hists[l], sc.w[l], None, sc.act, sc.y[l])
        q, k, v = _split(sc.y[l], d.h_k, d.h_v, d.d_k)
        L.lumo_tree_gdn_verify_pending(d1, sc.desc, q, k, v, sc.t["g"][l], sc.t["beta"][l], states[l], sc.o[l],
                                       sp.desc, sp.max_path, sp.path_out, sp.path_len, sp.t["k"][l],
                                       sp.t["v"][l], sp.t["g"][l], sp.t["beta"][l])
    L.lumo_gdn_commit_hist_layers(d, sc.desc, sc.max_path, sc.accepted, sc.path_out, sc.path_len, sc.channels,
                                  [sc.x[l] for l in range(nl)], hists)
    torch.cuda.synchronize()
    return dict(y=[sp.y, sc.y], o=sc.o, state=torch.cat(states, dim=1), hist=torch.cat(hists, dim=1),
                path_len=[sp.path_len, sc.path_len])


def _assert_same(a, b, what):
    for it in range(2):
        assert torch.equal(a["y"][it].view(torch.int16), b["y"][it].view(torch.int16)), (what, "y", it)
        assert torch.equal(a["path_len"][it], b["path_len"][it]), (what, "path_len", it)
    assert torch.equal(a["o"].view(torch.int16), b["o"].view(torch.int16)), (what, "o")
    assert torch.equal(a["state"], b["state"]), (what, "state", int((a["state"] != b["state"]).sum()))
    assert torch.equal(a["hist"].view(torch.int16), b["hist"].view(torch.int16)), (what, "hist")


def test_per_layer_flow_edge_cases():
    wls = _edge_workloads()
    say("[gpu] per-layer flow, edge cases")
    a, b = _stacked(wls), _layers(wls)
    assert a["path_len"][0].cpu().numpy().tolist() == [20, 3, 0, -1, int(trees.depths(wls[0].parents[4]).max()) + 1]
    assert not torch.equal(a["state"], torch.from_numpy(wls[0].arrays["state0"]).cuda())
    _assert_same(a, b, "edge cases")


def test_per_layer_flow_batched():
    wl = configs.build("batched", n_layers=4)
    d = wl
    assert d.n_req * d.n_layers * d.h_k >= 256 > d.n_req * d.h_k  # 64-column stacked, 32-column per layer
    say("[gpu] per-layer flow, batched workload, 4 layers")
    a, b = _stacked([wl, wl]), _layers([wl, wl])
    assert int((a["path_len"][0] > 0).sum()) > 0
    _assert_same(a, b, "batched")


def _empty_desc(n_req):
    """A batch of n_req requests without nodes (WY plan): nothing to verify, or nothing
    pending."""
    return L.TreeDesc.build(np.zeros(n_req + 1, np.int32), np.zeros(0, np.int32), np.ones(n_req, np.int32),
                            L.LUMO_POLICY_WY)


def _pair_layers(wls):
    """_layers with the layer calls paired: layer l's verification (nothing pending for
    l >= 1) and, in the same launch, the publication of the pending path into layer
    l + 1's state bank (lumo_tree_gdn_verify_pending_pair)."""
    sp, sc = (_step(w) for w in wls)
    d = sp.dims
    nl = d.n_layers
    d1 = L.dims(d.n_req, 1, d.h_k, d.h_v, d.d_k, d.d_v, d.op_dtype)
    empty = _empty_desc(d.n_req)
    states = [sp.state[:, l:l + 1].contiguous() for l in range(nl)]
    hists = [sp.hist[:, l:l + 1].contiguous() for l in range(nl)]
    for l in range(nl):
        L.lumo_tree_conv_gather(d1, sp.desc, sp.channels, sp.x[l], hists[l], sp.w[l], None, sp.act, sp.y[l])
    sp.t["q"], sp.t["k"], sp.t["v"] = _split(sp.y, d.h_k, d.h_v, d.d_k)
    L.lumo_gdn_commit_hist_layers(d, sp.desc, sp.max_path, sp.accepted, sp.path_out, sp.path_len, sp.channels,
                                  [sp.x[l] for l in range(nl)], hists)

    def publish(l):  # the pending path into layer l's bank, nothing to verify
        return L.pending_call(d1, empty, None, None, None, None, None, states[l], None, sp.desc, sp.max_path,
                              sp.path_out, sp.path_len, sp.t["k"][l], sp.t["v"][l], sp.t["g"][l], sp.t["beta"][l])

    for l in range(nl):
        L.lumo_tree_conv_gather(d1, sc.desc, sc.channels, sc.x[l], hists[l], sc.w[l], None, sc.act, sc.y[l])
        q, k, v = _split(sc.y[l], d.h_k, d.h_v, d.d_k)
        pend = sp.desc if l == 0 else empty  # layer 0 publishes its own path
        a = L.pending_call(d1, sc.desc, q, k, v, sc.t["g"][l], sc.t["beta"][l], states[l], sc.o[l], pend,
                           sp.max_path, sp.path_out, sp.path_len, sp.t["k"][l], sp.t["v"][l], sp.t["g"][l],
                           sp.t["beta"][l])
        L.lumo_tree_gdn_verify_pending_pair(a, publish(l + 1) if l + 1 < nl else None)
    L.lumo_gdn_commit_hist_layers(d, sc.desc, sc.max_path, sc.accepted, sc.path_out, sc.path_len, sc.channels,
                                  [sc.x[l] for l in range(nl)], hists)
    torch.cuda.synchronize()
    return dict(y=[sp.y, sc.y], o=sc.o, state=torch.cat(states, dim=1), hist=torch.cat(hists, dim=1),
                path_len=[sp.path_len, sc.path_len])


@pytest.mark.parametrize("case", ["edge", "batched"])
def test_paired_layer_calls_flow(case):
    """The per-layer flow with each layer's verification paired with the publication
    of the next layer's state in one launch: bit for bit the stacked flow."""
    wls = _edge_workloads() if case == "edge" else [configs.build("batched", n_layers=4)] * 2
    say(f"[gpu] paired layer calls, {case}")
    a, b = _stacked(wls), _pair_layers(wls)
    _assert_same(a, b, case)


def test_verify_pending_pair_equals_two_calls():
    """lumo_tree_gdn_verify_pending_pair against the same two calls made one after the
    other: a verification that publishes its pending path with the publication of that
    path into another bank; a verification with nothing pending with a publication; a
    call alone. Outputs and every state bank bit for bit; 16-level trees (the depth-16
    instance) and the batched trees (depth 8)."""
    for name, over in (("batched", dict(n_layers=2)), ("widedeep", dict(n_req=4, n_layers=2))):
        wl = configs.build(name, with_conv=False, **over)
        st = GdnTreeStep.from_workload(wl, policy=L.LUMO_POLICY_WY, with_conv=False)
        d = st.dims
        d1 = L.dims(d.n_req, 1, d.h_k, d.h_v, d.d_k, d.d_v, d.op_dtype)
        empty = _empty_desc(d.n_req)
        st.commit(defer=True)
        torch.cuda.synchronize()
        assert int((st.path_len > 0).sum()) > 0
        say(f"[gpu] verify_pending_pair {name}")
        t = {key: [st.t[key][l] for l in range(2)] for key in ("q", "k", "v", "g", "beta")}

        def call(l, state, o, tree, pend, use):
            args = (t["q"][l], t["k"][l], t["v"][l], t["g"][l], t["beta"][l]) if tree is st.desc else (None,) * 5
            return dict(args=(d1, tree) + args + (state, o if tree is st.desc else None, pend, st.max_path,
                                                   st.path_out, st.path_len, t["k"][l], t["v"][l], t["g"][l],
                                                   t["beta"][l]), use=use)

        for pend_a, with_b in ((st.desc, True), (empty, True), (st.desc, False)):
            res = []
            for paired in (False, True):
                banks = [st.state0[:, l:l + 1].contiguous() for l in range(2)]
                o = torch.zeros_like(st.o[0])
                ca = call(0, banks[0], o, st.desc, pend_a, True)
                cb = call(1, banks[1], None, empty, st.desc, with_b)
                if paired:
                    L.lumo_tree_gdn_verify_pending_pair(L.pending_call(*ca["args"]),
                                                        L.pending_call(*cb["args"]) if with_b else None)
                else:
                    L.lumo_tree_gdn_verify_pending(*ca["args"])
                    if with_b:
                        L.lumo_tree_gdn_verify_pending(*cb["args"])
                torch.cuda.synchronize()
                res.append((o.clone(), banks[0].clone(), banks[1].clone()))
            (o1, s1, u1), (o2, s2, u2) = res
            assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)), (name, with_b)
            assert torch.equal(s1, s2) and torch.equal(u1, u2), (name, with_b)
            assert with_b == (not torch.equal(u2, st.state0[:, 1:2])), (name, with_b)  # published, or untouched
