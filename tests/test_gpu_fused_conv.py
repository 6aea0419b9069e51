"""The tree conv fused into the WY verification (lumo_tree_gdn_verify_conv_pending).

The fused call must equal, bit for bit, the two calls it replaces: the conv with the
pending history publication (lumo_tree_conv_gather_pending) followed by the
verification with the pending state publication (lumo_tree_gdn_verify_pending) on the
conv output split into queries, keys and values, the pending path's keys and values
being the previous iteration's conv output. Outputs, the published state bank and the
published history are compared for an iteration that publishes the previous one's
accepted paths (a 20-node path staged in two rounds, a path into a request with no
nodes in this tree, an empty and an invalid path), and over two iterations of the
benchmark's serving loop (nothing pending, then the first iteration's paths) on the
full batched workload and a 16-level one (chainmix); also with operand preparation, with a
conv bias with and without the SiLU, and against the oracle directly (conv then
verification) on the one-layer workload.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle  # noqa: E402
import paper_2609_23900_amd as L  # noqa: E402
from paper_2609_23900_amd.step import GdnTreeStep  # noqa: E402
from lumo_synth import configs, trees  # noqa: E402
from lumo_synth import operands as ops  # noqa: E402
import gpu_util as gu  # noqa: E402
import pins  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _step(wl, arrays=None, prep=None, act=1):
    a = dict(wl.arrays if arrays is None else arrays)
    return GdnTreeStep(n_req=wl.n_req, n_layers=wl.n_layers, h_k=wl.h_k, h_v=wl.h_v, d_k=wl.d_k,
                       d_v=wl.d_v, op_dtype=wl.op_dtype, node_off=wl.node_off, parent=wl.parent_flat,
                       n_rows=wl.n_rows, arrays=a, policy=L.LUMO_POLICY_WY, max_path=wl.max_path,
                       accepted=wl.accepted, channels=wl.channels, prep=prep, act=act)


def _split(st):
    """The conv output y [layers][rows][q | k | v] as contiguous q, k, v tensors."""
    n_layers, rows, _ = st.y.shape
    hk, hv, d = st.dims.h_k, st.dims.h_v, st.dims.d_k
    q = st.y[..., :hk * d].reshape(n_layers, rows, hk, d).contiguous()
    k = st.y[..., hk * d:2 * hk * d].reshape(n_layers, rows, hk, d).contiguous()
    v = st.y[..., 2 * hk * d:].reshape(n_layers, rows, hv, d).contiguous()
    return q, k, v


def _pair(h_k=2, h_v=4, seed=41):
    """Two iterations over the same 5 requests (the deferred-publication edge cases)."""
    rng = np.random.default_rng(seed)
    prev_par = [trees.chain(20), np.array([-1, 0, 0, 1], np.int32), np.array([-1], np.int32),
                trees.FIG1_PARENT, trees.random_tree(rng, 40, 8, trees.bmax_uniform(3))]
    cur_par = [trees.random_tree(rng, 30, 8, trees.bmax_uniform(3)), np.zeros(0, np.int32),
               trees.chain(5), np.zeros(0, np.int32),
               trees.random_tree(rng, 50, 9, trees.bmax_uniform(4))]
    C = 2 * h_k * 128 + h_v * 128
    wls = []
    for par, n_rows, mp, s in ((prev_par, [20, 5, 1, 9, 40], 24, seed), (cur_par, [31, 2, 5, 0, 50], 16, seed + 1)):
        wl = pins.make_wl(par, d_k=128, d_v=128, h_k=h_k, h_v=h_v, op_dtype=ops.BF16, n_rows=n_rows,
                          n_layers=2, max_path=mp)
        wl.channels = C
        wl.arrays = ops.make_gdn_operands(s, n_req=5, n_layers=2, total_rows=wl.total_rows, h_k=h_k, h_v=h_v,
                                          d_k=128, d_v=128, op_dtype=ops.BF16)
        wl.arrays.update(ops.make_conv_operands(s, n_req=5, n_layers=2, total_rows=wl.total_rows, channels=C,
                                                op_dtype=ops.BF16))
        wls.append(wl)
    prev, cur = wls
    # the conv taps are the layer's weights: the same in both iterations
    cur.arrays["w"] = prev.arrays["w"]
    if prev.arrays.get("bias") is not None:
        cur.arrays["bias"] = prev.arrays["bias"]
    deep = int(np.argmax(trees.depths(prev_par[4])))
    prev.accepted = np.array([19, 3, -1, 99, deep], np.int32)
    cur.accepted = np.array([-1] * 5, np.int32)
    return prev, cur


def _two_iterations(prev, cur, prep=None, act=1):
    """(fused, unfused) results of the second iteration: cur publishing prev's accepted
    paths (prev itself is only planned and its paths derived: its 20-node chain is beyond
    the WY form). Each side carries its own history and state bank."""
    out = {}
    for side in ("fused", "split"):
        sp = _step(prev, prep=prep, act=act)
        sc = _step(cur, prep=prep, act=act)
        sc.hist = sp.hist  # one history and one state bank across the iterations
        sp.commit(defer=True, with_conv=False)  # derives the accepted paths only
        if side == "fused":
            sc.verify_conv_pending(sp, state=sp.state)
        else:
            sp.conv()  # the previous iteration's conv output: the pending keys and values
            sp.t["q"], sp.t["k"], sp.t["v"] = _split(sp)
            sc.conv_pending(sp)
            sc.t["q"], sc.t["k"], sc.t["v"] = _split(sc)
            sc.verify_pending(sp, state=sp.state)
        torch.cuda.synchronize()
        out[side] = dict(o=sc.o.clone(), state=sp.state.clone(), hist=sp.hist.clone(),
                         path_len=sp.path_len.cpu().numpy())
    return out["fused"], out["split"]


def _assert_equal(a, b, what):
    for key in ("o", "state", "hist"):
        x, y = a[key], b[key]
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y), (what, key, int((x != y).sum()))


def test_fused_equals_conv_then_verify_edge_cases():
    prev, cur = _pair()
    say("[gpu] fused conv pending pair")
    fused, split = _two_iterations(prev, cur)
    pl = fused["path_len"]
    assert pl.tolist()[:4] == [20, 3, 0, -1], pl
    _assert_equal(fused, split, "pending pair")
    # the publications happened: history and state of request 0 changed
    sp0 = _step(prev)
    assert not torch.equal(fused["hist"][0], sp0.hist[0])
    assert not torch.equal(fused["state"][0], sp0.state0[0])
    # nothing pending for request 2 (empty path), request 3 (invalid path): untouched
    for r in (2, 3):
        assert torch.equal(fused["hist"][r].view(torch.int16), sp0.hist[r].view(torch.int16)), r
        assert torch.equal(fused["state"][r], sp0.state0[r]), r


def test_fused_with_operand_preparation():
    prev, cur = _pair(seed=53)
    rng = np.random.default_rng(5)
    a_log = torch.from_numpy((0.5 * rng.standard_normal((2, 4))).astype(np.float32)).cuda()
    dt_bias = torch.from_numpy(rng.standard_normal((2, 4)).astype(np.float32)).cuda()
    prep = L.Prep(L.LUMO_PREP_QK_NORM | L.LUMO_PREP_RAW_GATES, 1e-6, a_log, dt_bias)
    say("[gpu] fused conv pending, prepared operands")
    fused, split = _two_iterations(prev, cur, prep)
    _assert_equal(fused, split, "prep")


@pytest.mark.parametrize("act", [0, 1])
def test_fused_with_bias_and_activation(act):
    """A conv bias (per layer and channel, shared by the iterations) with and without the
    SiLU: the fused walk and the pending path's conv add the bias first and apply the
    activation only when asked, as the conv kernels do."""
    prev, cur = _pair(seed=67)
    rng = np.random.default_rng(67 + act)
    C = prev.channels
    bias = (0.5 * rng.standard_normal((2, C))).astype(np.float32)
    prev.arrays["bias"] = bias
    cur.arrays["bias"] = bias
    a_log = torch.from_numpy((0.5 * rng.standard_normal((2, 4))).astype(np.float32)).cuda()
    dt_bias = torch.from_numpy(rng.standard_normal((2, 4)).astype(np.float32)).cuda()
    prep = L.Prep(L.LUMO_PREP_QK_NORM | L.LUMO_PREP_RAW_GATES, 1e-6, a_log, dt_bias)
    say(f"[gpu] fused conv pending, bias, act={act}")
    fused, split = _two_iterations(prev, cur, prep, act=act)
    _assert_equal(fused, split, f"bias act={act}")
    # the bias and the activation are observable: without them the outputs differ
    if act == 1:
        prev.arrays["bias"] = None
        cur.arrays["bias"] = None
        plain, _ = _two_iterations(prev, cur, prep, act=act)
        assert not torch.equal(plain["o"].view(torch.int16), fused["o"].view(torch.int16))
    else:
        silu, _ = _two_iterations(prev, cur, prep, act=1)
        assert not torch.equal(silu["o"].view(torch.int16), fused["o"].view(torch.int16))


@pytest.mark.parametrize("name", ["batched", "chainmix"])
def test_fused_full_size_bitwise(name):
    """The benchmark's serving loop, two iterations over the same tree: fused against
    the two calls, every output, state and history entry."""
    wl = configs.build(name)
    say(f"[gpu] fused conv pending {name}")
    res = {}
    for side in ("fused", "split"):
        st = _step(wl)
        for it in range(2):
            if side == "fused":
                st.verify_conv_pending(st)
            else:
                kv = (st.t["k"], st.t["v"])
                st.conv_pending(st)
                q, k, v = _split(st)
                if it == 0:
                    st.t["q"], st.t["k"], st.t["v"] = q, k, v
                    st.verify_pending(st)
                else:  # the pending path's keys and values are the previous conv output
                    st.t["k"], st.t["v"] = kv
                    L.lumo_tree_gdn_verify_pending(st.dims, st.desc, q, k, v, st.t["g"], st.t["beta"], st.state,
                                                   st.o, st.desc, st.max_path, st.path_out, st.path_len,
                                                   kv[0], kv[1], st.t["g"], st.t["beta"])
                    st.t["q"], st.t["k"], st.t["v"] = q, k, v
            st.commit(defer=True, with_conv=False)
        torch.cuda.synchronize()
        res[side] = dict(o=st.o, state=st.state, hist=st.hist)
    _assert_equal(res["fused"], res["split"], name)


def test_fused_against_oracle_layer1():
    """Independently of the other kernels: the fused outputs of one iteration against
    the oracle's conv (rounded to bf16) then verification."""
    wl = configs.build("layer1")
    st = _step(wl)
    st.verify_conv_pending(st)
    torch.cuda.synchronize()
    y = oracle.conv_all(wl)  # [layers][rows][C] fp64
    yb = ops.to_bf16_bits(y.astype(np.float32))
    n_layers, rows, _ = yb.shape
    hk, hv, d = wl.h_k, wl.h_v, wl.d_k
    arrays = dict(wl.arrays)
    arrays["q"] = np.ascontiguousarray(yb[..., :hk * d].reshape(n_layers, rows, hk, d))
    arrays["k"] = np.ascontiguousarray(yb[..., hk * d:2 * hk * d].reshape(n_layers, rows, hk, d))
    arrays["v"] = np.ascontiguousarray(yb[..., 2 * hk * d:].reshape(n_layers, rows, hv, d))
    inst = [(0, 0, h) for h in range(hv)]
    worst = gu.check_outputs(wl, gu.to_np(st.o), inst, arrays=arrays)
    say(f"  layer1 fused worst max-rel {worst:.3e}")
