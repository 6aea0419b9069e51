"""Recurrent agreement under paired error bounds (Sec. VII-D, Eq. (7), Tab. V; the same
rule as Eq. (6) of Sec. VII-C).

The paper qualifies a verification method against a sequential GPU recurrence: for
every cell (recurrent instance, output node or publication, value head), with errors
measured against the float64 recurrence and reduced over the cell's vector (output)
or matrix (state) entries, both the root-mean-square and the maximum absolute error
must satisfy
    E_method <= 1.10 E_seq + 2^-24 M_64 + 2^-149,
M_64 being the same reduction of the float64 reference. Method: the WY verification
and the deferred publication; sequential comparator: the sequential path scan and the
eager replay.

  * the paper's configuration: the 28-node draft geometry, 48 recurrent instances
    (layers) x 48 value heads, bf16 operands and outputs; 64,512 output cells;
    publications of 1, 6 and 11 updates from a fresh state, 6,912 state cells;
  * the benchmark's launch configuration on the batched workload (the depth-8 WY
    instance, two value heads per block): the previous iteration's accepted paths
    published inside the verification, every node of every request and head on 12 of
    the 48 layers (196,608 output cells, 3,072 state cells);
  * the depth-16 instance on widedeep and chainmix (every cell of the one layer);
  * the tree conv fused into the verification, with the queries and keys normalised
    and the gates taken from raw inputs in the kernel (the benchmark's fused step),
    against the conv kernel followed by the prepared sequential scan; the float64
    recurrence reads the conv kernel's outputs (the conv itself is held to the oracle
    by the parity tests, and the fused kernel equals the two kernels bit for bit).
The reference of the outputs after a publication starts from the float64 published
state rounded once to fp32 (a 2^-24 relative perturbation, inside the rule's slack).
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
import gpu_util as gu  # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def cells_outside(method, seq, ref):
    """Cells (all axes but the last) where the RMS or the max-abs bound fails."""
    em, es = method - ref, seq - ref

    def rms(x):
        return np.sqrt(np.mean(x * x, axis=-1))

    def mx(x):
        return np.max(np.abs(x), axis=-1)

    bad_rms = rms(em) > 1.10 * rms(es) + 2.0 ** -24 * rms(ref) + 2.0 ** -149
    bad_max = mx(em) > 1.10 * mx(es) + 2.0 ** -24 * mx(ref) + 2.0 ** -149
    return int(np.sum(bad_rms | bad_max)), bad_rms.size


@pytest.fixture(scope="module")
def wl():
    return configs.build("paper28", with_conv=False, n_layers=48, h_k=16, h_v=48)


def _step(wl, policy):
    return GdnTreeStep.from_workload(wl, policy=policy, with_conv=False)


def test_paired_bounds_outputs(wl):
    say("[gpu] paired bounds: outputs")
    swy, sseq = _step(wl, L.LUMO_POLICY_WY), _step(wl, L.LUMO_POLICY_PATHS)
    swy.verify()
    sseq.verify()
    torch.cuda.synchronize()
    rows = oracle.plan.flat_rows(wl.parents, wl.row_off)
    o_wy = gu.to_np(swy.o)[:, rows].astype(np.float64)
    o_seq = gu.to_np(sseq.o)[:, rows].astype(np.float64)
    o_ref = oracle.verify_all(wl)[:, rows]
    assert not np.array_equal(o_wy, o_seq)  # distinct arithmetic, so the comparison means something
    bad, total = cells_outside(o_wy, o_seq, o_ref)
    say(f"  output cells outside the paired bounds: {bad} of {total}")
    assert total == 48 * 28 * 48
    assert bad == 0
    # the bound has teeth: a perturbation of a quarter of a bf16 step fails many cells
    noisy = o_wy + 2.0 ** -10 * np.abs(o_wy) * np.where(o_wy >= o_ref, 1.0, -1.0)
    assert cells_outside(noisy, o_seq, o_ref)[0] > total // 10


def test_paired_bounds_publications(wl):
    say("[gpu] paired bounds: publications of 1, 6, 11 updates")
    depth = trees.depths(wl.parents[0])
    bad_all, total_all = 0, 0
    for n_upd in (1, 6, 11):
        acc = np.array([int(np.where(depth == n_upd - 1)[0][0])], np.int32)
        eager = _step(wl, L.LUMO_POLICY_PATHS)
        eager.accepted.copy_(torch.from_numpy(acc))
        eager.commit()
        dfr = _step(wl, L.LUMO_POLICY_WY)
        dfr.accepted.copy_(torch.from_numpy(acc))
        dfr.commit(defer=True)
        dfr.verify_pending(dfr)
        torch.cuda.synchronize()
        ref, _, pl = oracle.commit(wl, accepted=acc)
        assert pl[0] == n_upd
        shape = (wl.n_layers, wl.h_v, -1)
        s_seq = eager.state.cpu().numpy()[0].reshape(shape).astype(np.float64)
        s_m = dfr.state.cpu().numpy()[0].reshape(shape).astype(np.float64)
        bad, total = cells_outside(s_m, s_seq, ref[0].reshape(shape))
        say(f"  {n_upd} updates: state cells outside {bad} of {total}")
        bad_all += bad
        total_all += total
    assert total_all == 6912
    assert bad_all == 0


# ---------------------------------------------------------------- the benchmark's workloads

_LAYERS = {"batched": list(range(0, 48, 4)), "widedeep": [0], "chainmix": [0]}


def _sliced(wl, layers, arrays):
    """A copy of the workload restricted to the given layers (operands and states)."""
    import copy
    w2 = copy.copy(wl)
    w2.n_layers = len(layers)
    a = {}
    for key in ("q", "k", "v", "g", "beta"):
        a[key] = np.ascontiguousarray(arrays[key][layers])
    a["state0"] = np.ascontiguousarray(arrays["state0"][:, layers])
    w2.arrays = a
    return w2


@pytest.mark.parametrize("name", ["batched", "widedeep", "chainmix"])
def test_paired_bounds_benchmark_step(name):
    say(f"[gpu] paired bounds: {name}, deferred publication + WY verification vs eager replay + scan")
    wl = configs.build(name, with_conv=False)
    layers = _LAYERS[name]
    m = _step(wl, L.LUMO_POLICY_WY)
    m.commit(defer=True)  # derives the accepted paths
    m.verify_pending(m)   # publishes them into the state bank, then verifies from it
    c = _step(wl, L.LUMO_POLICY_PATHS)
    c.commit()            # eager replay into the state bank
    c.verify()            # sequential scans from the published state
    torch.cuda.synchronize()
    # float64: publication, then the recurrence from the published state
    ref_state, _, _ = oracle.commit(wl)
    arrays = dict(wl.arrays)
    arrays["state0"] = ref_state.astype(np.float32)
    ws = _sliced(wl, layers, arrays)
    rows = oracle.plan.flat_rows(wl.parents, wl.row_off)
    o_ref = oracle.verify_all(ws)[:, rows]
    o_m = gu.to_np(m.o)[layers][:, rows].astype(np.float64)
    o_c = gu.to_np(c.o)[layers][:, rows].astype(np.float64)
    assert not np.array_equal(o_m, o_c)
    bad_o, tot_o = cells_outside(o_m, o_c, o_ref)
    shape = (wl.n_req, len(layers), wl.h_v, -1)
    s_m = m.state.cpu().numpy()[:, layers].reshape(shape).astype(np.float64)
    s_c = c.state.cpu().numpy()[:, layers].reshape(shape).astype(np.float64)
    s_r = ref_state[:, layers].reshape(shape)
    published = np.array([wl.accepted[r] >= 0 for r in range(wl.n_req)])
    bad_s, tot_s = cells_outside(s_m[published], s_c[published], s_r[published])
    say(f"  output cells outside {bad_o} of {tot_o}; state cells outside {bad_s} of {tot_s}")
    assert tot_o == len(layers) * wl.total_nodes * wl.h_v
    assert bad_o == 0 and bad_s == 0


def test_paired_bounds_fused_conv():
    say("[gpu] paired bounds: fused conv + prepared WY vs conv + prepared sequential scan")
    wl = configs.build("batched")
    layers = _LAYERS["batched"]
    rng = np.random.default_rng(5)
    a_log = (0.5 * rng.standard_normal((wl.n_layers, wl.h_v))).astype(np.float32)
    dt_bias = rng.standard_normal((wl.n_layers, wl.h_v)).astype(np.float32)
    flags = L.LUMO_PREP_QK_NORM | L.LUMO_PREP_RAW_GATES
    gprep = L.Prep(flags, 1e-6, torch.from_numpy(a_log).cuda(), torch.from_numpy(dt_bias).cuda())
    a = dict(wl.arrays)
    a["g"] = rng.standard_normal(a["g"].shape).astype(np.float32)      # raw gate inputs
    a["beta"] = rng.standard_normal(a["beta"].shape).astype(np.float32)
    acc = np.full(wl.n_req, -1, np.int32)  # nothing pending: this iteration's verification alone

    def step(policy):
        return GdnTreeStep(n_req=wl.n_req, n_layers=wl.n_layers, h_k=wl.h_k, h_v=wl.h_v, d_k=wl.d_k,
                           d_v=wl.d_v, op_dtype=wl.op_dtype, node_off=wl.node_off, parent=wl.parent_flat,
                           n_rows=wl.n_rows, arrays=a, policy=policy, max_path=wl.max_path, accepted=acc,
                           channels=wl.channels, prep=gprep)
    m = step(L.LUMO_POLICY_WY)
    m.commit(defer=True, with_conv=False)
    m.verify_conv_pending(m)
    c = step(L.LUMO_POLICY_RECOMPUTE)
    c.conv()
    hk, d = wl.h_k, wl.d_k
    y = c.y
    c.t["q"] = y[..., :hk * d].reshape(wl.n_layers, -1, hk, d).contiguous()
    c.t["k"] = y[..., hk * d:2 * hk * d].reshape(wl.n_layers, -1, hk, d).contiguous()
    c.t["v"] = y[..., 2 * hk * d:].reshape(wl.n_layers, -1, wl.h_v, d).contiguous()
    c.verify()
    torch.cuda.synchronize()
    assert np.array_equal(m.path_len.cpu().numpy(), np.zeros(wl.n_req, np.int32))
    bits = {key: c.t[key].view(torch.int16).cpu().numpy().view(np.uint16) for key in ("q", "k", "v")}
    ra = dict(bits, g=a["g"], beta=a["beta"], state0=a["state0"])
    ws = _sliced(wl, layers, ra)
    oprep = oracle.Prep(flags, 1e-6, a_log[layers], dt_bias[layers])
    rows = oracle.plan.flat_rows(wl.parents, wl.row_off)
    o_ref = oracle.verify_all(ws, prep=oprep)[:, rows]
    o_m = gu.to_np(m.o)[layers][:, rows].astype(np.float64)
    o_c = gu.to_np(c.o)[layers][:, rows].astype(np.float64)
    assert not np.array_equal(o_m, o_c)
    bad, total = cells_outside(o_m, o_c, o_ref)
    say(f"  output cells outside {bad} of {total}")
    assert total == len(layers) * wl.total_nodes * wl.h_v
    assert bad == 0
