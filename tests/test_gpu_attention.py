"""GPU parity of tree attention (lumo_tree_attention) against the fp64 oracle.

Outputs are bf16: per (query row, head) the max relative error over the head's d
values (max |gpu - ref| / max |ref|) must stay within 2e-2; the log-sum-exp is fp32
and is held to 1e-4 relative. Shapes cover every supported head grouping, contexts
that are empty or not multiples of the 64-key tile, several partition counts, a
request without nodes, deep and wide trees, and pad rows that hold NaN.
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
from lumo_synth import trees  # noqa: E402
from lumo_synth import operands as ops  # noqa: E402

D = 128


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bf16(rng, shape, scale=1.0):
    return ops.to_bf16_bits((scale * rng.standard_normal(shape)).astype(np.float32))


def make_case(seed, parents, n_rows, n_ctx, h_q, h_kv, pad_nan=True):
    rng = np.random.default_rng(seed)
    row_off = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    total = int(row_off[-1])
    ctx_off = np.concatenate([[0], np.cumsum(n_ctx)]).astype(np.int32)
    a = dict(q=bf16(rng, (total, h_q, D)), k_tree=bf16(rng, (total, h_kv, D)),
             v_tree=bf16(rng, (total, h_kv, D)), k_ctx=bf16(rng, (max(int(ctx_off[-1]), 1), h_kv, D)),
             v_ctx=bf16(rng, (max(int(ctx_off[-1]), 1), h_kv, D)))
    if pad_nan:
        rows = set(oracle.plan.flat_rows(parents, row_off).tolist()) if total else set()
        pad = [x for x in range(total) if x not in rows]
        for key in ("q", "k_tree", "v_tree"):
            a[key][pad] = np.uint16(0x7FC0)
    node_off = np.concatenate([[0], np.cumsum([len(p) for p in parents])]).astype(np.int32)
    return row_off, total, ctx_off, node_off, a


def run_gpu(parents, n_rows, node_off, ctx_off, a, h_q, h_kv, n_split, scale):
    desc = L.TreeDesc.build(node_off, np.concatenate(parents) if parents else np.zeros(0, np.int32),
                            np.asarray(n_rows, np.int32))
    d = L.attn_dims(len(parents), h_q, h_kv)
    dev = {k: torch.from_numpy(v).cuda() for k, v in a.items()}
    total = int(sum(n_rows))
    o = torch.zeros((total, h_q, D), dtype=torch.int16, device="cuda")
    lse = torch.full((total, h_q), 7.0, dtype=torch.float32, device="cuda")
    ws = torch.empty(L.lumo_tree_attention_workspace_bytes(d, desc.plan, n_split) // 4 + 1,
                     dtype=torch.float32, device="cuda")
    max_ctx = int(np.max(np.diff(ctx_off))) if len(ctx_off) > 1 else 0
    L.lumo_tree_attention(d, desc, torch.from_numpy(ctx_off).cuda(), max_ctx, scale, dev["q"],
                          dev["k_ctx"], dev["v_ctx"], dev["k_tree"], dev["v_tree"], o, lse, n_split, ws)
    torch.cuda.synchronize()
    return gu_bf16(o), lse.cpu().numpy()


def gu_bf16(t):
    return ops.bf16_bits_to_f32(t.cpu().numpy().view(np.uint16)).astype(np.float64)


def check(parents, row_off, total, ctx_off, a, o, lse, h_q, h_kv, scale, tol=2e-2):
    ref_o, ref_l = oracle.tree_attention(parents, row_off, total, ctx_off, a["q"], a["k_ctx"], a["v_ctx"],
                                         a["k_tree"], a["v_tree"], h_q=h_q, h_kv=h_kv, d=D,
                                         op_dtype=ops.BF16, scale=scale)
    rows = oracle.plan.flat_rows(parents, row_off)
    worst = 0.0
    for x in rows:
        for h in range(h_q):
            den = np.max(np.abs(ref_o[x, h]))
            e = np.max(np.abs(o[x, h] - ref_o[x, h])) / den
            worst = max(worst, e)
            assert e <= tol, f"row {x} head {h}: max rel err {e:.3e}"
            assert abs(lse[x, h] - ref_l[x, h]) <= 1e-4 * max(1.0, abs(ref_l[x, h])), (x, h)
    pad = [x for x in range(total) if x not in set(rows.tolist())]
    assert np.all(o[pad] == 0) and np.all(lse[pad] == 7.0)  # pad rows untouched
    return worst


@pytest.mark.parametrize("h_q,h_kv,n_split", [(4, 2, 3), (8, 8, 1), (8, 2, 7), (16, 2, 2)])
def test_tree_attention_parity(h_q, h_kv, n_split):
    """Four requests: the Fig. 1 tree with 100 context tokens, a 40-node tree with 1000,
    a 20-node chain with none, a request without nodes; head groupings 2, 1, 4 and 8."""
    rng = np.random.default_rng(5)
    parents = [trees.FIG1_PARENT, trees.random_tree(rng, 40, 8, trees.bmax_uniform(4)), trees.chain(20),
               np.zeros(0, np.int32)]
    n_rows = [8, 41, 20, 2]
    n_ctx = [100, 1000, 0, 37]
    scale = 1.0 / np.sqrt(D)
    row_off, total, ctx_off, node_off, a = make_case(11, parents, n_rows, n_ctx, h_q, h_kv)
    say(f"[gpu] tree attention h_q={h_q} h_kv={h_kv} n_split={n_split}")
    o, lse = run_gpu(parents, n_rows, node_off, ctx_off, a, h_q, h_kv, n_split, scale)
    worst = check(parents, row_off, total, ctx_off, a, o, lse, h_q, h_kv, scale)
    say(f"  worst max-rel {worst:.3e}")


def test_tree_attention_wide_tree_and_split_invariance():
    """A 150-node tree (three 64-key tree tiles, five query chunks): every partition count
    gives the oracle's result, and repeated calls are bitwise identical."""
    rng = np.random.default_rng(6)
    parents = [trees.random_tree(rng, 150, 12, trees.bmax_root_skewed)]
    n_rows, n_ctx = [150], [777]
    h_q, h_kv, scale = 4, 2, 0.05
    row_off, total, ctx_off, node_off, a = make_case(12, parents, n_rows, n_ctx, h_q, h_kv)
    outs = []
    for n_split in (1, 4, 13):
        o, lse = run_gpu(parents, n_rows, node_off, ctx_off, a, h_q, h_kv, n_split, scale)
        check(parents, row_off, total, ctx_off, a, o, lse, h_q, h_kv, scale)
        outs.append(o)
    o2, _ = run_gpu(parents, n_rows, node_off, ctx_off, a, h_q, h_kv, 13, scale)
    assert np.array_equal(o2, outs[-1])


def test_tree_attention_paper_geometry_long_context():
    """The evaluated geometry (28 nodes in 32 rows) over a 131,072-token context, 16 query
    heads in pairs on 8 key/value heads; checked on all nodes of four heads."""
    parents = [trees.paper_geometry_tree()]
    n_rows, n_ctx = [32], [131072]
    h_q, h_kv = 16, 8
    scale = 1.0 / np.sqrt(D)
    row_off, total, ctx_off, node_off, a = make_case(13, parents, n_rows, n_ctx, h_q, h_kv)
    desc = L.TreeDesc.build(node_off, parents[0], np.asarray(n_rows, np.int32))
    n_split = L.lumo_tree_attention_splits(L.attn_dims(1, h_q, h_kv), desc.plan, 131072)
    say(f"[gpu] tree attention paper geometry, n_split={n_split}")
    o, lse = run_gpu(parents, n_rows, node_off, ctx_off, a, h_q, h_kv, n_split, scale)
    # the oracle on heads 0, 5, 10, 15 only (sub-arrays keep the head grouping)
    for h in (0, 5, 10, 15):
        g = h // 2
        sub = dict(q=a["q"][:, h:h + 1], k_ctx=a["k_ctx"][:, g:g + 1], v_ctx=a["v_ctx"][:, g:g + 1],
                   k_tree=a["k_tree"][:, g:g + 1], v_tree=a["v_tree"][:, g:g + 1])
        ref_o, ref_l = oracle.tree_attention(parents, row_off, total, ctx_off, sub["q"], sub["k_ctx"],
                                             sub["v_ctx"], sub["k_tree"], sub["v_tree"], h_q=1, h_kv=1,
                                             d=D, op_dtype=ops.BF16, scale=scale)
        rows = oracle.plan.flat_rows(parents, row_off)
        for x in rows:
            e = np.max(np.abs(o[x, h] - ref_o[x, 0])) / np.max(np.abs(ref_o[x, 0]))
            assert e <= 2e-2, (x, h, e)
            assert abs(lse[x, h] - ref_l[x, 0]) <= 1e-4 * abs(ref_l[x, 0]), (x, h)
