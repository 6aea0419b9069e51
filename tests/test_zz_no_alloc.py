"""lumo_tree_attention_noalloc: tree attention (Sec. V-B) for callers that cannot
allocate device memory, through the C ABI.

The entry point keeps the key ranges' partial results in the library's fixed
per-device scratch array instead of a caller workspace. Two calls in a row, the
second smaller than the first (so the array still holds the first call's partial
results), must each equal lumo_tree_attention with a caller workspace filled with
garbage, bit for bit (same kernels, same partition count, so the same reduction
order), and the smaller one also the fp64 oracle within the bf16 tolerance. A shape
whose partial results exceed the array is refused before any launch.
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


def _bf16(rng, shape):
    return ops.to_bf16_bits(rng.standard_normal(shape).astype(np.float32))


def _case(seed, parents, n_rows, n_ctx, h_q, h_kv):
    rng = np.random.default_rng(seed)
    row_off = np.concatenate([[0], np.cumsum(n_rows)]).astype(np.int32)
    total = int(row_off[-1])
    ctx_off = np.concatenate([[0], np.cumsum(n_ctx)]).astype(np.int32)
    n_tok = max(int(ctx_off[-1]), 1)
    a = dict(q=_bf16(rng, (total, h_q, D)), k_tree=_bf16(rng, (total, h_kv, D)),
             v_tree=_bf16(rng, (total, h_kv, D)), k_ctx=_bf16(rng, (n_tok, h_kv, D)),
             v_ctx=_bf16(rng, (n_tok, h_kv, D)))
    node_off = np.concatenate([[0], np.cumsum([len(p) for p in parents])]).astype(np.int32)
    desc = L.TreeDesc.build(node_off, np.concatenate(parents), np.asarray(n_rows, np.int32))
    return dict(parents=parents, row_off=row_off, total=total, ctx_off=ctx_off, a=a, desc=desc,
                h_q=h_q, h_kv=h_kv, max_ctx=int(np.max(np.diff(ctx_off))))


def _run(c, n_split, noalloc):
    d = L.attn_dims(len(c["parents"]), c["h_q"], c["h_kv"])
    dev = {k: torch.from_numpy(v).cuda() for k, v in c["a"].items()}
    ctx = torch.from_numpy(c["ctx_off"]).cuda()
    o = torch.full((c["total"], c["h_q"], D), 0x7FC0, dtype=torch.int16, device="cuda")
    lse = torch.full((c["total"], c["h_q"]), 7.0, dtype=torch.float32, device="cuda")
    scale = 1.0 / np.sqrt(D)
    if noalloc:
        L.lumo_tree_attention_noalloc(d, c["desc"], ctx, c["max_ctx"], scale, dev["q"], dev["k_ctx"],
                                      dev["v_ctx"], dev["k_tree"], dev["v_tree"], o, lse, n_split)
    else:
        nb = L.lumo_tree_attention_workspace_bytes(d, c["desc"].plan, n_split)
        ws = torch.full((nb // 4 + 1,), float("nan"), dtype=torch.float32, device="cuda")
        L.lumo_tree_attention(d, c["desc"], ctx, c["max_ctx"], scale, dev["q"], dev["k_ctx"], dev["v_ctx"],
                              dev["k_tree"], dev["v_tree"], o, lse, n_split, ws)
    torch.cuda.synchronize()
    rows = oracle.plan.flat_rows(c["parents"], c["row_off"])
    return o.cpu().numpy()[rows], lse.cpu().numpy()[rows]


def _same(x, y):
    return np.array_equal(x.view(np.uint16 if x.dtype == np.int16 else np.uint32),
                          y.view(np.uint16 if y.dtype == np.int16 else np.uint32))


def test_noalloc_matches_workspace_call_twice_then_smaller():
    big = _case(9, [trees.paper_geometry_tree()], [32], [131072], 16, 8)
    d_big = L.attn_dims(1, 16, 8)
    n_big = L.lumo_tree_attention_splits(d_big, big["desc"].plan, big["max_ctx"])
    need = L.lumo_tree_attention_workspace_bytes(d_big, big["desc"].plan, n_big)
    say(f"[gpu] noalloc attention: paper geometry, 131072 context tokens, n_split {n_big}, {need} B")
    assert need <= L.LUMO_TREE_ATTENTION_SCRATCH_BYTES
    o1, l1 = _run(big, n_big, noalloc=True)
    o0, l0 = _run(big, n_big, noalloc=False)
    assert _same(o1, o0) and _same(l1, l0)
    assert np.all(np.isfinite(l1))

    rng = np.random.default_rng(4)
    small_par = [trees.random_tree(rng, 40, 7, trees.bmax_uniform(3)), trees.FIG1_PARENT.copy(),
                 np.array([-1], np.int32)]
    small = _case(5, small_par, [43, 7, 2], [37, 0, 100], 4, 2)
    say("[gpu] noalloc attention: three requests (40, 7, 1 nodes), contexts 37 / 0 / 100, n_split 3")
    o2, l2 = _run(small, 3, noalloc=True)
    o3, l3 = _run(small, 3, noalloc=False)
    assert _same(o2, o3) and _same(l2, l3)
    ref_o, ref_l = oracle.tree_attention(small_par, small["row_off"], small["total"], small["ctx_off"],
                                         small["a"]["q"], small["a"]["k_ctx"], small["a"]["v_ctx"],
                                         small["a"]["k_tree"], small["a"]["v_tree"], h_q=4, h_kv=2, d=D,
                                         op_dtype=ops.BF16, scale=1.0 / np.sqrt(D))
    rows = oracle.plan.flat_rows(small_par, small["row_off"])
    got = ops.bf16_bits_to_f32(o2.view(np.uint16)).astype(np.float64)
    ro, rl = ref_o[rows], ref_l[rows]
    err = np.max(np.abs(got - ro), axis=-1) / np.max(np.abs(ro), axis=-1)
    assert float(np.max(err)) <= 2e-2
    np.testing.assert_allclose(l2, rl, rtol=1e-4)

    # the big call again after the small one: the same result as the first time
    o4, l4 = _run(big, n_big, noalloc=True)
    assert _same(o4, o1) and _same(l4, l1)


def test_noalloc_refuses_partials_beyond_the_array():
    c = _case(6, [trees.paper_geometry_tree()], [32], [4096], 16, 8)
    d = L.attn_dims(1, 16, 8)
    n_split = 127  # 128 ranges x 32 rows x 16 heads x 129 floats > 32 MiB
    assert L.lumo_tree_attention_workspace_bytes(d, c["desc"].plan, n_split) > L.LUMO_TREE_ATTENTION_SCRATCH_BYTES
    with pytest.raises(L.LumoError) as ei:
        _run(c, n_split, noalloc=True)
    assert ei.value.status == L.LUMO_ESPACE and "scratch" in str(ei.value)
