"""Helpers of the GPU parity tests: run the HIP path through the C ABI and compare
with the oracle (fp64) under the stated tolerances."""
from __future__ import annotations

import numpy as np

import oracle
from lumo_synth import operands as ops

# Tolerances on max relative error per instance (max|gpu-ref| / max|ref|):
# fp32 operands 1e-4, bf16 operands 2e-2 (outputs are bf16-rounded); the fp32
# published states are held to 1e-4 in both cases (the oracle reads the same
# rounded operands, so only fp32 arithmetic separates them).
TOL_F32 = 1e-4
TOL_BF16 = 2e-2
TOL_STATE = 1e-4


def out_tol(wl):
    return TOL_F32 if wl.op_dtype == ops.F32 else TOL_BF16


def to_np(t):
    """Device tensor -> float32 numpy (bf16 decoded exactly)."""
    import torch
    if t.dtype == torch.bfloat16:
        bits = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return ops.bf16_bits_to_f32(bits)
    return t.cpu().numpy()


def max_rel(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    if den == 0:
        return float(np.max(np.abs(gpu)))
    return float(np.max(np.abs(gpu - ref)) / den)


def node_rows(wl, r):
    return oracle.plan.rows_of(wl.parents[r], int(wl.row_off[r]))


def sample_instances(wl, n, seed=0):
    rng = np.random.default_rng(seed)
    allc = [(r, l, h) for r in range(wl.n_req) for l in range(wl.n_layers) for h in range(wl.h_v)]
    if len(allc) <= n:
        return allc
    idx = rng.choice(len(allc), size=n, replace=False)
    return [allc[i] for i in sorted(idx)]


def check_outputs(wl, o_gpu, instances, tol=None, arrays=None):
    """Per-instance max relative error of GPU outputs vs the oracle; returns the worst."""
    tol = out_tol(wl) if tol is None else tol
    worst = 0.0
    for (r, l, h) in instances:
        n = len(wl.parents[r])
        ref = oracle.verify_nodes(wl, r, l, h, list(range(n)), arrays=arrays)
        rows = node_rows(wl, r)
        got = o_gpu[l, rows, h, :]
        assert np.all(np.isfinite(got)), (r, l, h)
        e = max_rel(got, ref)
        worst = max(worst, e)
        assert e <= tol, f"instance {(r, l, h)}: max rel err {e:.3e} > {tol:.1e}"
    return worst


def check_states(wl, st_gpu, st_ref, instances, tol=TOL_STATE):
    worst = 0.0
    for (r, l, h) in instances:
        e = max_rel(st_gpu[r, l, h], st_ref[r, l, h])
        worst = max(worst, e)
        assert e <= tol, f"state {(r, l, h)}: max rel err {e:.3e} > {tol:.1e}"
    return worst
