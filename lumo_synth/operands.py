"""Seeded synthetic operands for tree GDN verification.

Value distributions (identical for every configuration):
  q, k ~ N(0, 1), each k row (node, key head) L2-normalised in float64 then rounded
  v ~ N(0, 1)
  beta = sigmoid(N(0, 1)), g = -softplus(N(0, 1))  (decay alpha = exp(g))
  initial recurrent state ~ N(0, 0.1^2)
  conv input x ~ N(0, 1), committed conv history ~ N(0, 1), taps ~ U(-1/2, 1/2)

All arrays use the physical-row layouts of the library boundary:
  q, k   [layers][rows][h_k][d_k]       (operand dtype)
  v      [layers][rows][h_v][d_v]       (operand dtype)
  g, beta[layers][rows][h_v]            float32
  state  [requests][layers][h_v][d_k][d_v] float32 (key-major)
  x      [layers][rows][C]              (operand dtype)
  hist   [requests][layers][3][C]       (operand dtype)
  w      [layers][C][4]                 float32
bf16 data is held as uint16 bit patterns. Nothing here evaluates the recurrence.

Large arrays are filled in independent chunks, each from its own PCG64 stream keyed
by (seed, array id, chunk id), so the values do not depend on the thread count.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F32 = 0
BF16 = 1

_CHUNK = 1 << 22


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32/float64 values to bfloat16 (round to nearest even); returns uint16 bits."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    b = f.view(np.uint32)
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    out = rounded.astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def as_float(a: np.ndarray, op_dtype: int) -> np.ndarray:
    """Decode an operand array (float32 or bf16 bits) to float32 values."""
    if op_dtype == F32:
        return np.asarray(a, dtype=np.float32)
    return bf16_bits_to_f32(a)


def _kind_fn(kind: str, out_dtype: int, row: int):
    def normal(g, n):
        return g.standard_normal(size=n, dtype=np.float32)

    def fin(a):
        if out_dtype == BF16:
            return to_bf16_bits(a)
        return a.astype(np.float32, copy=False)

    if kind == "normal":
        return lambda g, n: fin(normal(g, n))
    if kind == "state":
        return lambda g, n: normal(g, n) * np.float32(0.1)
    if kind == "unit_rows":
        def f(g, n):
            a = normal(g, n).astype(np.float64).reshape(-1, row)
            a /= np.sqrt((a * a).sum(axis=1, keepdims=True))
            return fin(a.reshape(-1))
        return f
    if kind == "sigmoid":
        return lambda g, n: (1.0 / (1.0 + np.exp(-normal(g, n).astype(np.float64)))).astype(np.float32)
    if kind == "neg_softplus":
        return lambda g, n: (-np.logaddexp(0.0, normal(g, n).astype(np.float64))).astype(np.float32)
    if kind == "taps":
        return lambda g, n: g.uniform(-0.5, 0.5, size=n).astype(np.float32)
    raise KeyError(kind)


def fill(shape, seed: int, array_id: int, kind: str, out_dtype: int = F32) -> np.ndarray:
    """Deterministic chunked fill of an array of the given shape."""
    shape = tuple(int(s) for s in shape)
    n = int(np.prod(shape))
    row = shape[-1]
    chunk = max(row, (_CHUNK // row) * row)
    fn = _kind_fn(kind, out_dtype, row)
    dt = np.uint16 if (out_dtype == BF16 and kind in ("normal", "unit_rows")) else np.float32
    out = np.empty(n, dtype=dt)
    n_chunks = (n + chunk - 1) // chunk

    def work(c):
        lo = c * chunk
        hi = min(n, lo + chunk)
        g = np.random.default_rng([seed, array_id, c])
        out[lo:hi] = fn(g, hi - lo)

    if n_chunks == 1:
        work(0)
    else:
        with ThreadPoolExecutor(min(16, os.cpu_count() or 1)) as ex:
            list(ex.map(work, range(n_chunks)))
    return out.reshape(shape)


def make_gdn_operands(seed: int, *, n_req, n_layers, total_rows, h_k, h_v, d_k, d_v, op_dtype):
    """Per-row q/k/v/g/beta and per-request initial state."""
    return dict(
        q=fill((n_layers, total_rows, h_k, d_k), seed, 1, "normal", op_dtype),
        k=fill((n_layers, total_rows, h_k, d_k), seed, 2, "unit_rows", op_dtype),
        v=fill((n_layers, total_rows, h_v, d_v), seed, 3, "normal", op_dtype),
        g=fill((n_layers, total_rows, h_v), seed, 4, "neg_softplus"),
        beta=fill((n_layers, total_rows, h_v), seed, 5, "sigmoid"),
        state0=fill((n_req, n_layers, h_v, d_k, d_v), seed, 6, "state"),
    )


def make_conv_operands(seed: int, *, n_req, n_layers, total_rows, channels, op_dtype):
    return dict(
        x=fill((n_layers, total_rows, channels), seed, 7, "normal", op_dtype),
        hist=fill((n_req, n_layers, 3, channels), seed, 8, "normal", op_dtype),
        w=fill((n_layers, channels, 4), seed, 9, "taps"),
    )
