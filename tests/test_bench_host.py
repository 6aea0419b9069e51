"""Host logic of bench.py: the algorithmic bytes and flops its roofline divides by (set
against the per-unit figures of the batched workload: 6 d^2 flop and 776 operand bytes
per head-node update, 64 KiB of fp32 state per instance read once, a state read and
written per instance by the commit), the percentile helper, and the one-GPU guard."""
from __future__ import annotations

import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from lumo_synth import configs  # noqa: E402


def path_len(parent, a):
    n = 0
    while a != -1:
        n, a = n + 1, int(parent[a])
    return n


def test_algorithmic_work_batched():
    wl, _ = configs.topology("batched")
    ab = bench.alg_bytes_flops(wl)
    hn = 8 * 64 * 48 * 32
    inst = 8 * 48 * 32
    assert wl.head_node_updates == hn
    assert ab["verify_flops"] == hn * 6 * 128 * 128                      # 77.3 GFLOP
    assert ab["verify_bytes"] == hn * 776 + inst * 128 * 128 * 4          # 1,415.6 MB
    assert abs(ab["verify_bytes"] / 1e6 - 1415.6) < 0.1
    lens = [path_len(p, a) for p, a in zip(wl.parents, wl.accepted)]
    assert all(1 <= x <= 8 for x in lens)
    upd = sum(lens) * 48 * 32
    assert ab["commit_updates"] == upd
    assert ab["commit_bytes"] == inst * 2 * 65536 + upd * (128 + 256 + 8)
    assert ab["pub_bytes"] == ab["commit_bytes"] - inst * 65536
    # history publication: three x rows read and three entries written per (request, layer)
    assert ab["hist_pub_bytes"] == 8 * 48 * 3 * 8192 * 2 * 2
    # x read + y written and the history read (824.2 MB), plus the taps (6.3 MB)
    assert ab["conv_bytes"] == 512 * 48 * 8192 * 4 + 8 * 48 * 3 * 8192 * 2 + 48 * 8192 * 16
    assert abs(ab["conv_bytes"] / 1e6 - 830.5) < 0.1


def test_algorithmic_work_counts_each_node_once():
    """Head-node updates count nodes once, whatever their depth; f32 operands double the
    operand bytes but not the state bytes."""
    wl, _ = configs.topology("tiny")
    ab = bench.alg_bytes_flops(wl)
    n = len(wl.parents[0])
    assert wl.head_node_updates == n * wl.n_layers * wl.h_v
    per = (2 * wl.d_k * 4) / (wl.h_v // wl.h_k) + wl.d_v * 4 + 8 + wl.d_v * 4
    assert ab["verify_bytes"] == wl.head_node_updates * per + wl.n_layers * wl.h_v * wl.d_k * wl.d_v * 4


def test_percentiles():
    xs = list(np.arange(1.0, 101.0))
    assert bench.pct(xs) == [11.0, 51.0, 91.0]
    assert bench.pct([2.5]) == [2.5, 2.5, 2.5]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""
