"""Benchmark of one speculative verification step of tree GDN on one MI355X.

A step is one pass of the whole hot path over the batch: tree causal-conv gather,
path verification of every node, and publication of the accepted path (device path
derivation, replay into the native state, conv-history update). Consecutive steps
form a serving loop: each verify reads the state the previous commit published.

Prints one JSON line: head-node updates per second (tree nodes x layers x value
heads, each node counted once) over K steps replayed from captured graphs of ten steps
(--eager: launched one by one from Python), the roofline of the dominant kernel
(verify) with its duration measured by HIP events on the launch stream (an eager pass
of K steps with events around every stage) and set against the published peak and
against a plain device copy timed in the same run, the other kernels' durations,
per-step percentiles, and the fp64 CPU oracle timed on a bounded sample of the same
workload (all host cores, and one thread).

  python bench.py [--steps K] [--warmup W] [--config batched] [--policy wy]
                  [--commit deferred|eager]
  (deferred: each step's conv first publishes the previous step's accepted path into
   the conv history, its verification publishes that path into the state in the same
   pass over the state, and the commit only derives the path; eager: the commit
   publishes the history and replays the path itself; wy policy only)
  python bench.py --copy-probe     # plain 1 GiB device copy (HBM counter calibration)
  python bench.py --attention      # tree attention over a 131,072-token context (separate line)
  python bench.py --select         # fused draft selection over 248,320-logit rows (separate line)

The roofline's `traffic` (measured HBM bytes per verify call) is reported from
profiles/traffic.json only while the verify kernel's sources hash to the value the
counters were taken with; after any change to them it is null until re-measured.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tree GDN head-node updates/sec + % of HBM/VALU roofline, 1 MI355X"
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, published
PEAK_VALU_F32_TFS = 157.3      # MI355X fp32 vector, published (256 CU x 2.4 GHz)
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "traffic.json")
# sources that determine the code of each policy's verify kernels
VERIFY_SOURCES = {
    "wy": ["verify_wy.hip", "verify_wy_body.inc", "verify_wy.h", "device_common.h", "internal.h", "launch.h"],
    "paths": ["verify_scan.hip", "device_common.h", "internal.h", "launch.h"],
    "wyv": ["verify_wyv.hip", "device_common.h", "internal.h", "launch.h"],
    "attention": ["attention.hip", "device_common.h", "internal.h", "launch.h"],
    "select": ["select.hip", "select.h", "device_common.h"],
}
ATTN_CONFIG = "paper28_ctx131072"


def verify_source_hash(policy):
    files = VERIFY_SOURCES.get(policy, VERIFY_SOURCES["paths"])
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2609_23900_amd", "csrc", f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def recorded_traffic(policy, config, commit="eager"):
    """Measured HBM bytes per verify call, if recorded for exactly these kernel sources."""
    try:
        with open(TRAFFIC_RECORD) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    for r in rec.get("records", []):
        if (r.get("policy") == policy and r.get("config") == config and r.get("commit", "eager") == commit
                and r.get("sources_sha256") == verify_source_hash(policy)):
            return r
    return None


def copy_rate(reps=3):
    """Milliseconds per plain device copy of 1 GiB (read) into 1 GiB (written), and the
    read + write rate in GB/s: the practical HBM ceiling a kernel is compared with."""
    import torch
    n = 256 * 1024 * 1024
    a = torch.ones(n, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del a, b
    return ms, 2 * n * 4 / (ms * 1e-3) / 1e9


def copy_probe():
    """A plain device copy of known size (1 GiB read + 1 GiB written, four times with the
    first as warm-up): the calibration of the HBM byte counters."""
    ms, gbs = copy_rate()
    print(json.dumps({"copy_probe_bytes": 256 * 1024 * 1024 * 4, "copies": 4, "ms_per_copy": round(ms, 4),
                      "read_plus_write_GBps": round(gbs, 1)}), flush=True)


def pct(xs):
    """10th, 50th and 90th percentiles (nearest rank) of a list of times."""
    ys = sorted(xs)
    return [round(ys[min(len(ys) - 1, int(q * len(ys)))], 4) for q in (0.1, 0.5, 0.9)]


def host_cpu():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


WORKLOAD_TEXT = {
    "tiny": "Fig. 1 tree, 1 request, 1 head, d=16, fp32 operands",
    "layer1": "1 request x 1 GDN layer x 32 value heads (16 key heads), d_k=d_v=128, one 64-node tree (depth<=8, branching 1-4), bf16 operands, fp32 state",
    "batched": "8 requests x 48 GDN layers x 32 value heads (16 key heads), d_k=d_v=128, per-request 64-node trees (depth<=8, branching 1-4), bf16 operands, fp32 state, commit of accepted paths of length 1-8, conv C=8192",
    "widedeep": "32 requests x 1 layer x 32 value heads, d=128, 256-node trees (depth<=16, root-skewed branching 1-6), bf16 operands",
    "chainmix": "64 requests x 1 layer x 32 value heads, d=128: 32 chains of 16 + 32 trees of 128 nodes, bf16 operands, accepted lengths 0-16",
    "paper28": "1 request x 1 layer x 32 value heads, d=128, the 28-node draft geometry padded to 32 rows",
}


ATTN_WORKLOAD = ("tree attention: the 28-node draft geometry in 32 rows, 1 request, 131,072 context "
                 "tokens, 16 query heads in pairs on 8 key/value heads, d=128, bf16")


def attention_bench(args):
    """Tree attention (lumo_tree_attention) on the evaluated geometry: HBM-bound by the
    context keys and values; one step = one attention layer's call."""
    import numpy as np
    import torch

    import paper_2609_23900_amd as L
    from lumo_synth import operands as ops
    from lumo_synth import trees

    par = trees.paper_geometry_tree()
    n_ctx, h_q, h_kv, d = 131072, 16, 8, 128
    desc = L.TreeDesc.build(np.array([0, len(par)], np.int32), par, np.array([32], np.int32))
    dims = L.attn_dims(1, h_q, h_kv, d)
    rng = np.random.default_rng(9)

    def bf(shape):
        return torch.from_numpy(ops.to_bf16_bits(rng.standard_normal(shape).astype(np.float32))).cuda()

    q, kt, vt = bf((32, h_q, d)), bf((32, h_kv, d)), bf((32, h_kv, d))
    kc, vc = bf((n_ctx, h_kv, d)), bf((n_ctx, h_kv, d))
    ctx_off = torch.tensor([0, n_ctx], dtype=torch.int32, device="cuda")
    o = torch.zeros((32, h_q, d), dtype=torch.int16, device="cuda")
    lse = torch.zeros((32, h_q), dtype=torch.float32, device="cuda")
    n_split = L.lumo_tree_attention_splits(dims, desc.plan, n_ctx)
    ws = torch.empty(L.lumo_tree_attention_workspace_bytes(dims, desc.plan, n_split) // 4 + 1,
                     dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    def step():
        L.lumo_tree_attention(dims, desc, ctx_off, n_ctx, 1.0 / np.sqrt(d), q, kc, vc, kt, vt, o, lse,
                              n_split, ws, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    nodes = len(par)
    alg = 2 * n_ctx * h_kv * d * 2 + 32 * (h_q + 2 * h_kv) * d * 2 + nodes * h_q * (d * 2 + 4)
    ach = alg / (ms * 1e-3) / 1e9
    out = {"metric": "tree attention query-head rows/sec + % of HBM roofline, 1 MI355X",
           "value": round(nodes * h_q / (ms * 1e-3), 1), "unit": "query-head rows/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (N(0,1) queries, keys and values)",
           "config": {"workload": ATTN_WORKLOAD, "n_split": n_split},
           "roofline": {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None,
                        "kernel": "tree attention call (partition kernel + merge kernel)",
                        "per_launch": f"{alg / 1e6:.1f} MB algorithmic (context keys and values once)"}}
    tr = recorded_traffic("attention", ATTN_CONFIG, "n/a")
    if tr is not None:
        out["roofline"]["traffic"] = {"fetch_bytes": tr["fetch_bytes"], "write_bytes": tr["write_bytes"],
                                      "total_bytes": tr["fetch_bytes"] + tr["write_bytes"],
                                      "unit": "B per attention call", "source": "profiles/traffic.json"}
    if not args.no_copy:
        _, cgbs = copy_rate()
        out["roofline"]["practical"] = {"copy_GBps": round(cgbs, 1), "frac_of_copy": round(ach / cgbs, 4),
                                        "what": "plain 1 GiB device copy (read + write) timed in this run"}
    print(json.dumps(out), flush=True)


SEL_VOCAB = 248320
SEL_ROTATE_BYTES = 508e6  # logits cycled per replay: twice the 256 MB Infinity Cache


def select_bench(args):
    """Fused draft selection (lumo_draft_select): one call per drafting depth ranks one
    full-vocabulary logits row per request (k = 3 candidates plus the spine token).
    HBM-bound: every logit is read once. Calls are captured in a graph, one call per
    logits buffer, and the graph is replayed, so the time is the device's (Python's
    launch cost excluded) and, with about 508 MB of logits cycled, the reads come from
    HBM rather than the Infinity Cache; `resident` repeats one buffer instead. Two batch
    sizes: 8 rows (the batched workload's requests; a few microseconds, so launch
    latency weighs in) and 64 rows."""
    import numpy as np
    import torch

    import oracle
    import paper_2609_23900_amd as L
    from lumo_synth import operands as ops

    rng = np.random.default_rng(3)
    k, ties = 3, 1
    res = {}
    host8 = None
    for rows, dt, name in ((8, ops.F32, "rows8_f32"), (64, ops.BF16, "rows64_bf16")):
        esz = 2 if dt == ops.BF16 else 4
        nbuf = max(2, int(SEL_ROTATE_BYTES // (rows * SEL_VOCAB * esz)))
        x = (rng.standard_normal((rows, SEL_VOCAB)) * 3).astype(np.float32)
        if dt == ops.BF16:
            t0 = torch.from_numpy(ops.to_bf16_bits(x).view(np.int16)).cuda().view(torch.bfloat16)
        else:
            t0 = torch.from_numpy(x).cuda()
            host8 = x
        bufs = [t0] + [t0[:, torch.randperm(SEL_VOCAB, device="cuda")].contiguous() for _ in range(nbuf - 1)]
        n_split = L.lumo_draft_select_splits(rows, SEL_VOCAB, dt)
        ws = torch.zeros(max(16, L.lumo_draft_select_workspace_bytes(rows, k, n_split)), dtype=torch.uint8,
                         device="cuda")
        spine = torch.zeros(rows, dtype=torch.int32, device="cuda")
        cand = torch.zeros((rows, k), dtype=torch.int32, device="cuda")
        out = {}
        for mode in ("rotating", "resident"):
            seq = bufs if mode == "rotating" else [t0] * len(bufs)
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):  # eager warm-up on the capture's stream
                for b in seq:
                    L.lumo_draft_select(b, k, ties, spine, cand, n_split, ws)
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for b in seq:
                    L.lumo_draft_select(b, k, ties, spine, cand, n_split, ws)
            stream = torch.cuda.current_stream()
            reps = max(1, -(-args.steps // len(seq)))
            for _ in range(max(1, args.warmup // len(seq))):
                g.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(reps):
                g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            out[mode] = e0.elapsed_time(e1) / (reps * len(seq))
            out[mode + "_calls"] = reps * len(seq)
            del g
        want = oracle.draft_select(x if dt == ops.F32 else ops.to_bf16_bits(x), k=k, op_dtype=dt, ties=ties)
        L.lumo_draft_select(t0, k, ties, spine, cand, n_split, ws)
        assert np.array_equal(spine.cpu().numpy(), want[0]) and np.array_equal(cand.cpu().numpy(), want[1])
        ms = out["rotating"]
        nbytes = rows * SEL_VOCAB * esz + rows * (k + 1) * 4
        ach = nbytes / (ms * 1e-3) / 1e9
        res[name] = {"rows": rows, "dtype": "bf16" if dt == ops.BF16 else "f32", "n_split": n_split,
                     "us_per_call": round(ms * 1e3, 3), "rows_per_s": round(rows / (ms * 1e-3), 1),
                     "alg_bytes": nbytes, "achieved_GBps": round(ach, 1), "frac": round(ach / PEAK_HBM_GBS, 4),
                     "calls_timed": out["rotating_calls"], "buffers_cycled": len(bufs),
                     "resident_us_per_call": round(out["resident"] * 1e3, 3)}
        del bufs, t0
    main = res["rows8_f32"]
    out = {"metric": "draft selection logits rows/sec + % of HBM roofline, 1 MI355X",
           "value": main["rows_per_s"], "unit": "logits rows/s", "n_gpus": 1, "steps": main["calls_timed"],
           "warmup": args.warmup, "ms_per_step": round(main["us_per_call"] / 1e3, 6),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": f"{main['dtype']} logits, exact ordering on 64-bit integer ranking words",
           "data": "synthetic (N(0, 9) logits)",
           "config": {"workload": f"draft selection: 8 rows x {SEL_VOCAB:,} float32 logits, argmax + ordered "
                                  "top-3 (ties: higher index first), graph-replayed, 508 MB of logits cycled",
                      "n_split": main["n_split"]},
           "roofline": {"bound": "hbm", "achieved": main["achieved_GBps"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": main["frac"], "traffic": None,
                        "kernel": "selection call (part kernel + merge kernel)",
                        "per_launch": f"{main['alg_bytes'] / 1e6:.2f} MB algorithmic (every logit once)"},
           "batches": res}
    tr = recorded_traffic("select", "rows8_f32", "n/a")
    if tr is not None:
        out["roofline"]["traffic"] = {"fetch_bytes": tr["fetch_bytes"], "write_bytes": tr["write_bytes"],
                                      "total_bytes": tr["fetch_bytes"] + tr["write_bytes"],
                                      "unit": "B per selection call", "source": "profiles/traffic.json"}
    if not args.no_cpu:
        import time
        oracle.draft_select(host8[:1], k=k, op_dtype=ops.F32, ties=ties)
        reps, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < min(args.cpu_budget, 5.0) or reps == 0:
            oracle.draft_select(host8, k=k, op_dtype=ops.F32, ties=ties, n_threads=1)
            reps += 1
        dt_s = (time.perf_counter() - t0) / reps
        out["cpu_baseline"] = {"value": round(8 / dt_s, 1), "unit": "logits rows/s", "cores": 1, "kind": "oracle",
                               "sample": f"the same 8 rows, {reps} repetitions, one thread",
                               "host": host_cpu()}
    print(json.dumps(out), flush=True)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def alg_bytes_flops(wl):
    """Algorithmic HBM bytes and flops of verify, commit and conv for one step."""
    opb = 4 if wl.op_dtype == 0 else 2
    grp = wl.h_v // wl.h_k
    hn = wl.head_node_updates
    mat = wl.d_k * wl.d_v * 4
    inst = wl.n_req * wl.n_layers * wl.h_v
    per_hn = (2 * wl.d_k * opb) / grp + wl.d_v * opb + 8 + wl.d_v * opb  # q,k shared; v; g,beta; o
    v_bytes = hn * per_hn + inst * mat
    v_flops = hn * 6 * wl.d_k * wl.d_v
    plen = sum(min(int(oracle_depth(p, a)), wl.max_path) for p, a in zip(wl.parents, wl.accepted))
    c_upd = plen * wl.n_layers * wl.h_v
    active = sum(1 for p, a in zip(wl.parents, wl.accepted) if a >= 0)
    c_bytes = active * wl.n_layers * wl.h_v * 2 * mat + c_upd * ((wl.d_k * opb) / grp + wl.d_v * opb + 8)
    c_flops = c_upd * 4 * wl.d_k * wl.d_v
    # publication folded into the next verification: the state is read there anyway, so
    # what it adds is the state written back and the path's operand rows
    pub_bytes = c_bytes - active * wl.n_layers * wl.h_v * mat
    # conv history publication (up to three x rows of the path read, three entries
    # written per request and layer), in the commit or deferred into the next conv
    hist_pub_bytes = active * wl.n_layers * 3 * wl.channels * opb * 2
    # x read and y written per (layer, node), the committed history read per (request,
    # layer), four fp32 taps per (layer, channel)
    conv_bytes = (wl.total_nodes * wl.n_layers * wl.channels * opb * 2
                  + wl.n_req * wl.n_layers * 3 * wl.channels * opb + wl.n_layers * wl.channels * 16)
    # conv fused into the verification (deferred): the verify bytes (its q, k, v read as
    # x channels), the publication, the history read and written, the taps; no y
    fused_bytes = (v_bytes + pub_bytes + wl.n_req * wl.n_layers * 3 * wl.channels * opb
                   + active * wl.n_layers * 3 * wl.channels * opb + wl.n_layers * wl.channels * 16)
    return dict(verify_bytes=v_bytes, verify_flops=v_flops, commit_bytes=c_bytes, pub_bytes=pub_bytes,
                commit_flops=c_flops, conv_bytes=conv_bytes, commit_updates=c_upd,
                hist_pub_bytes=hist_pub_bytes, fused_bytes=fused_bytes)


def oracle_depth(parent, a):
    if a < 0:
        return 0
    d, x = 0, int(a)
    while x != -1:
        d += 1
        x = int(parent[x])
    return d


def cpu_baseline(wl, budget_s=12.0):
    """fp64 oracle (conv + verify + commit) on the first k layers of the workload, k chosen
    so that the run takes about budget_s seconds, with OpenMP over the host cores; scaled
    to head-node updates/s. Also the same oracle on one thread over one layer."""
    import numpy as np

    import oracle
    from lumo_synth import configs

    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)

    def sub(k):
        a = wl.arrays
        arr = {"q": a["q"][:k], "k": a["k"][:k], "v": a["v"][:k], "g": a["g"][:k],
               "beta": a["beta"][:k], "state0": np.ascontiguousarray(a["state0"][:, :k]),
               "x": a["x"][:k], "hist": np.ascontiguousarray(a["hist"][:, :k]), "w": a["w"][:k]}
        return configs.Workload(**{**wl.__dict__, "n_layers": k, "arrays": arr})

    def run(k, nt):
        w = sub(k)
        t0 = time.perf_counter()
        oracle.conv_all(w)
        oracle.verify_all(w, n_threads=nt)
        oracle.commit(w, n_threads=nt)
        return time.perf_counter() - t0, w.head_node_updates

    t1, hn1 = run(1, threads)
    k = 1
    if t1 < budget_s and wl.n_layers > 1:
        k = int(min(wl.n_layers, max(1, budget_s // max(t1, 1e-3))))
        t1, hn1 = run(k, threads) if k > 1 else (t1, hn1)
    ts, hns = run(1, 1)
    return {"value": hn1 / t1, "unit": "head-node updates/s", "cores": threads, "kind": "oracle",
            "sample": f"conv + verify + commit of {k} of {wl.n_layers} layers "
                      f"({hn1} head-node updates), all requests and heads, {t1:.1f} s",
            "one_thread": {"value": hns / ts, "sample": f"1 layer ({hns} head-node updates), {ts:.1f} s"},
            "host": host_cpu()}


def per_layer_launches(args, n_layers):
    """Library calls per per-layer step: conv and verify per layer (one fused call with
    --fused), and the commit."""
    return (1 if args.fused else 2) * n_layers + 1


def per_layer_graph_ms(args, st, stream):
    """The step as the paper's per-layer structure runs it: for every layer its own conv
    and verify calls (n_layers = 1), each layer with its own state bank
    [req][1][h_v][d_k][d_v] and conv history [req][1][3][C], the per-node tensors sliced
    by layer. The commit is one launch for all layers: it derives the accepted path and
    publishes it into every layer's conv history (lumo_gdn_commit_hist_layers). The
    states are published by the verification launches: layer 0's verification publishes
    its own, and every layer's verification runs in one launch with the publication
    into the next layer's state bank (lumo_tree_gdn_verify_pending_pair), so that the
    publication runs beside the verification instead of before it. With --fused one
    call per layer does the conv, both publications and the verification, and the
    commit only derives the path. Ten steps are captured in one graph and replayed.
    Returns ms per step."""
    import numpy as np
    import torch

    import paper_2609_23900_amd as L

    d = st.dims
    nl = d.n_layers
    d1 = L.dims(d.n_req, 1, d.h_k, d.h_v, d.d_k, d.d_v, d.op_dtype)
    states = [st.state[:, l:l + 1].contiguous() for l in range(nl)]
    hists = [st.hist[:, l:l + 1].contiguous() for l in range(nl)]

    bias = [None] * nl if st.bias is None else [st.bias[l] for l in range(nl)]
    xs = [st.x[l] for l in range(nl)]
    # each layer's gate parameters (raw gates): the one-layer calls read row 0
    preps = [None] * nl if st.prep is None else [
        L.Prep(st.prep.c.flags, st.prep.c.qk_eps, None if st.prep.a_log is None else st.prep.a_log[l:l + 1],
               None if st.prep.dt_bias is None else st.prep.dt_bias[l:l + 1]) for l in range(nl)]
    empty = L.TreeDesc.build(np.zeros(d.n_req + 1, np.int32), np.zeros(0, np.int32), np.ones(d.n_req, np.int32),
                             L.LUMO_POLICY_WY)
    calls = []  # (layer l's verification, the publication into layer l + 1's bank)
    for l in range(nl):
        t = {key: st.t[key][l] for key in ("q", "k", "v", "g", "beta")}
        calls.append((
            L.pending_call(d1, st.desc, t["q"], t["k"], t["v"], t["g"], t["beta"], states[l], st.o[l],
                           st.desc if l == 0 else empty, st.max_path, st.path_out, st.path_len, t["k"], t["v"],
                           t["g"], t["beta"], preps[l]),
            L.pending_call(d1, empty, None, None, None, None, None, states[l], None, st.desc, st.max_path,
                           st.path_out, st.path_len, t["k"], t["v"], t["g"], t["beta"], preps[l])))

    def one_step():
        for l in range(nl):
            x, y, w = st.x[l], st.y[l], st.w[l]
            g, b = st.t["g"][l], st.t["beta"][l]
            if args.fused:  # conv, publications and verification of the layer in one call
                L.lumo_tree_gdn_verify_conv_pending(d1, st.desc, st.channels, x, hists[l], w, bias[l], st.act, g, b,
                                                    states[l], st.o[l], st.desc, st.max_path, st.path_out,
                                                    st.path_len, x, g, b, None, preps[l])
                continue
            L.lumo_tree_conv_gather(d1, st.desc, st.channels, x, hists[l], w, bias[l], st.act, y)
            L.lumo_tree_gdn_verify_pending_pair(calls[l][0], calls[l + 1][1] if l + 1 < nl else None)
        if args.fused:
            st.commit(None, defer=True, with_conv=False)
        else:
            L.lumo_gdn_commit_hist_layers(d, st.desc, st.max_path, st.accepted, st.path_out, st.path_len,
                                          st.channels, xs, hists)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        one_step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    per = 10
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(per):
            one_step()
    g.replay()
    torch.cuda.synchronize()
    reps = max(1, args.steps // per)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / (reps * per)
    log(f"[bench] per-layer graph-replayed step {ms:.4f} ms ({per_layer_launches(args, nl)} launches per step)")
    del g
    return ms


def arithmetic_label(wl, policy, args):
    """What the timed path computes in: operand and output type, state type, and where
    the O(d^2) products run."""
    import paper_2609_23900_amd as L
    ops_t = "bf16" if wl.op_dtype == 1 else "f32"
    if policy == L.LUMO_POLICY_WY and wl.op_dtype == 0:
        return f"{ops_t} operands/outputs, f32 state; WY form on the vector ALUs in f32"
    if policy == L.LUMO_POLICY_WY:
        core = "R0.[K|Q] on bf16 MFMA with R0 split into bf16 hi+lo (16 significant bits), f32 accumulate"
        if args.fused:
            core = "tree conv in f32 (one bf16 cast); " + core
        return f"{ops_t} operands/outputs, f32 state and recurrence; {core}"
    return f"{ops_t} operands/outputs, f32 state; f32 VALU recurrence"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="batched")
    ap.add_argument("--policy", default="wy")
    ap.add_argument("--commit", choices=("deferred", "eager"), default=None,
                    help="deferred (default where the workload's shapes allow it) or eager")
    ap.add_argument("--prep", action="store_true",
                    help="prepare operands in the kernels (query/key normalisation, gates from raw "
                         "inputs; wy policy): g and beta are then read as raw inputs")
    ap.add_argument("--f32", action="store_true",
                    help="fp32 operands and outputs (the wy policy then runs its vector-ALU kernel, and the "
                         "commit replays eagerly: the deferred publication lives in the matrix-core kernel)")
    ap.add_argument("--copy-probe", action="store_true", help="only run the counter-calibration copy")
    ap.add_argument("--attention", action="store_true", help="only run the tree-attention benchmark")
    ap.add_argument("--select", action="store_true", help="only run the draft-selection benchmark")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle leg")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--no-copy", action="store_true", help="skip the device-copy reference rate")
    ap.add_argument("--fused", action="store_true",
                    help="the conv fused into the verification (one kernel per step besides the path "
                         "derivation; wy policy, deferred commit)")
    ap.add_argument("--per-layer", action="store_true",
                    help="also time the step as one call per layer (conv and verify of each layer "
                         "with its own state and history bank, one path derivation), all captured in "
                         "one graph (wy policy, deferred commit)")
    ap.add_argument("--eager", action="store_true",
                    help="time the K steps as launched from Python (default: the K steps replayed from a "
                         "captured graph of ten steps, so Python's launch cost is not timed); the stage "
                         "breakdown always comes from an eager pass of K steps")
    ap.add_argument("--graph", action="store_true", help="(the default; kept for old command lines)")
    args = ap.parse_args()
    args.commit_explicit = args.commit is not None
    args.commit = args.commit or "deferred"
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the step shards "
              "by request with no cross-GPU exchange; see the design notes)", file=sys.stderr)
        sys.exit(2)

    if args.copy_probe:
        copy_probe()
        return
    if args.select:
        select_bench(args)
        return
    if args.attention:
        attention_bench(args)
        return

    import numpy as np
    import torch

    import paper_2609_23900_amd as L
    from paper_2609_23900_amd.step import GdnTreeStep
    from lumo_synth import configs

    policy = L.POLICIES[args.policy]
    deferred = args.commit == "deferred" and policy == L.LUMO_POLICY_WY and not args.f32
    if args.fused and not deferred:
        sys.exit("--fused needs the wy policy and the deferred commit")
    if args.fused and not args.prep:
        # conv outputs are not unit-norm keys: as in the model, the queries and keys are
        # normalised after the conv (in the kernel), else the replays diverge
        sys.exit("--fused needs --prep (query/key normalisation of the conv outputs)")
    log(f"[bench] generating {args.config}")
    wl = configs.build(args.config, op_dtype=0) if args.f32 else configs.build(args.config)
    if deferred and not (wl.op_dtype == 1 and wl.d_k == 128 and wl.d_v == 128):
        # the deferred publication runs in the matrix-core WY kernel: bf16, d_k = d_v = 128
        if args.fused or args.per_layer or args.commit_explicit:
            sys.exit(f"the deferred commit needs bf16 operands with d_k = d_v = 128 ({args.config} is not)")
        deferred = False
        args.commit = "eager"
        log(f"[bench] {args.config}: eager commit (the deferred publication takes bf16 operands with d = 128)")
    log(f"[bench] uploading; policy {args.policy}")
    prep = None
    if args.prep:
        if policy != L.LUMO_POLICY_WY:
            sys.exit("--prep needs the wy policy")
        rng = np.random.default_rng(5)
        a_log = torch.from_numpy((0.5 * rng.standard_normal((wl.n_layers, wl.h_v))).astype(np.float32)).cuda()
        dt_bias = torch.from_numpy(rng.standard_normal((wl.n_layers, wl.h_v)).astype(np.float32)).cuda()
        prep = L.Prep(L.LUMO_PREP_QK_NORM | L.LUMO_PREP_RAW_GATES, 1e-6, a_log, dt_bias)
    st = GdnTreeStep.from_workload(wl, policy=policy, keep_state0=False, prep=prep)
    stream = torch.cuda.current_stream()

    # The deferred conv publishes the previous step's history in its own launch only
    # when it takes the depth-first kernel (bf16, trees of at most 16 levels, at least
    # four blocks per CU); otherwise it needs a launch of its own for it, and the commit
    # publishes the history instead, in the launch that derives the path.
    dfs_conv = (not args.f32 and st.plan.max_depth <= 16
                and wl.n_req * wl.n_layers * ((wl.channels + 2047) // 2048) >= 4 * 256)
    hist_in_commit = deferred and not args.fused and not dfs_conv

    def step(ev=None, s=stream):  # s=None: the current stream (a graph's capture stream)
        if ev is not None:
            ev[0].record(stream)
        if args.fused:
            pass  # the conv runs inside the verification
        elif deferred and not hist_in_commit:
            st.conv_pending(st, s)  # publishes the previous step's history, then the conv
        else:
            st.conv(s)
        if ev is not None:
            ev[1].record(stream)
        if args.fused:
            st.verify_conv_pending(st, s)  # publishes history and path, conv, verification
        elif deferred:
            st.verify_pending(st, s)  # publishes the previous step's path, then verifies
        else:
            st.verify(s)
        if ev is not None:
            ev[2].record(stream)
        st.commit(s, defer=deferred, with_conv=not deferred or hist_in_commit)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup done; timing {args.steps} steps")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(args.steps):
        step(evs[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    conv_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    ver_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    com_ms = sum(e[2].elapsed_time(e[3]) for e in evs) / args.steps
    ms_step = total_ms / args.steps
    step_dist = pct([e[0].elapsed_time(e[3]) for e in evs])
    ver_dist = pct([e[1].elapsed_time(e[2]) for e in evs])
    log(f"[bench] step {ms_step:.3f} ms (conv {conv_ms:.3f}, verify {ver_ms:.3f}, commit {com_ms:.3f})")
    graph_ms = None
    if not args.eager:
        per = 10 if args.steps % 10 == 0 else 1  # exactly K steps in the timed replays
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step(s=None)  # one eager step on the capture's stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(per):
                step(s=None)
        g.replay()
        torch.cuda.synchronize()
        reps = args.steps // per
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(reps):
            g.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        graph_ms = g0.elapsed_time(g1) / (reps * per)
        log(f"[bench] graph-replayed step {graph_ms:.4f} ms")
        del g
    assert torch.isfinite(st.state).all().item(), "non-finite state"

    ab = alg_bytes_flops(wl)
    hn = wl.head_node_updates
    if policy == L.LUMO_POLICY_WY:
        vb = ab["fused_bytes"] if args.fused else ab["verify_bytes"] + (ab["pub_bytes"] if deferred else 0)
        ach = vb / (ver_ms * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": None}
    else:
        vb = ab["verify_bytes"]
        ach = ab["verify_flops"] / (ver_ms * 1e-3) / 1e12
        roof = {"bound": "alu", "achieved": round(ach, 2), "peak": PEAK_VALU_F32_TFS,
                "unit": "TFLOP/s", "frac": round(ach / PEAK_VALU_F32_TFS, 4), "traffic": None}
    mode = "deferred" if deferred else "eager"
    if policy == L.LUMO_POLICY_WY and wl.op_dtype == 0:  # the vector-ALU WY kernel
        tr = recorded_traffic("wyv", args.config + "_f32", mode)
    else:
        tr = recorded_traffic(args.policy, args.config + ("_f32" if wl.op_dtype == 0 else ""),
                              "fused" if args.fused else mode)
    if tr is not None:
        roof["traffic"] = {"fetch_bytes": tr["fetch_bytes"], "write_bytes": tr["write_bytes"],
                           "total_bytes": tr["fetch_bytes"] + tr["write_bytes"], "unit": "B per verify call",
                           "source": "profiles/traffic.json"}
    roof["kernel"] = ("tree conv + verify + publication of the previous path (one kernel)" if args.fused
                      else "verify + publication of the previous path" if deferred
                      else "verify (WY form on the vector ALUs)" if policy == L.LUMO_POLICY_WY and wl.op_dtype == 0
                      else "verify")
    roof["per_launch"] = (f"{ab['verify_flops'] / 1e9:.2f} GFLOP, {vb / 1e6:.1f} MB algorithmic per verify call")
    kernels = {
        "conv_gather_ms": round(conv_ms, 4),
        "conv_hbm_frac": None if args.fused else round((ab["conv_bytes"] + (ab["hist_pub_bytes"] if deferred else 0))
                                                       / (conv_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "verify_ms": round(ver_ms, 4),
        "commit_ms": round(com_ms, 4),
        "step_ms_p10_p50_p90": step_dist,
        "verify_ms_p10_p50_p90": ver_dist,
    }
    kernels["eager_step_ms"] = round(ms_step, 4)
    if graph_ms is not None:
        kernels["graph_step_ms"] = round(graph_ms, 4)
        ms_step = graph_ms  # the headline: K steps replayed from captured graphs
    if args.per_layer:
        if not deferred:
            sys.exit("--per-layer needs the wy policy and the deferred commit")
        pl_ms = per_layer_graph_ms(args, st, stream)
        kernels["per_layer_graph_step_ms"] = round(pl_ms, 4)
        kernels["per_layer_launches_per_step"] = per_layer_launches(args, wl.n_layers)
    if not deferred:
        kernels["commit_hbm_frac"] = round(ab["commit_bytes"] / (com_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
    out = {
        "metric": METRIC, "value": round(hn / (ms_step * 1e-3), 1), "unit": "head-node updates/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": arithmetic_label(wl, policy, args),
        "data": "synthetic (seeded trees and operands shaped like the paper's workloads)",
        "config": {"workload": f"{args.config}: " + (WORKLOAD_TEXT[args.config].replace("bf16 operands", "fp32 operands")
                                                      if wl.op_dtype == 0 else WORKLOAD_TEXT[args.config]),
                   "policy": args.policy, "commit": mode, "conv": "fused into verify" if args.fused else "separate",
                   "conv_history_published_in": ("verify" if args.fused else "conv" if deferred and not hist_in_commit
                                                 else "commit"),
                   "head_node_updates_per_step": hn,
                   "operand_prep": "qk_norm+raw_gates" if args.prep else "none",
                   "operands": "bf16" if wl.op_dtype == 1 else "f32"},
        "roofline": roof, "kernels": kernels,
    }
    if not args.no_copy:
        cms, cgbs = copy_rate()
        roof["practical"] = {"copy_GBps": round(cgbs, 1), "frac_of_copy": round(roof["achieved"] / cgbs, 4)
                             if roof["unit"] == "GB/s" else None,
                             "what": "plain 1 GiB device copy (read + write) timed in this run"}
    if not args.no_cpu:
        log("[bench] CPU oracle leg")
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
