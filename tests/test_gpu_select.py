"""Fused draft selection on the GPU (Sec. V-D) against the oracle, through the C ABI.

The outputs are indices, so they must match bit for bit: the spine (argmax, lowest
maximal index) and the k ordered candidates (top-k under either tie direction), for
float32 and bfloat16 logits, over rows with heavy ties, NaN with any payload, +-inf
and +-0, ragged vocabularies, padded row strides whose padding holds NaN, and five
block-count settings per case (one part, two, three, the suggested count, and more
parts than the row has 16-byte vectors), all sharing one workspace that is filled with
garbage before each case. A captured graph of four selection levels is replayed 24 times on
fresh logits, every replay checked. The paper geometry (248,320 logits per row) is
checked on every row.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
from lumo_synth import operands as ops  # noqa: E402

pytestmark = pytest.mark.gpu

SPECIAL = np.array([np.nan, np.inf, -np.inf, 1.5, 1.5, -0.0, 0.0, 2.0, -3.0], np.float32)
VOCABS = [1, 2, 3, 4, 5, 7, 8, 9, 16, 31, 33, 64, 100, 257, 1000, 4097, 10007]
PAPER_VOCAB = 248320


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_23900_amd as L
    return L


def _nan_payloads(rng, shape):
    """float32 NaNs with random payloads and either sign."""
    bits = (rng.integers(1, 1 << 22, size=shape, dtype=np.int64) | 0x7f800000
            | (rng.integers(0, 2, size=shape, dtype=np.int64) << 31)).astype(np.uint32)
    return bits.view(np.float32)


def gen_logits(rng, kind, rows, vocab):
    """float32 logits [rows][vocab] of one distribution family."""
    if kind == "normal":
        return (rng.standard_normal((rows, vocab)) * 3).astype(np.float32)
    if kind == "levels":  # few distinct values: ties everywhere
        x = rng.integers(0, 5, size=(rows, vocab)).astype(np.float32) * 0.25 - 1.0
        x[rng.random((rows, vocab)) < 0.05] = -np.inf
        return x
    if kind == "special":
        x = SPECIAL[rng.integers(0, len(SPECIAL), size=(rows, vocab))]
        m = rng.random((rows, vocab)) < 0.5
        x = np.where(m, x, rng.standard_normal((rows, vocab)).astype(np.float32))
        nanm = np.isnan(x)
        x[nanm] = _nan_payloads(rng, int(nanm.sum()))
        return x.astype(np.float32)
    if kind == "equal":
        return np.full((rows, vocab), -0.5, np.float32)
    if kind == "max_last":  # the maximum (tied) in the row's last entries
        x = (rng.standard_normal((rows, vocab))).astype(np.float32)
        x[:, -1] = 9.0
        if vocab > 2:
            x[:, -3] = 9.0
        return x
    if kind == "zeros":  # -0 and +0 only: all equal
        return np.where(rng.random((rows, vocab)) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    raise ValueError(kind)


KINDS = ["normal", "levels", "special", "equal", "max_last", "zeros"]


def to_device(x32, dtype, ld):
    """Logits on the device as [rows][ld] (padding columns hold NaN) plus the numpy
    values the oracle ranks (bf16 bit patterns for bf16)."""
    rows, vocab = x32.shape
    if dtype == ops.BF16:
        bits = ops.to_bf16_bits(x32)
        nanm = np.isnan(x32)
        # keep NaN payload diversity in bf16: random payload bits in the low 7 bits
        bits[nanm] = (bits[nanm] & 0xff80) | 0x0040 | (np.arange(int(nanm.sum())) % 63).astype(np.uint16)
        full = np.full((rows, ld), 0x7fc1, np.uint16)
        full[:, :vocab] = bits
        t = torch.from_numpy(full.view(np.int16)).cuda().view(torch.bfloat16)
        return t, bits
    full = np.full((rows, ld), np.nan, np.float32)
    full[:, :vocab] = x32
    return torch.from_numpy(full).cuda(), x32


def run_gpu(L, t, vocab, k, ties, n_split, ws):
    rows = t.shape[0]
    spine = torch.full((rows,), -7, dtype=torch.int32, device="cuda")
    cand = torch.full((rows, k), -7, dtype=torch.int32, device="cuda")
    L.lumo_draft_select(t, k, ties, spine, cand, n_split, ws if n_split > 1 else None, vocab=vocab)
    return spine.cpu().numpy(), cand.cpu().numpy()


def splits_for(L, rows, vocab, dtype):
    per = 8 if dtype == ops.BF16 else 4
    nvec = (vocab + per - 1) // per
    return sorted({1, 2, 3, L.lumo_draft_select_splits(rows, vocab, dtype), min(4096, nvec + 5)})


def test_select_cases_exact(lib):
    L = lib
    rng = np.random.default_rng(2609)
    ws = torch.zeros(8 << 20, dtype=torch.uint8, device="cuda")
    n_cases = n_runs = 0
    for dtype in (ops.F32, ops.BF16):
        for vocab in VOCABS:
            for kind in KINDS:
                rows = int(rng.integers(1, 6))
                ld = vocab + int(rng.choice([0, 0, 1, 5, 8]))
                x32 = gen_logits(rng, kind, rows, vocab)
                t, ref_in = to_device(x32, dtype, ld)
                ws.fill_(0xA5)  # no initial contents are needed
                for ties in (0, 1):
                    for k in sorted({1, min(3, vocab), min(8, vocab)}):
                        want = oracle.draft_select(ref_in, k=k, op_dtype=dtype, ties=ties)
                        n_cases += 1
                        for n_split in splits_for(L, rows, vocab, dtype):
                            assert L.lumo_draft_select_workspace_bytes(rows, k, n_split) <= ws.numel()
                            got = run_gpu(L, t, vocab, k, ties, n_split, ws)
                            ctx = (dtype, vocab, ld, kind, rows, ties, k, n_split)
                            assert np.array_equal(got[0], want[0]), ("spine", ctx, got[0], want[0])
                            assert np.array_equal(got[1], want[1]), ("cand", ctx, got[1], want[1])
                            n_runs += 1
    print(f"{n_cases} cases, {n_runs} configurations, all exact")
    assert n_cases >= 1000


@pytest.mark.parametrize("dtype", [ops.F32, ops.BF16])
def test_select_paper_vocabulary(lib, dtype):
    """8 rows (one per request at one drafting depth) of 248,320 logits, k = 3, every
    row, both tie directions, heavy-tie and plain distributions, suggested split."""
    L = lib
    rng = np.random.default_rng(11 + dtype)
    rows = 8
    n_split = L.lumo_draft_select_splits(rows, PAPER_VOCAB, dtype)
    ws = torch.zeros(L.lumo_draft_select_workspace_bytes(rows, 3, n_split), dtype=torch.uint8, device="cuda")
    for kind in ("normal", "levels", "special"):
        x32 = gen_logits(rng, kind, rows, PAPER_VOCAB)
        t, ref_in = to_device(x32, dtype, PAPER_VOCAB)
        for ties in (0, 1):
            want = oracle.draft_select(ref_in, k=3, op_dtype=dtype, ties=ties)
            got = run_gpu(L, t, PAPER_VOCAB, 3, ties, n_split, ws)
            assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1]), (kind, ties)


def test_select_tie_direction_is_observable(lib):
    """Negative control: on a row of equal logits the two tie directions give different
    candidates, so a kernel that ignored `ties` would fail the exact checks."""
    L = lib
    x = torch.full((2, 1000), 0.25, dtype=torch.float32, device="cuda")
    ws = torch.zeros(4096, dtype=torch.uint8, device="cuda")
    a = run_gpu(L, x, 1000, 3, 0, 3, ws)
    b = run_gpu(L, x, 1000, 3, 1, 3, ws)
    assert a[1].tolist() == [[0, 1, 2]] * 2 and b[1].tolist() == [[999, 998, 997]] * 2
    assert a[0].tolist() == b[0].tolist() == [0, 0]


def test_select_large_batch(lib):
    """64 rows of bf16 logits (the chain-and-tree mix's request count), sampled rows
    checked, suggested split, repeated calls identical."""
    L = lib
    rng = np.random.default_rng(5)
    rows, k = 64, 3
    x32 = gen_logits(rng, "normal", rows, PAPER_VOCAB)
    t, ref_in = to_device(x32, ops.BF16, PAPER_VOCAB)
    n_split = L.lumo_draft_select_splits(rows, PAPER_VOCAB, ops.BF16)
    ws = torch.zeros(L.lumo_draft_select_workspace_bytes(rows, k, n_split), dtype=torch.uint8, device="cuda")
    got = run_gpu(L, t, PAPER_VOCAB, k, 1, n_split, ws)
    again = run_gpu(L, t, PAPER_VOCAB, k, 1, n_split, ws)
    assert np.array_equal(got[0], again[0]) and np.array_equal(got[1], again[1])
    sample = [0, 1, 17, 40, 63]
    want = oracle.draft_select(ref_in[sample], k=k, op_dtype=ops.BF16, ties=1)
    assert np.array_equal(got[0][sample], want[0]) and np.array_equal(got[1][sample], want[1])


def test_select_graph_replays(lib):
    """A captured four-level selection graph (one call per drafting depth, 8 rows of
    248,320 float32 logits each, k = 3) replayed 24 times; before each replay every
    level's logits are overwritten with fresh values, and every replay's outputs must
    equal the oracle's."""
    L = lib
    rng = np.random.default_rng(24)
    rows, k, levels, ties = 8, 3, 4, 1
    n_split = L.lumo_draft_select_splits(rows, PAPER_VOCAB, ops.F32)
    logits = [torch.zeros((rows, PAPER_VOCAB), dtype=torch.float32, device="cuda") for _ in range(levels)]
    spine = [torch.zeros(rows, dtype=torch.int32, device="cuda") for _ in range(levels)]
    cand = [torch.zeros((rows, k), dtype=torch.int32, device="cuda") for _ in range(levels)]
    ws = torch.zeros(L.lumo_draft_select_workspace_bytes(rows, k, n_split), dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):  # one eager run before capture
        for lv in range(levels):
            L.lumo_draft_select(logits[lv], k, ties, spine[lv], cand[lv], n_split, ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for lv in range(levels):
            L.lumo_draft_select(logits[lv], k, ties, spine[lv], cand[lv], n_split, ws)
    torch.cuda.synchronize()
    for rep in range(24):
        host = []
        for lv in range(levels):
            kind = ("normal", "levels", "special")[(rep + lv) % 3]
            x = gen_logits(rng, kind, rows, PAPER_VOCAB)
            host.append(x)
            logits[lv].copy_(torch.from_numpy(x))
            spine[lv].fill_(-1)
            cand[lv].fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for lv in range(levels):
            want = oracle.draft_select(host[lv], k=k, op_dtype=ops.F32, ties=ties)
            assert np.array_equal(spine[lv].cpu().numpy(), want[0]), (rep, lv)
            assert np.array_equal(cand[lv].cpu().numpy(), want[1]), (rep, lv)
