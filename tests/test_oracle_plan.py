"""Descriptor derivations of the oracle (oracle/plan.py) against the hand-derived
Fig. 1 descriptor and structural properties on random trees."""
import numpy as np
import pytest

from oracle import plan
from lumo_synth import trees
import pins


def test_fig1_descriptor_golden():
    gd = pins.load_golden("fig1_descriptor.json")
    par = gd["parent"]
    assert plan.depth(par) == gd["depth"]
    assert plan.leaves(par) == gd["leaves"]
    assert plan.paths(par) == gd["paths"]
    assert plan.spine(par) == gd["spine"]
    assert plan.slot_map(par) == gd["slot"]
    order = sorted(range(len(par)), key=lambda i: gd["slot"][i])
    assert order == gd["physical_order"]
    path, L = plan.accepted_path(par, gd["accepted"], 4)
    assert path[:L] == gd["accepted_path"] and L == gd["accepted_len"]
    assert path[L:] == [-1] * (4 - L)


def test_fig1_conv_sources():
    par = trees.FIG1_PARENT
    rows = plan.rows_of(par, 0)
    src = plan.conv_sources(par, rows)
    # root: hist 0, 1, 2 then itself
    assert src[0] == [-1, -2, -3, rows[0]]
    # f (depth 3): m, a, c, f
    assert src[6] == [rows[0], rows[1], rows[3], rows[6]]
    # e (depth 2): hist[2], m, b, e
    assert src[5] == [-3, rows[0], rows[2], rows[5]]


@pytest.mark.parametrize("seed", range(20))
def test_random_tree_properties(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 80))
    par = trees.random_tree(rng, n, int(rng.integers(2, 12)) if n > 1 else 1, trees.bmax_uniform(4))
    plan.validate(par)
    slot = plan.slot_map(par)
    assert sorted(slot) == list(range(n))
    sp = plan.spine(par)
    assert [slot[x] for x in sp] == list(range(len(sp)))
    rest = [i for i in range(n) if i not in set(sp)]
    assert [slot[x] for x in rest] == list(range(len(sp), n))
    covered = set()
    for p in plan.paths(par):
        assert p[0] == 0
        for a, b in zip(p, p[1:]):
            assert par[b] == a
        covered.update(p)
    assert covered == set(range(n))
    own = plan.owner_leaf(par)
    for i in range(n):
        assert i in plan.ancestry(par, own[i])


def test_paper_geometry():
    par = trees.paper_geometry_tree()
    assert len(par) == 28
    assert max(plan.depth(par)) == 11          # root + eleven draft levels
    plan.validate(par)


@pytest.mark.parametrize("bad", [[0], [-1, 1], [-1, 2, 0], [-1, -1], [-1, 0, 5]])
def test_validate_rejects(bad):
    with pytest.raises(ValueError):
        plan.validate(bad)


def test_request_without_nodes():
    """An empty request contributes no rows and no sources; its neighbours keep theirs."""
    empty = np.zeros(0, np.int32)
    assert plan.spine(empty) == [] and plan.slot_map(empty) == []
    rows = plan.flat_rows([np.array([-1, 0], np.int32), empty, np.array([-1], np.int32)],
                          np.array([0, 2, 2], np.int32))
    assert rows.tolist() == [0, 1, 2]
