"""Pins of trees from arbitrary parent arrays (third-level cascade, sec. 4.3;
independent resampling)."""

import numpy as np
import pytest

from oracle.tree import (build_tree, resample_parents, third_level_parents, tree_from_parents)

GOLDEN = "tests/golden/tree_third_level_gamma5.txt"


def read_golden():
    rows = {"anc": []}
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if not line:
            continue
        key, *vals = line.split()
        if key == "anc":
            rows["anc"].append({int(v) for v in vals})
        else:
            rows[key] = [int(v) for v in vals]
    return rows


def test_hand_worked_third_level_tree():
    g = read_golden()
    parent = third_level_parents(5, [2], [3])
    assert parent == g["parent"]
    t = tree_from_parents(parent)
    assert t.position == g["depth"]
    assert t.path == g["path"]
    assert t.ancestors == g["anc"]
    assert t.p == [2, 3]                       # re-anchor depths of the two extra paths


@pytest.mark.parametrize("B,p", [(16, []), (16, [3, 9]), (16, [1, 5, 12, 15]), (8, list(range(1, 8)))])
def test_canonical_parents_reproduce_the_canonical_tree(B, p):
    c = build_tree(B, p)
    g = tree_from_parents(c.parent, B)
    assert g.position == c.position          # depth by walking == block position by construction
    assert g.path == c.path                  # path-start rule == branch numbering
    assert g.p == c.p
    assert np.array_equal(g.packed_mask(), c.packed_mask())


def test_resample_chains_closed_form():
    B, chains = 6, 3
    t = tree_from_parents(resample_parents(B, chains))
    assert t.N == 1 + chains * (B - 1)
    for n in range(1, t.N):
        k, d = (n - 1) // (B - 1), (n - 1) % (B - 1) + 1
        # root plus the chain's own nodes of depth <= d
        assert t.ancestors[n] == {0} | {1 + k * (B - 1) + j for j in range(d)}
        assert t.position[n] == d and t.path[n] == k
    assert t.p == [1] * (chains - 1)


def test_random_tree_invariants():
    rng = np.random.default_rng(4)
    for _ in range(50):
        N = int(rng.integers(1, 120))
        parent = [-1] + [int(rng.integers(0, n)) for n in range(1, N)]
        t = tree_from_parents(parent)
        for n in range(N):
            assert len(t.ancestors[n]) == t.position[n] + 1
            if n:
                assert t.ancestors[parent[n]] < t.ancestors[n]
        W = (N + 31) // 32
        m = t.packed_mask(W)
        assert all(bin(int.from_bytes(m[n].tobytes(), "little")).count("1") == t.position[n] + 1 for n in range(N))


def test_invalid_parents_rejected():
    with pytest.raises(ValueError):
        tree_from_parents([0, 0])
    with pytest.raises(ValueError):
        tree_from_parents([-1, 1])
    with pytest.raises(ValueError):
        third_level_parents(5, [2], [2])
