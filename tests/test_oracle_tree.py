"""Pins of the tree oracle: hand-written fixtures, closed forms, special cases."""

import itertools

import numpy as np
import pytest

from oracle.tree import build_tree, mask_words, validate
from tests.golden_io import read_tree


@pytest.mark.parametrize("name", ["tree_gamma4_p12.txt", "tree_gamma6_p245.txt"])
def test_hand_written_trees(name):
    g = read_tree(name)
    t = build_tree(g["B"], g["p"])
    assert t.N == len(g["nodes"])
    for row in g["nodes"]:
        n = row["node"]
        assert t.position[n] == row["position"], n
        assert t.path[n] == row["path"], n
        assert t.parent[n] == row["parent"], n
        assert t.ancestors[n] == row["anc"], n
    assert t.path_leaf() == g["leaves"]
    # the packed mask carries exactly the hand-written sets
    pm = t.packed_mask()
    for row in g["nodes"]:
        bits = {m for m in range(32 * pm.shape[1]) if (int(pm[row["node"], m // 32]) >> (m % 32)) & 1}
        assert bits == row["anc"]


def all_subsets(B):
    for K in range(B):
        yield from itertools.combinations(range(1, B), K)


@pytest.mark.parametrize("B", [2, 3, 4, 5, 6, 7, 8])
def test_closed_form_node_count_and_popcount(B):
    for p in all_subsets(B):
        t = build_tree(B, p)
        assert t.N == B + sum(B - x for x in p)
        pm = t.packed_mask()
        for n in range(t.N):
            pop = sum(bin(int(w)).count("1") for w in pm[n])
            assert pop == t.position[n] + 1          # depth + 1 (ancestors incl. self)


def test_chain_is_block_causal():
    # K = 0: the tree is the first-draft block alone, the mask is lower triangular
    for B in (2, 5, 16, 33, 64):
        t = build_tree(B, [])
        assert np.array_equal(t.visible(), np.tril(np.ones((B, B), bool)))


def test_branch_shares_prefix():
    # every branch node sees main nodes 0..p-1 and its own branch up to itself
    rng = np.random.default_rng(0)
    for _ in range(50):
        B = int(rng.integers(2, 40))
        K = int(rng.integers(0, B))
        p = sorted(rng.choice(np.arange(1, B), size=K, replace=False).tolist())
        t = build_tree(B, p)
        off = B
        for k, pk in enumerate(p, start=1):
            for j in range(pk, B):
                n = off + (j - pk)
                assert t.path[n] == k and t.position[n] == j
                expect = set(range(pk)) | set(range(off, n + 1))
                assert t.ancestors[n] == expect
            off += B - pk


def test_mask_width_and_bit_order():
    assert mask_words(16) == 5                       # 136 nodes at most
    assert mask_words(2) == 1 and mask_words(64) == 65
    t = build_tree(16, list(range(1, 16)))
    assert t.N == 136
    pm = t.packed_mask()
    assert pm.shape == (136, 5)
    # the last node (index 135) sees itself: word 4, bit 7
    assert (int(pm[135, 4]) >> 7) & 1 == 1
    assert int(pm[0, 0]) == 1 and all(int(w) == 0 for w in pm[0, 1:])


def test_unsorted_input_is_canonicalised():
    a, b = build_tree(16, [9, 3, 12]), build_tree(16, [3, 9, 12])
    assert a.parent == b.parent and a.p == [3, 9, 12]


@pytest.mark.parametrize("B,p", [(1, []), (4, [0]), (4, [4]), (4, [2, 2]), (3, [1, 2, 1])])
def test_validation(B, p):
    with pytest.raises(ValueError):
        validate(B, p)
