"""Pins of the acceptance oracle: hand-worked cases, brute force, closed forms."""

import itertools

import numpy as np
import pytest

from oracle.accept import accept_by_alive, accept_by_paths
from oracle.tree import build_tree
from tests.closed_forms import expected_accept_len
from tests.golden_io import read_accept, read_tree


@pytest.mark.parametrize("how", [accept_by_paths, accept_by_alive])
def test_hand_worked_cases(how):
    g = read_tree("tree_gamma4_p12.txt")
    t = build_tree(g["B"], g["p"])
    for case in read_accept("accept_gamma4_p12.txt"):
        r = how(t, case["draft"], case["argmax"])
        assert (r.L, r.best_path, r.node) == (case["L"], case["path"], case["node"]), case["name"]
        assert r.path_nodes == case["nodes"], case["name"]
        assert r.tokens == case["tokens"], case["name"]


def tokens_for_pattern(t, pattern):
    """Tokens realising a match pattern: argmax[n] = n, a match copies it."""
    argmax = list(range(1000, 1000 + t.N))
    draft = [0] * t.N
    for c in range(1, t.N):
        draft[c] = argmax[t.parent[c]] if pattern[c - 1] else 7
    return draft, argmax


def test_brute_force_all_tiny_trees():
    """Every tree with B <= 5 and every match pattern: both derivations agree, and
    the exact expectation over patterns equals the independent closed form."""
    cases = 0
    for B in range(2, 6):
        for K in range(B):
            for p in itertools.combinations(range(1, B), K):
                t = build_tree(B, p)
                nm = t.N - 1
                for q in (0.7,):
                    e_exact = 0.0
                    for bits in itertools.product((0, 1), repeat=nm):
                        draft, argmax = tokens_for_pattern(t, bits)
                        a = accept_by_paths(t, draft, argmax)
                        b = accept_by_alive(t, draft, argmax)
                        assert (a.L, a.best_path, a.node, a.path_nodes, a.tokens) == \
                               (b.L, b.best_path, b.node, b.path_nodes, b.tokens)
                        k = sum(bits)
                        e_exact += q ** k * (1 - q) ** (nm - k) * a.L
                        cases += 1
                    assert e_exact == pytest.approx(expected_accept_len(B, p, q), abs=1e-12)
    assert cases == 37866


@pytest.mark.parametrize("p,expect", [([], 2.3223), ([1, 2], 4.4185), ([1, 2, 3, 4], 5.1366),
                                      ([5, 9, 12, 14], 2.7200)])
def test_closed_form_reference_values(p, expect):
    # B = 16, q = 0.7; the chain value is the geometric sum of 0.7^j, j = 1..15
    assert expected_accept_len(16, p, 0.7) == pytest.approx(expect, abs=5e-5)
    if not p:
        assert expected_accept_len(16, p, 0.7) == pytest.approx(sum(0.7 ** j for j in range(1, 16)), abs=1e-12)


def test_derivations_agree_at_block_16():
    rng = np.random.default_rng(11)
    for _ in range(300):
        K = int(rng.integers(0, 9))
        p = rng.choice(np.arange(1, 16), size=K, replace=False)
        t = build_tree(16, p)
        argmax = rng.integers(0, 5, size=t.N)         # small vocab: many matches and ties
        draft = rng.integers(0, 5, size=t.N)
        a, b = accept_by_paths(t, draft, argmax), accept_by_alive(t, draft, argmax)
        assert (a.L, a.best_path, a.node, a.path_nodes, a.tokens) == \
               (b.L, b.best_path, b.node, b.path_nodes, b.tokens)
        assert len(a.tokens) == a.L + 1 and len(a.path_nodes) == a.L + 1
