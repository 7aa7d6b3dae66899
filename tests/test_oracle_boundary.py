"""Pins of the rejection-boundary posterior (Eq. 4) and top-K selection (Eq. 5)."""

import numpy as np
import pytest

from oracle.boundary import rejection_posterior, reanchor_positions, top_k_prefixes
from tests.golden_io import read_boundary


def test_hand_worked_example():
    g = read_boundary("boundary_gamma4.txt")
    r = rejection_posterior(g["conf"])
    np.testing.assert_allclose(r, g["r"], atol=1e-15)
    assert top_k_prefixes(r, 2) == g["top2"]
    assert top_k_prefixes(r, 1) == g["top1"]
    assert reanchor_positions(g["conf"], 2) == [i + 1 for i in g["top2"]]


def test_telescoping_sum():
    # exactly-i-accepted events for i = 0..gamma-2 plus all-accepted partition the space
    rng = np.random.default_rng(12)
    for gamma in (2, 4, 16, 32):
        for _ in range(20):
            c = rng.random(gamma - 1)
            r = rejection_posterior(c)
            assert len(r) == gamma - 1
            assert sum(r) + float(np.prod(c)) == pytest.approx(1.0, abs=1e-15)


def test_constant_confidence_is_geometric():
    for c in (0.1, 0.5, 0.9):
        r = rejection_posterior([c] * 15)
        np.testing.assert_allclose(r, [c ** i * (1 - c) for i in range(15)], rtol=1e-14)
        for K in range(0, 16):
            assert top_k_prefixes(r, K) == list(range(K))


def test_ties_go_to_smaller_prefix():
    assert top_k_prefixes([0.2, 0.3, 0.3, 0.2], 1) == [1]
    assert top_k_prefixes([0.2, 0.3, 0.3, 0.2], 3) == [0, 1, 2]


def test_nan_posterior_ranks_last():
    # confidences outside [0, 1]: 0 * (1 - inf) and 0 * inf are NaN, and
    # 0.5 * (1 - inf) is -inf
    r = rejection_posterior([0.0, float("inf"), 0.5])
    assert r[0] == 1.0 and np.isnan(r[1]) and np.isnan(r[2])
    assert top_k_prefixes(r, 2) == [0, 1]
    r = rejection_posterior([0.5, float("inf"), 0.5])
    assert r[:2] == [0.5, -float("inf")] and r[2] == float("inf")
    nan = float("nan")
    assert top_k_prefixes([nan, 0.1, nan, 0.3], 2) == [1, 3]
    assert top_k_prefixes([nan, 0.1, nan, 0.3], 3) == [0, 1, 3]      # first NaN by index
    assert top_k_prefixes([nan, -float("inf"), nan], 2) == [0, 1]     # -inf ranks above NaN
    assert top_k_prefixes([nan] * 4, 4) == [0, 1, 2, 3]
