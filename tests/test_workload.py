"""The seeded input generator: determinism, recipe, and the token model."""

import numpy as np
import pytest
import torch

from oracle.accept import accept_by_alive
from oracle.tree import build_tree
from paper_2606_04446_amd import workload as wl
from tests.closed_forms import expected_accept_len


def trees_of(layout):
    trees = [build_tree(layout.spec.B, layout.p[b, :layout.K[b]]) for b in range(layout.batch)]
    ip = np.concatenate([[0], np.cumsum([t.N for t in trees])]).astype(np.int32)
    parent = np.concatenate([t.parent for t in trees]).astype(np.int32)
    return trees, ip, parent


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_layout_recipe(cfg):
    a, b = wl.draw_layout(cfg), wl.draw_layout(cfg)
    assert np.array_equal(a.p, b.p) and np.array_equal(a.page_table, b.page_table)
    spec = wl.WORKLOADS[cfg]
    assert a.batch == spec.batch and (a.K == spec.K).all()
    lo, hi = spec.ctx
    assert ((a.ctx_len >= lo) & (a.ctx_len <= hi)).all()
    for r in range(a.batch):
        row = a.p[r, :a.K[r]]
        assert len(set(row.tolist())) == len(row) and row.min() >= 1 and row.max() <= spec.B - 1
        npg = (a.ctx_len[r] + 15) // 16
        assert (a.page_table[r, :npg] < a.num_pages).all()
    used = np.concatenate([a.page_table[r, :(a.ctx_len[r] + 15) // 16] for r in range(a.batch)])
    assert len(np.unique(used)) == len(used) == a.num_pages   # every page used exactly once


def test_beta_rule_picks_lowest_confidence():
    rng = np.random.default_rng([5, 0])
    conf = rng.beta(5.0, 2.0, size=15)
    p = wl.draw_positions(np.random.default_rng([5, 0]), 16, 4, "beta_lowest")
    lowest = sorted(sorted(range(15), key=lambda j: (conf[j], j))[:4])
    assert p.tolist() == [j + 1 for j in lowest]


def test_tensors_deterministic_and_bf16_rounded():
    lay = wl.draw_layout(1)
    trees, ip, _ = trees_of(lay)
    t1 = wl.draw_tensors(lay, int(ip[-1]), dtype="bf16")
    t2 = wl.draw_tensors(lay, int(ip[-1]), dtype="bf16")
    for k in t1:
        assert torch.equal(t1[k], t2[k])
    assert t1["q"].dtype == torch.bfloat16 and t1["q"].shape == (ip[-1], 32, 128)
    assert t1["k_cache"].shape == (lay.num_pages, 8, 16, 128)


def test_poisoned_slack():
    lay = wl.custom_layout(4, [[1], [2, 3]], [20, 32], hq=2, hkv=1)
    ip = np.array([0, 7, 7 + 7], np.int32)
    t = wl.draw_tensors(lay, int(ip[-1]), dtype="f32", poison_slack=True)
    pg = lay.page_table[0, 1]
    assert (t["k_cache"][pg, :, 4:] == 1e4).all() and (t["k_cache"][pg, :, :4].abs() < 100).all()


def test_token_model_matches_closed_form():
    """Mean accepted length over many generated requests vs the exact expectation."""
    p = [5, 9, 12, 14]
    lay = wl.custom_layout(16, [p] * 4000, [0] * 4000, seed=3)
    trees, ip, parent = trees_of(lay)
    draft, argmax = wl.draw_tokens(lay, ip, parent, agree=0.7)
    L = [accept_by_alive(trees[b], draft[ip[b]:ip[b + 1]], argmax[ip[b]:ip[b + 1]]).L for b in range(lay.batch)]
    exact = expected_accept_len(16, p, 0.7)
    se = np.std(L) / np.sqrt(len(L))
    assert abs(np.mean(L) - exact) < 4 * se
    # mismatching drafts never equal the parent's prediction
    nonroot = parent >= 0
    base = np.repeat(ip[:-1], np.diff(ip))
    match = draft[nonroot] == argmax[(base + parent)[nonroot]]
    assert abs(match.mean() - 0.7) < 0.01
