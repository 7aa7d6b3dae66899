"""GPU parity of the integer steps: tree build and accept path, bit-exact."""

import itertools

import numpy as np
import pytest
import torch

from oracle.accept import accept_by_alive, accept_by_paths
from oracle.tree import build_tree
from paper_2606_04446_amd import workload as wl
from tests.gpu_cases import Case, d2sd, oracle_tree_arrays

pytestmark = pytest.mark.gpu


def run_tree(B, p_rows):
    m = d2sd()
    K = np.array([len(r) for r in p_rows], np.int32)
    kmax = max(1, int(K.max(initial=0)))
    p = np.zeros((len(p_rows), kmax), np.int32)
    for b, r in enumerate(p_rows):
        p[b, :len(r)] = r
    ip, W = m.tree_plan(B, K, p)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    got = m.tree_build(B, dev(K), dev(p), dev(ip), int(ip[-1]), W)
    trees = [build_tree(B, r) for r in p_rows]
    want = oracle_tree_arrays(trees, W, kmax)
    names = ["parent", "depth", "path_id", "anc_mask", "path_leaf"]
    for name, w in zip(names, want):
        g = got[name].cpu().numpy()
        assert np.array_equal(g, w), (name, B)
    return ip, got, trees


@pytest.mark.parametrize("B", [2, 3, 5, 8])
def test_tree_every_branch_set(B):
    rows = [list(c) for K in range(B) for c in itertools.combinations(range(1, B), K)]
    run_tree(B, rows)


@pytest.mark.parametrize("B", [16, 33, 64])
def test_tree_random_and_extremes(B):
    rng = np.random.default_rng(B)
    rows = [[], list(range(1, B)), [1], [B - 1], list(range(B - 1, 0, -1))]
    for _ in range(60):
        K = int(rng.integers(0, B))
        rows.append(rng.permutation(np.arange(1, B))[:K].tolist())   # unsorted
    run_tree(B, rows)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_tree_and_accept_workloads(cfg):
    case = Case(wl.draw_layout(cfg), tensors=False)
    want = oracle_tree_arrays(case.trees, case.W, case.layout.kmax)
    for name, w in zip(["parent", "depth", "path_id", "anc_mask", "path_leaf"], want):
        assert np.array_equal(case.tree[name].cpu().numpy(), w), name
    got = {k: v.cpu().numpy() for k, v in case.accept().items()}
    for b in range(case.layout.batch):
        a = case.oracle_accept(b)
        pn, tk = a.padded(case.B)
        assert (got["accept_len"][b], got["best_path"][b], got["accept_node"][b]) == (a.L, a.best_path, a.node), b
        assert got["path_nodes"][b].tolist() == pn and got["out_tokens"][b].tolist() == tk, b


def test_accept_every_match_pattern_tiny_trees():
    """All 37,866 (tree, match pattern) cases with B <= 5, one launch per B."""
    m = d2sd()
    total_cases = 0
    for B in range(2, 6):
        p_rows, pats = [], []
        for K in range(B):
            for p in itertools.combinations(range(1, B), K):
                N = B + sum(B - x for x in p)
                for bits in itertools.product((0, 1), repeat=N - 1):
                    p_rows.append(list(p))
                    pats.append(bits)
        ip, tree, trees = run_tree(B, p_rows)
        draft = np.zeros(int(ip[-1]), np.int32)
        argmax = np.zeros(int(ip[-1]), np.int32)
        for b, (t, bits) in enumerate(zip(trees, pats)):
            s = int(ip[b])
            argmax[s:s + t.N] = 1000 + np.arange(t.N)
            for c in range(1, t.N):
                draft[s + c] = argmax[s + t.parent[c]] if bits[c - 1] else 7
        dev = lambda a: torch.from_numpy(a).cuda()
        got = m.accept_path(B, dev(ip), int(ip[-1]), tree["parent"], tree["depth"], tree["path_id"],
                            dev(draft), dev(argmax))
        got = {k: v.cpu().numpy() for k, v in got.items()}
        for b, t in enumerate(trees):
            s, e = int(ip[b]), int(ip[b + 1])
            a = accept_by_paths(t, draft[s:e], argmax[s:e])
            pn, tk = a.padded(B)
            assert (got["accept_len"][b], got["best_path"][b], got["accept_node"][b]) == (a.L, a.best_path, a.node)
            assert got["path_nodes"][b].tolist() == pn and got["out_tokens"][b].tolist() == tk
        total_cases += len(trees)
    assert total_cases == 37866


def test_accept_large_blocks_small_vocab():
    """B = 64 (up to 2080 nodes per request) with a 3-token vocabulary: long
    accepted runs, many ties."""
    m = d2sd()
    rng = np.random.default_rng(7)
    B = 64
    rows = [list(range(1, B)), [], [1, 2, 3], [63, 40, 5]]
    for _ in range(12):
        rows.append(rng.permutation(np.arange(1, B))[:int(rng.integers(0, B))].tolist())
    ip, tree, trees = run_tree(B, rows)
    draft = rng.integers(0, 2, size=int(ip[-1])).astype(np.int32)
    argmax = rng.integers(0, 2, size=int(ip[-1])).astype(np.int32)
    dev = lambda a: torch.from_numpy(a).cuda()
    got = m.accept_path(B, dev(ip), int(ip[-1]), tree["parent"], tree["depth"], tree["path_id"], dev(draft),
                        dev(argmax))
    got = {k: v.cpu().numpy() for k, v in got.items()}
    for b, t in enumerate(trees):
        s, e = int(ip[b]), int(ip[b + 1])
        a = accept_by_alive(t, draft[s:e], argmax[s:e])
        pn, tk = a.padded(B)
        assert (got["accept_len"][b], got["best_path"][b], got["accept_node"][b]) == (a.L, a.best_path, a.node), b
        assert got["path_nodes"][b].tolist() == pn and got["out_tokens"][b].tolist() == tk, b
