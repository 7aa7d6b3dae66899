"""Pins of the accepted-path commit (sec. 3.3): checked through the context
read (page-table gather), which is written independently of the commit."""

import numpy as np

from oracle.accept import accept_by_alive
from oracle.attention import gather_context
from oracle.commit import commit_accepted
from oracle.tree import build_tree


def make_case(rng, batch=3, B=8, hkv=2, D=8, P=4):
    trees = [build_tree(B, sorted(rng.choice(np.arange(1, B), size=2, replace=False))) for _ in range(batch)]
    ip = np.concatenate([[0], np.cumsum([t.N for t in trees])]).astype(np.int64)
    ctx = np.array([0, 15, 33][:batch])            # empty, ends one short of a page, mid-page
    max_pages = (ctx.max() + B + P - 1) // P + 1
    num_pages = batch * max_pages + 3
    table = rng.permutation(num_pages)[:batch * max_pages].reshape(batch, max_pages)
    kc = rng.standard_normal((num_pages, hkv, P, D))
    vc = rng.standard_normal((num_pages, hkv, P, D))
    kt = rng.standard_normal((ip[-1], hkv, D))
    vt = rng.standard_normal((ip[-1], hkv, D))
    return trees, ip, ctx, table, kc, vc, kt, vt


def test_committed_context_is_old_context_plus_accepted_path():
    rng = np.random.default_rng(5)
    P = 4
    trees, ip, ctx, table, kc, vc, kt, vt = make_case(rng, P=P)
    B = trees[0].B
    accs = []
    for b, t in enumerate(trees):
        # a draft/argmax pattern accepting a random prefix of a random path
        draft = rng.integers(0, 5, t.N)
        argmax = rng.integers(0, 5, t.N)
        accs.append(accept_by_alive(t, draft, argmax))
    path_nodes = np.array([a.padded(B)[0] for a in accs])
    L = np.array([a.L for a in accs])
    kc2, vc2, ctx2 = commit_accepted(kc, vc, table, ctx, ip, path_nodes, L, kt, vt, P)
    assert np.array_equal(ctx2, ctx + L + 1)
    for b in range(len(trees)):
        k_old, v_old = gather_context(kc, vc, table[b], ctx[b], P)
        k_new, v_new = gather_context(kc2, vc2, table[b], ctx2[b], P)
        nodes = ip[b] + np.asarray(accs[b].path_nodes)
        np.testing.assert_array_equal(k_new, np.concatenate([k_old, kt[nodes]]))
        np.testing.assert_array_equal(v_new, np.concatenate([v_old, vt[nodes]]))
        # the path starts at the root (the anchor) and descends one depth per token
        assert accs[b].path_nodes[0] == 0
        assert [trees[b].position[n] for n in accs[b].path_nodes] == list(range(L[b] + 1))


def test_commit_touches_only_the_new_positions():
    rng = np.random.default_rng(6)
    P = 4
    trees, ip, ctx, table, kc, vc, kt, vt = make_case(rng, P=P)
    B = trees[0].B
    L = np.array([0, B - 1, 3])
    path_nodes = np.full((3, B), -1)
    for b in range(3):
        path_nodes[b, :L[b] + 1] = np.arange(L[b] + 1)      # main chain
    kc2, vc2, _ = commit_accepted(kc, vc, table, ctx, ip, path_nodes, L, kt, vt, P)
    touched = np.zeros(kc.shape[:3], bool)
    for b in range(3):
        for d in range(L[b] + 1):
            pos = ctx[b] + d
            touched[table[b, pos // P], :, pos % P] = True
    np.testing.assert_array_equal(kc2[~touched], kc[~touched])
    np.testing.assert_array_equal(vc2[~touched], vc[~touched])
    assert touched.sum() == (L + 1).sum() * kc.shape[1]
