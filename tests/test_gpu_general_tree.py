"""GPU parity on trees given as parent arrays (third-level cascade, sec. 4.3;
independent resampling): the builder bit for bit, then cascade attention and
the accept path over such trees against the oracle."""

import numpy as np
import pytest
import torch

from oracle.accept import accept_by_alive
from oracle.attention import gather_context, request_attention
from oracle.tree import build_tree, resample_parents, third_level_parents, tree_from_parents
from paper_2606_04446_amd import workload as wl
from tests.gpu_cases import TOL, max_abs

pytestmark = pytest.mark.gpu


def d2sd():
    from paper_2606_04446_amd import d2sd as m
    return m


def build_on_device(trees, W=None):
    m = d2sd()
    dev = torch.device("cuda")
    ip = np.concatenate([[0], np.cumsum([t.N for t in trees])]).astype(np.int32)
    parent = np.concatenate([t.parent for t in trees]).astype(np.int32)
    max_nodes = max(t.N for t in trees)
    W = W or (max_nodes + 31) // 32
    out = m.tree_from_parents(torch.from_numpy(ip).to(dev), int(ip[-1]), max_nodes,
                              torch.from_numpy(parent).to(dev), W)
    torch.cuda.synchronize()
    return ip, parent, W, {k: v.cpu().numpy() for k, v in out.items()}


def check_builder(trees, W=None):
    ip, parent, W, got = build_on_device(trees, W)
    assert np.array_equal(got["depth"], np.concatenate([t.position for t in trees]))
    assert np.array_equal(got["path_id"], np.concatenate([t.path for t in trees]))
    assert np.array_equal(got["anc_mask"], np.concatenate([t.packed_mask(W) for t in trees]).view(np.int32))


def random_trees(rng, count, max_n, max_depth=None):
    out = []
    for _ in range(count):
        N = int(rng.integers(1, max_n + 1))
        parent = [-1]
        depth = [0]
        for n in range(1, N):
            while True:
                q = int(rng.integers(max(0, n - 40), n))
                if max_depth is None or depth[q] + 1 <= max_depth:
                    break
            parent.append(q)
            depth.append(depth[q] + 1)
        out.append(tree_from_parents(parent))
    return out


def test_builder_random_trees():
    rng = np.random.default_rng(21)
    check_builder(random_trees(rng, 40, 300))
    check_builder(random_trees(rng, 8, 2080))                 # largest node count, 65 mask words


def test_builder_third_level_and_resample_shapes():
    rng = np.random.default_rng(22)
    trees = []
    for _ in range(24):
        B = int(rng.integers(3, 33))
        K = int(rng.integers(1, min(B - 2, 8) + 1))
        p = sorted(rng.choice(np.arange(1, B - 1), size=K, replace=False).tolist())
        q = [int(rng.integers(pk + 1, B)) for pk in p]
        trees.append(tree_from_parents(third_level_parents(B, p, q), B))
        trees.append(tree_from_parents(resample_parents(B, int(rng.integers(1, 6))), B))
    check_builder(trees)


def test_builder_matches_canonical_builder():
    m = d2sd()
    rng = np.random.default_rng(23)
    B, Kmax = 16, 8
    ps = [sorted(rng.choice(np.arange(1, B), size=int(rng.integers(0, Kmax + 1)), replace=False).tolist())
          for _ in range(30)]
    trees = [build_tree(B, p) for p in ps]
    W = m.mask_words(B)
    check_builder(trees, W)
    ip, parent, _, got = build_on_device(trees, W)
    K = np.array([len(p) for p in ps], np.int32)
    P = np.zeros((len(ps), Kmax), np.int32)
    for b, p in enumerate(ps):
        P[b, :len(p)] = p
    dev = torch.device("cuda")
    t = lambda a: torch.from_numpy(a).to(dev)
    canon = m.tree_build(B, t(K), t(P), t(ip), int(ip[-1]), W)
    torch.cuda.synchronize()
    for k in ("depth", "path_id", "anc_mask"):
        assert np.array_equal(canon[k].cpu().numpy(), got[k]), k


@pytest.mark.parametrize("shape", ["third_level", "resample"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attention_and_accept_on_general_trees(shape, dtype):
    m = d2sd()
    B = 16
    rng = np.random.default_rng(24)
    ctx = [0, 77, 300, 1000]
    if shape == "third_level":
        parents = [third_level_parents(B, [2, 6, 11], [5, 9, 14]), third_level_parents(B, [1], [2]),
                   third_level_parents(B, [3, 4], [15, 15]), third_level_parents(B, [7], [8])]
    else:
        parents = [resample_parents(B, c) for c in (1, 2, 3, 5)]
    trees = [tree_from_parents(pa, B) for pa in parents]
    lay = wl.custom_layout(B, [[] for _ in ctx], ctx, hq=8, hkv=2, dtype=dtype, seed=5)
    dev = torch.device("cuda")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    ip, parent, W, built = build_on_device(trees)
    total, max_nodes = int(ip[-1]), max(tr.N for tr in trees)
    x = wl.draw_tensors(lay, total, device=dev, dtype=dtype)
    out, lse = m.cascade_verify_attention(x["q"], x["k_cache"], x["v_cache"], t(lay.page_table), t(lay.ctx_len),
                                          x["k_tree"], x["v_tree"], t(ip), t(built["anc_mask"]),
                                          total_nodes=total, max_nodes=max_nodes, max_ctx_len=max(ctx))
    draft, argmax = wl.draw_tokens(lay, ip, parent)
    acc = m.accept_path(B, t(ip), total, t(parent), t(built["depth"]), t(built["path_id"]), t(draft), t(argmax))
    torch.cuda.synchronize()
    for b, tr in enumerate(trees):
        s, e = int(ip[b]), int(ip[b + 1])
        kc, vc = gather_context(x["k_cache"].double().cpu().numpy(), x["v_cache"].double().cpu().numpy(),
                                lay.page_table[b], ctx[b], 16)
        ow, lw = request_attention(x["q"][s:e].double().cpu().numpy(), kc, vc,
                                   x["k_tree"][s:e].double().cpu().numpy(), x["v_tree"][s:e].double().cpu().numpy(), tr)
        err = max(max_abs(out[s:e].double().cpu().numpy(), ow), max_abs(lse[s:e].cpu().numpy(), lw))
        assert err <= TOL[dtype], (shape, b, err)
        a = accept_by_alive(tr, draft[s:e], argmax[s:e])
        assert int(acc["accept_len"][b]) == a.L and int(acc["accept_node"][b]) == a.node
        assert int(acc["best_path"][b]) == a.best_path
        pn, tk = a.padded(B)
        assert acc["path_nodes"][b].cpu().tolist() == pn and acc["out_tokens"][b].cpu().tolist() == tk
