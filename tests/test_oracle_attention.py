"""Pins of the attention oracle against a library routine and closed forms."""

import math

import numpy as np
import pytest
import torch

from oracle.attention import attend, batch_attention, gather_context, merge_states, request_attention
from oracle.tree import build_tree
from tests.golden_io import read_tree


def sdpa(q, k, v, mask=None, causal=False):
    """torch's scaled-dot-product attention in float64 on the CPU (library routine)."""
    q = torch.from_numpy(q)[None, None]
    k = torch.from_numpy(k)[None, None]
    v = torch.from_numpy(v)[None, None]
    m = None if mask is None else torch.from_numpy(mask)[None, None]
    return torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=m, is_causal=causal)[0, 0].numpy()


def rand_request(rng, B, p, C, hq=4, hkv=2, D=16):
    t = build_tree(B, p)
    q = rng.standard_normal((t.N, hq, D))
    kc = rng.standard_normal((C, hkv, D))
    vc = rng.standard_normal((C, hkv, D))
    kt = rng.standard_normal((t.N, hkv, D))
    vt = rng.standard_normal((t.N, hkv, D))
    return t, q, kc, vc, kt, vt


@pytest.mark.parametrize("name,C", [("tree_gamma4_p12.txt", 7), ("tree_gamma6_p245.txt", 33),
                                    ("tree_gamma6_p245.txt", 0)])
def test_matches_sdpa_with_hand_written_mask(name, C):
    g = read_tree(name)
    rng = np.random.default_rng(1)
    t, q, kc, vc, kt, vt = rand_request(rng, g["B"], g["p"], C)
    o, _ = request_attention(q, kc, vc, kt, vt, t)
    N = t.N
    mask = np.zeros((N, C + N), bool)
    mask[:, :C] = True
    for row in g["nodes"]:                     # mask from the fixture, not the oracle
        for m in row["anc"]:
            mask[row["node"], C + m] = True
    G = q.shape[1] // kc.shape[1]
    for hq in range(q.shape[1]):
        h = hq // G                            # grouped-query mapping
        keys = np.concatenate([kc[:, h], kt[:, h]])
        vals = np.concatenate([vc[:, h], vt[:, h]])
        ref = sdpa(q[:, hq], keys, vals, mask)
        np.testing.assert_allclose(o[:, hq], ref, atol=1e-12, rtol=0)


def test_chain_without_context_is_causal_attention():
    rng = np.random.default_rng(2)
    t, q, kc, vc, kt, vt = rand_request(rng, 16, [], 0, hq=2, hkv=2)
    o, _ = request_attention(q, kc, vc, kt, vt, t)
    for h in range(2):
        ref = sdpa(q[:, h], kt[:, h], vt[:, h], causal=True)
        np.testing.assert_allclose(o[:, h], ref, atol=1e-12, rtol=0)


def test_root_is_plain_decode_attention():
    # the anchor sees the context and itself only
    rng = np.random.default_rng(3)
    t, q, kc, vc, kt, vt = rand_request(rng, 16, [3, 7], 50, hq=2, hkv=1)
    o, _ = request_attention(q, kc, vc, kt, vt, t, nodes=[0])
    for hq in range(2):
        keys = np.concatenate([kc[:, 0], kt[:1, 0]])
        vals = np.concatenate([vc[:, 0], vt[:1, 0]])
        ref = sdpa(q[:1, hq], keys, vals)
        np.testing.assert_allclose(o[0, hq], ref[0], atol=1e-12, rtol=0)


def test_zero_query_gives_mean_of_visible_values():
    rng = np.random.default_rng(4)
    t, q, kc, vc, kt, vt = rand_request(rng, 6, [2, 4, 5], 9, hq=2, hkv=1)
    q[:] = 0.0
    o, lse = request_attention(q, kc, vc, kt, vt, t)
    for n in range(t.N):
        rows = [vc[c, 0] for c in range(9)] + [vt[m, 0] for m in sorted(t.ancestors[n])]
        np.testing.assert_allclose(o[n, 0], np.mean(rows, axis=0), atol=1e-13)
        assert lse[n, 0] == pytest.approx(math.log(len(rows)), abs=1e-13)


def test_saturated_softmax_picks_best_key():
    rng = np.random.default_rng(5)
    t, q, kc, vc, kt, vt = rand_request(rng, 4, [1, 2], 5, hq=1, hkv=1)
    q *= 1000.0
    o, lse = request_attention(q, kc, vc, kt, vt, t)
    assert np.isfinite(o).all() and np.isfinite(lse).all()
    for n in range(t.N):
        keys = list(kc[:, 0]) + [kt[m, 0] for m in sorted(t.ancestors[n])]
        vals = list(vc[:, 0]) + [vt[m, 0] for m in sorted(t.ancestors[n])]
        best = int(np.argmax([q[n, 0] @ k for k in keys]))
        np.testing.assert_allclose(o[n, 0], vals[best], atol=1e-9)


def test_probabilities_sum_to_one():
    rng = np.random.default_rng(6)
    q = rng.standard_normal((7, 8))
    k = rng.standard_normal((20, 8))
    vis = rng.random((7, 20)) < 0.5
    vis[:, 0] = True
    _, _, probs = attend(q, k, k, vis, 0.3, return_probs=True)
    np.testing.assert_allclose(probs.sum(1), 1.0, atol=1e-12)
    assert (probs[~vis] == 0).all()


def test_cascade_form_equals_single_pass():
    rng = np.random.default_rng(7)
    for C in (0, 1, 17, 64):
        t, q, kc, vc, kt, vt = rand_request(rng, 16, [2, 5, 11], C)
        o, lse = request_attention(q, kc, vc, kt, vt, t, "cascade")
        op, lp = request_attention(q, kc, vc, kt, vt, t, "prefix")
        ot, lt = request_attention(q, kc, vc, kt, vt, t, "tree")
        om, lm = merge_states(op, lp, ot, lt)
        np.testing.assert_allclose(om, o, atol=1e-12, rtol=0)
        np.testing.assert_allclose(lm, lse, atol=1e-12, rtol=0)
        if C == 0:
            assert (lp == -np.inf).all() and (op == 0).all()


def test_merge_state_special_cases():
    o_a = np.array([[1.0, 2.0]]); o_b = np.array([[3.0, 5.0]])
    o, l = merge_states(o_a, np.array([-np.inf]), o_b, np.array([0.25]))
    np.testing.assert_array_equal(o, o_b); assert l[0] == 0.25
    o, l = merge_states(o_a, np.array([-np.inf]), o_b, np.array([-np.inf]))
    assert (o == 0).all() and l[0] == -np.inf
    o, l = merge_states(o_a, np.array([math.log(3.0)]), o_b, np.array([0.0]))  # weights 3:1
    np.testing.assert_allclose(o, (3 * o_a + o_b) / 4, atol=1e-15)
    assert l[0] == pytest.approx(math.log(4.0), abs=1e-15)


def test_page_permutation_invariance_and_gather():
    rng = np.random.default_rng(8)
    P, Hkv, D, C = 16, 2, 8, 45
    logical_k = rng.standard_normal((3, Hkv, P, D))          # 3 logical pages
    logical_v = rng.standard_normal((3, Hkv, P, D))
    outs = []
    for perm in ([0, 1, 2, 3, 4], [4, 2, 0, 1, 3]):
        kc = np.full((5, Hkv, P, D), 99.0); vc = np.full((5, Hkv, P, D), 99.0)
        table = np.array(perm[:3])
        kc[table] = logical_k; vc[table] = logical_v
        k, v = gather_context(kc, vc, table, C, P)
        assert k.shape == (C, Hkv, D)
        np.testing.assert_array_equal(k[:, 1], logical_k[:, 1].reshape(-1, D)[:C])
        outs.append((k, v))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])


def test_batch_wrapper_matches_per_request():
    rng = np.random.default_rng(9)
    trees = [build_tree(4, [1, 2]), build_tree(4, [])]
    N = [t.N for t in trees]
    ip = np.array([0, N[0], N[0] + N[1]])
    P, Hkv, D, hq = 16, 1, 8, 2
    ctx = np.array([20, 3])
    table = np.array([[2, 0], [1, 0]])
    inputs = dict(q=rng.standard_normal((ip[-1], hq, D)), k_cache=rng.standard_normal((3, Hkv, P, D)),
                  v_cache=rng.standard_normal((3, Hkv, P, D)), k_tree=rng.standard_normal((ip[-1], Hkv, D)),
                  v_tree=rng.standard_normal((ip[-1], Hkv, D)), page_table=table, ctx_len=ctx, node_indptr=ip)
    o, lse = batch_attention(inputs, trees)
    for b in range(2):
        kc, vc = gather_context(inputs["k_cache"], inputs["v_cache"], table[b], ctx[b], P)
        s, e = ip[b], ip[b + 1]
        ob, lb = request_attention(inputs["q"][s:e], kc, vc, inputs["k_tree"][s:e], inputs["v_tree"][s:e], trees[b])
        np.testing.assert_array_equal(o[s:e], ob)
