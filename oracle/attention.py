"""Verify attention over the candidate tree (oracle; test infrastructure).

Sec. 3.3 (iv): the target model verifies the K+1 candidates in one forward
pass with shared-prefix cascade attention; sec. 1 (contribution 2): the shared
context is reused instead of being replicated per candidate. Cascade attention
is an exact refactoring of ordinary softmax attention, so this oracle computes
the definition directly: every tree node's query attends to all context keys
and to the keys of its ancestors-or-self in the tree, in one softmax.

Readings (the paper states no layer shapes or attention details):
  * softmax scale 1/sqrt(head_dim) unless given; query head h uses KV head
    floor(h / G), G = query heads / KV heads (grouped-query attention);
  * a node sees the whole context (no window) and its ancestors including
    itself; the anchor (root) is a tree node, not context;
  * queries and keys arrive already position-encoded.

Everything is float64. A row with no visible key gets output 0 and
lse = -inf (only possible for the context-only state of an empty context).
"""

from __future__ import annotations

import math

import numpy as np


def gather_context(k_cache, v_cache, page_table_row, ctx_len: int, page_size: int):
    """Logical context K/V of one request, [C, Hkv, D] float64, through its page table.

    k_cache/v_cache are [num_pages, Hkv, page_size, D]."""
    C = int(ctx_len)
    Hkv, D = k_cache.shape[1], k_cache.shape[3]
    if C == 0:
        z = np.zeros((0, Hkv, D), np.float64)
        return z, z.copy()
    npg = (C + page_size - 1) // page_size
    ids = np.asarray(page_table_row[:npg], np.int64)
    k = np.asarray(k_cache[ids], np.float64).transpose(0, 2, 1, 3).reshape(npg * page_size, Hkv, D)
    v = np.asarray(v_cache[ids], np.float64).transpose(0, 2, 1, 3).reshape(npg * page_size, Hkv, D)
    return k[:C], v[:C]


def attend(q, keys, vals, visible, scale: float, return_probs: bool = False):
    """Softmax attention by definition.

    q [R, D], keys/vals [T, D], visible [R, T] bool. Returns o [R, D], lse [R]
    (natural log of the sum of exp(score) over visible keys) and optionally the
    probability matrix [R, T]."""
    q = np.asarray(q, np.float64)
    keys = np.asarray(keys, np.float64)
    vals = np.asarray(vals, np.float64)
    R, T = q.shape[0], keys.shape[0]
    s = (q @ keys.T) * scale if T else np.zeros((R, 0))
    s = np.where(visible, s, -np.inf)
    o = np.zeros((R, q.shape[1]))
    lse = np.full(R, -np.inf)
    probs = np.zeros((R, T))
    for r in range(R):
        if not visible[r].any():
            continue
        m = s[r].max()
        e = np.exp(s[r] - m)                   # exp(-inf) = 0 for hidden keys
        l = e.sum()
        probs[r] = e / l
        o[r] = probs[r] @ vals
        lse[r] = m + math.log(l)
    return (o, lse, probs) if return_probs else (o, lse)


def request_attention(q, kc, vc, kt, vt, tree, stage: str = "cascade", scale=None,
                      nodes=None, heads=None):
    """Verify attention of one request.

    q [N, Hq, D]; kc/vc [C, Hkv, D] (gathered context); kt/vt [N, Hkv, D] tree
    keys/values in canonical node order; tree from oracle.tree.build_tree.
    stage: "cascade" (context + ancestors), "prefix" (context only) or "tree"
    (ancestors only). nodes/heads restrict the rows computed (default all).
    Returns o [len(nodes), len(heads), D], lse [len(nodes), len(heads)]."""
    N, Hq, D = q.shape
    C, Hkv = kc.shape[0], kt.shape[1]
    G = Hq // Hkv
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    nodes = list(range(N)) if nodes is None else list(nodes)
    heads = list(range(Hq)) if heads is None else list(heads)
    vis_tree = tree.visible()[nodes]                       # [R, N]
    use_ctx = stage in ("cascade", "prefix")
    use_tree = stage in ("cascade", "tree")
    o = np.zeros((len(nodes), len(heads), D))
    lse = np.zeros((len(nodes), len(heads)))
    for j, hq in enumerate(heads):
        h = hq // G
        keys, vals, vis = [], [], []
        if use_ctx:
            keys.append(kc[:, h]); vals.append(vc[:, h])
            vis.append(np.ones((len(nodes), C), bool))
        if use_tree:
            keys.append(kt[:, h]); vals.append(vt[:, h])
            vis.append(vis_tree)
        K_ = np.concatenate(keys, 0) if keys else np.zeros((0, D))
        V_ = np.concatenate(vals, 0) if vals else np.zeros((0, D))
        M_ = np.concatenate(vis, 1) if vis else np.zeros((len(nodes), 0), bool)
        o[:, j], lse[:, j] = attend(q[nodes, hq], K_, V_, M_, scale)
    return o, lse


def merge_states(o_a, lse_a, o_b, lse_b):
    """Log-sum-exp merge of two attention states over disjoint key sets.

    With weights w_x = exp(lse_x - m), m = max(lse_a, lse_b), the merged output
    is the weight-averaged output and the merged lse is m + ln(w_a + w_b); a
    state with lse = -inf carries no weight."""
    o_a, o_b = np.asarray(o_a, np.float64), np.asarray(o_b, np.float64)
    lse_a, lse_b = np.asarray(lse_a, np.float64), np.asarray(lse_b, np.float64)
    o = np.zeros(np.broadcast_shapes(o_a.shape, o_b.shape))
    lse = np.full(np.broadcast_shapes(lse_a.shape, lse_b.shape), -np.inf)
    for idx in np.ndindex(lse.shape):
        a, b = lse_a[idx], lse_b[idx]
        if a == -np.inf and b == -np.inf:
            continue
        m = max(a, b)
        wa, wb = math.exp(a - m), math.exp(b - m)
        o[idx] = (wa * o_a[idx] + wb * o_b[idx]) / (wa + wb)
        lse[idx] = m + math.log(wa + wb)
    return o, lse


def batch_attention(inputs: dict, trees, stage: str = "cascade", scale=None):
    """Verify attention of a whole batch (requests one at a time).

    inputs: float64-convertible arrays q [ΣN, Hq, D], k_cache, v_cache
    [pages, Hkv, P, D], k_tree, v_tree [ΣN, Hkv, D], and integer arrays
    page_table [batch, max_pages], ctx_len [batch], node_indptr [batch+1].
    Returns o [ΣN, Hq, D], lse [ΣN, Hq]."""
    q = inputs["q"]
    P = inputs["k_cache"].shape[2]
    ip = inputs["node_indptr"]
    o = np.zeros(q.shape)
    lse = np.zeros(q.shape[:2])
    for b, tree in enumerate(trees):
        s, e = int(ip[b]), int(ip[b + 1])
        kc, vc = gather_context(inputs["k_cache"], inputs["v_cache"], inputs["page_table"][b],
                                int(inputs["ctx_len"][b]), P)
        o[s:e], lse[s:e] = request_attention(np.asarray(q[s:e], np.float64), kc, vc,
                                             np.asarray(inputs["k_tree"][s:e], np.float64),
                                             np.asarray(inputs["v_tree"][s:e], np.float64),
                                             tree, stage, scale)
    return o, lse
