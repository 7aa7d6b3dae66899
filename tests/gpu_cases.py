"""Shared set-up of GPU parity cases: seeded inputs -> HIP path and oracle."""

from __future__ import annotations

import numpy as np
import torch

from oracle.accept import accept_by_alive, accept_by_paths
from oracle.attention import gather_context, request_attention
from oracle.tree import build_tree
from paper_2606_04446_amd import workload as wl

TOL = {"f32": 1e-4, "bf16": 2e-2}   # max abs error vs float64, fp32 accumulation


def d2sd():
    from paper_2606_04446_amd import d2sd as m
    return m


class Case:
    """One batch: layout, oracle trees, device inputs and the library's outputs."""

    def __init__(self, layout: wl.Layout, device="cuda", poison_slack=False, dtype=None, tensors=True):
        m = d2sd()
        self.layout = layout
        self.spec = layout.spec
        self.dtype = dtype or self.spec.dtype
        self.B = self.spec.B
        self.trees = [build_tree(self.B, layout.p[b, :layout.K[b]]) for b in range(layout.batch)]
        ip_oracle = np.concatenate([[0], np.cumsum([t.N for t in self.trees])]).astype(np.int32)
        self.node_indptr, self.W = m.tree_plan(self.B, layout.K, layout.p)
        assert np.array_equal(self.node_indptr, ip_oracle)
        self.total = int(self.node_indptr[-1])
        self.max_nodes = int(np.diff(self.node_indptr).max())
        self.dev = device
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.d_K = t(layout.K.astype(np.int32))
        self.d_p = t(layout.p.astype(np.int32))
        self.d_ip = t(self.node_indptr)
        self.d_ctx = t(layout.ctx_len.astype(np.int32))
        self.d_pt = t(layout.page_table.astype(np.int32))
        self.tree = m.tree_build(self.B, self.d_K, self.d_p, self.d_ip, self.total, self.W)
        self.parent_oracle = np.concatenate([t.parent for t in self.trees]).astype(np.int32)
        self.draft, self.argmax = wl.draw_tokens(layout, self.node_indptr, self.parent_oracle)
        self.x = wl.draw_tensors(layout, self.total, device=device, dtype=self.dtype,
                                 poison_slack=poison_slack) if tensors else None

    # ---- HIP path ----
    def attention(self, stage=0, kv_split=0, out=None, lse=None, host_offsets=False, row_group=0, packed=0):
        """host_offsets: hand the host copy of the node offsets to the planner,
        as the benchmark does (the automatic split then counts work items exactly)."""
        m = d2sd()
        x = self.x
        return m.cascade_verify_attention(
            x["q"], x["k_cache"], x["v_cache"], self.d_pt, self.d_ctx, x["k_tree"], x["v_tree"], self.d_ip,
            self.tree["anc_mask"], total_nodes=self.total, max_nodes=self.max_nodes,
            max_ctx_len=int(self.layout.ctx_len.max(initial=0)), stage=stage, kv_split=kv_split, out=out,
            lse=lse, node_indptr_host=self.node_indptr if host_offsets else None, row_group=row_group,
            packed=packed)

    def _args(self, kv_split=0, host_offsets=False, row_group=0, packed=0, stage=0):
        m = d2sd()
        x = self.x
        return m.attn_args(x["q"], x["k_cache"], x["v_cache"], self.d_pt, self.d_ctx, x["k_tree"], x["v_tree"],
                           self.d_ip, self.tree["anc_mask"], x["q"], None, total_nodes=self.total,
                           max_nodes=self.max_nodes, max_ctx_len=int(self.layout.ctx_len.max(initial=0)),
                           kv_split=kv_split, node_indptr_host=self.node_indptr if host_offsets else None,
                           row_group=row_group, packed=packed, stage=stage)

    def resolved_split(self, kv_split=0, host_offsets=False, **kw):
        """The split length the library takes for this batch."""
        return d2sd().cascade_kv_split(self._args(kv_split, host_offsets, **kw))

    def shape(self, kv_split=0, host_offsets=False, **kw):
        """(rows per workgroup, packed) the library takes for this batch."""
        return d2sd().cascade_shape(self._args(kv_split, host_offsets, **kw))

    def noncascade(self):
        m = d2sd()
        x = self.x
        return m.noncascade_verify_attention(
            x["q"], x["k_cache"], x["v_cache"], self.d_pt, self.d_ctx, x["k_tree"], x["v_tree"], self.d_ip,
            self.tree["anc_mask"], total_nodes=self.total, max_nodes=self.max_nodes,
            max_ctx_len=int(self.layout.ctx_len.max(initial=0)))

    def accept(self):
        m = d2sd()
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)
        return m.accept_path(self.B, self.d_ip, self.total, self.tree["parent"], self.tree["depth"],
                             self.tree["path_id"], t(self.draft), t(self.argmax))

    # ---- oracle ----
    def request_inputs(self, b):
        """float64 host copies of request b's inputs (exact stored values)."""
        s, e = int(self.node_indptr[b]), int(self.node_indptr[b + 1])
        C = int(self.layout.ctx_len[b])
        npg = (C + 15) // 16
        pages = torch.from_numpy(self.layout.page_table[b, :npg].astype(np.int64)).to(self.dev)
        kc = self.x["k_cache"].index_select(0, pages).double().cpu().numpy()
        vc = self.x["v_cache"].index_select(0, pages).double().cpu().numpy()
        table = np.arange(npg)
        kc, vc = gather_context(kc, vc, table, C, 16)
        q = self.x["q"][s:e].double().cpu().numpy()
        kt = self.x["k_tree"][s:e].double().cpu().numpy()
        vt = self.x["v_tree"][s:e].double().cpu().numpy()
        return q, kc, vc, kt, vt

    def oracle_attention(self, b, stage="cascade", nodes=None, heads=None):
        q, kc, vc, kt, vt = self.request_inputs(b)
        return request_attention(q, kc, vc, kt, vt, self.trees[b], stage, nodes=nodes, heads=heads)

    def oracle_accept(self, b):
        s, e = int(self.node_indptr[b]), int(self.node_indptr[b + 1])
        a = accept_by_paths(self.trees[b], self.draft[s:e], self.argmax[s:e])
        c = accept_by_alive(self.trees[b], self.draft[s:e], self.argmax[s:e])
        assert (a.L, a.best_path, a.node, a.path_nodes, a.tokens) == (c.L, c.best_path, c.node, c.path_nodes, c.tokens)
        return a


def oracle_tree_arrays(trees, W, kmax=None):
    parent = np.concatenate([t.parent for t in trees]).astype(np.int32)
    depth = np.concatenate([t.position for t in trees]).astype(np.int32)
    path = np.concatenate([t.path for t in trees]).astype(np.int32)
    mask = np.concatenate([t.packed_mask(W) for t in trees]).view(np.int32)
    kmax = max([t.K for t in trees] + [0]) if kmax is None else kmax
    leaf = np.full((len(trees), kmax + 1), -1, np.int32)
    for b, t in enumerate(trees):
        leaf[b, :t.K + 1] = t.path_leaf()
    return parent, depth, path, mask, leaf


def max_abs(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    both_inf = np.isneginf(a) & np.isneginf(b)       # equal -inf (an empty side) counts as exact
    with np.errstate(invalid="ignore"):
        d = np.abs(np.where(both_inf, 0.0, a - b))
    return float(np.nan_to_num(d, nan=np.inf).max(initial=0.0))
