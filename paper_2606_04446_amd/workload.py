"""Seeded synthetic inputs for one verify step (one attention layer).

This module only draws random inputs; it contains no step of the verify
computation and builds no tree. Tree sizes (``node_indptr``) and tree
topology (``parent``) are passed in by the caller, who gets them from the
library's host planner and tree builder or from the oracle.

Five workloads stand in for the paper's end-to-end runs (which use eight public
benchmarks with trained drafters, not available here): they take the paper's
default verify shape (block length 16, K branches around the default K = 4,
sec. 4.1) and a Qwen3-8B-class GQA head shape (32 query / 8 KV heads, head
dim 128). Draw order within a seed, fixed so that a seed names one workload:

  numpy stream 0: context lengths -> branch re-anchor positions -> page
                  permutation
  numpy stream 1: target argmax tokens -> agreement flags -> replacement tokens
  numpy stream 2: first-drafter confidences (device re-anchor selection input)
  numpy stream 3: sub-branch positions (third-level tree shape)
  numpy stream 4: uniforms of the sampling draws
  torch generator (seed): Q -> K cache -> V cache -> K tree -> V tree
  torch generator (seed + 2^32): target logits
"""

from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import numpy as np

VOCAB = 32000
PAGE = 16
HEAD_DIM = 128


@dataclasses.dataclass(frozen=True)
class Spec:
    """One synthetic verify workload."""

    name: str
    dtype: str                 # "f32" or "bf16"
    batch: int
    ctx: tuple                 # (lo, hi) inclusive; lo == hi for a fixed length
    hq: int
    hkv: int
    B: int = 16
    K: int = 4
    p_rule: str = "beta_lowest"  # "uniform" | "beta_lowest"
    permute_pages: bool = True
    agree: float = 0.7
    head_dim: int = HEAD_DIM
    page_size: int = PAGE


# The five workloads. p_rule "uniform": K distinct positions uniform in
# [1, B-1]. p_rule "beta_lowest": per-position confidence c_j ~ Beta(5, 2),
# j = 1..B-1, and the K positions with the lowest confidence (ties to the
# smaller j) become the re-anchor positions.
WORKLOADS = {
    1: Spec("ctx512-b1-fp32", "f32", 1, (512, 512), 32, 8, K=2, p_rule="uniform",
            permute_pages=False),
    2: Spec("ctx4096-b1-bf16", "bf16", 1, (4096, 4096), 32, 8, K=4),
    3: Spec("ctx1k-8k-b8-bf16", "bf16", 8, (1024, 8192), 32, 8, K=4),
    4: Spec("ctx16k-b32-bf16", "bf16", 32, (16384, 16384), 32, 8, K=8),
    5: Spec("ctx32k-b64-hq64-bf16", "bf16", 64, (32768, 32768), 64, 8, K=8),
}


@dataclasses.dataclass
class Layout:
    """Host-side description of one batch: branch sets, context and pages."""

    spec: Spec
    seed: int
    K: np.ndarray            # [batch] int32 branch counts
    p: np.ndarray            # [batch, Kmax] int32 re-anchor positions (row b: K[b] used)
    ctx_len: np.ndarray      # [batch] int32
    page_table: np.ndarray   # [batch, max_pages] int32
    num_pages: int

    @property
    def batch(self) -> int:
        return int(self.K.shape[0])

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def kmax(self) -> int:
        return int(self.p.shape[1])


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def draw_positions(rng: np.random.Generator, B: int, K: int, rule: str) -> np.ndarray:
    """K distinct re-anchor positions in [1, B-1] by the workload's rule."""
    if K == 0:
        return np.zeros(0, np.int32)
    if rule == "uniform":
        return np.sort(rng.choice(np.arange(1, B), size=K, replace=False)).astype(np.int32)
    if rule == "beta_lowest":
        conf = rng.beta(5.0, 2.0, size=B - 1)            # positions 1..B-1
        order = np.argsort(conf, kind="stable")[:K]      # lowest first, ties -> smaller j
        return np.sort(order + 1).astype(np.int32)
    raise ValueError(f"unknown p_rule {rule!r}")


def pages_for(ctx_len: Sequence[int], page_size: int, permute: bool,
              rng: Optional[np.random.Generator]) -> tuple[np.ndarray, int]:
    """Page table over a pool of sum(ceil(C_b/page)) pages; request b's logical
    pages take consecutive slots of a random permutation of the pool (or the
    identity). Unused table entries are 0 (a valid page that is never read)."""
    n = [(int(c) + page_size - 1) // page_size for c in ctx_len]
    total = int(sum(n))
    perm = rng.permutation(total) if (permute and total > 0) else np.arange(total)
    max_pages = max(1, max(n) if n else 1)
    table = np.zeros((len(n), max_pages), np.int32)
    off = 0
    for b, nb in enumerate(n):
        table[b, :nb] = perm[off:off + nb]
        off += nb
    return table, max(total, 1)


def draw_layout(cfg, seed: Optional[int] = None) -> Layout:
    """Layout of a numbered workload (seed defaults to the workload number) or of a Spec."""
    if isinstance(cfg, int):
        spec = WORKLOADS[cfg]
        seed = cfg if seed is None else seed
    else:
        spec = cfg
        seed = 0 if seed is None else seed
    rng = _rng(seed, 0)
    lo, hi = spec.ctx
    ctx = rng.integers(lo, hi + 1, size=spec.batch).astype(np.int32) if lo != hi \
        else np.full(spec.batch, lo, np.int32)
    p = np.zeros((spec.batch, max(spec.K, 1)), np.int32)
    for b in range(spec.batch):
        p[b, :spec.K] = draw_positions(rng, spec.B, spec.K, spec.p_rule)
    K = np.full(spec.batch, spec.K, np.int32)
    table, npages = pages_for(ctx, spec.page_size, spec.permute_pages, rng)
    return Layout(spec, seed, K, p, ctx, table, npages)


def custom_layout(B: int, p_rows: Sequence[Sequence[int]], ctx_len: Sequence[int], hq: int = 32,
                  hkv: int = 8, dtype: str = "bf16", seed: int = 0,
                  permute_pages: bool = True) -> Layout:
    """Layout with explicit branch sets and context lengths (edge-case tests)."""
    batch = len(p_rows)
    kmax = max([len(r) for r in p_rows] + [1])
    p = np.zeros((batch, kmax), np.int32)
    K = np.zeros(batch, np.int32)
    for b, r in enumerate(p_rows):
        K[b] = len(r)
        p[b, :len(r)] = r
    ctx = np.asarray(ctx_len, np.int32)
    spec = Spec("custom", dtype, batch, (int(ctx.min(initial=0)), int(ctx.max(initial=0))), hq, hkv,
                B=B, K=int(K.max(initial=0)), p_rule="explicit", permute_pages=permute_pages)
    table, npages = pages_for(ctx, PAGE, permute_pages, _rng(seed, 0))
    return Layout(spec, seed, K, p, ctx, table, npages)


def draw_confidences(layout: "Layout") -> np.ndarray:
    """First-drafter confidences c_1..c_{B-1} per request, Beta(5, 2), float32
    [batch, B-1] (numpy stream 2 of the layout seed); input of the device
    re-anchor selection."""
    spec = layout.spec
    rng = _rng(layout.seed, 2)
    return rng.beta(5.0, 2.0, size=(layout.batch, spec.B - 1)).astype(np.float32)


def draw_sub_branch_positions(layout: "Layout") -> np.ndarray:
    """Re-anchor position q_k of the sub-branch inside branch k's tail for the
    third-level tree shape: uniform in (p_k, B-1], or 0 (no sub-branch) when
    p_k = B-1. int32 [batch, Kmax] (numpy stream 3 of the layout seed)."""
    B = layout.spec.B
    rng = _rng(layout.seed, 3)
    q = np.zeros_like(layout.p)
    for b in range(layout.batch):
        for k in range(int(layout.K[b])):
            pk = int(layout.p[b, k])
            q[b, k] = int(rng.integers(pk + 1, B)) if pk < B - 1 else 0
    return q


def draw_tokens(layout: Layout, node_indptr: np.ndarray, parent: np.ndarray,
                agree: Optional[float] = None) -> tuple[np.ndarray, np.ndarray]:
    """Draft tokens and target argmax tokens for every tree node.

    target_argmax[n] is uniform over the vocabulary. For every non-root node c,
    draft[c] equals target_argmax[parent(c)] with probability `agree`
    (independently per node), else a uniform token among the other VOCAB-1
    ids. The root's draft entry (the anchor) is uniform. ``parent`` holds
    request-local parent indices (-1 at the root), as the tree builder emits.
    """
    q = layout.spec.agree if agree is None else agree
    rng = _rng(layout.seed, 1)
    total = int(node_indptr[-1])
    argmax = rng.integers(0, VOCAB, size=total).astype(np.int64)
    flags = rng.random(total) < q
    other = rng.integers(0, VOCAB - 1, size=total).astype(np.int64)
    draft = np.empty(total, np.int64)
    for b in range(layout.batch):
        s, e = int(node_indptr[b]), int(node_indptr[b + 1])
        par = np.asarray(parent[s:e], np.int64)
        for c in range(e - s):
            g = s + c
            if par[c] < 0:
                draft[g] = other[g]
                continue
            tgt = argmax[s + par[c]]
            draft[g] = tgt if flags[g] else (tgt + 1 + other[g]) % VOCAB
    return draft.astype(np.int32), argmax.astype(np.int32)


def logit_boost(vocab: int, sigma: float, p_top: float) -> float:
    """Logit added to one token so that it takes about probability p_top at
    T = 1 against vocab - 1 others with N(0, sigma^2) logits: the others'
    exp-sum is about vocab * exp(sigma^2 / 2)."""
    return float(np.log(vocab * np.exp(sigma * sigma / 2.0) * p_top / (1.0 - p_top)))


def draw_logits(layout: Layout, preferred: np.ndarray, vocab: int = VOCAB, device="cpu", dtype: str = "bf16",
                sigma: float = 2.0, p_top: float = 0.7, chunk_rows: int = 1024):
    """Target next-token logits per tree node, [len(preferred), vocab]: every
    logit N(0, sigma^2), plus logit_boost(vocab, sigma, p_top) on the node's
    preferred token (the target argmax drawn by draw_tokens), so that at T = 1
    the preferred token is drawn with probability about p_top and acceptance
    resembles the greedy workloads'. Drawn in fp32 from a torch generator
    seeded with seed + 2^32, rounded to the element type."""
    import torch

    dt = torch_dtype(dtype)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(layout.seed) + (1 << 32))
    n = len(preferred)
    out = torch.empty((n, vocab), dtype=dt, device=device)
    boost = logit_boost(vocab, sigma, p_top)
    pref = torch.as_tensor(np.asarray(preferred, np.int64), device=device)
    for s in range(0, n, chunk_rows):
        e = min(n, s + chunk_rows)
        x = torch.randn((e - s, vocab), generator=gen, device=device, dtype=torch.float32) * sigma
        x[torch.arange(e - s, device=device), pref[s:e]] += boost
        out[s:e] = x.to(dt)
    return out


def draw_uniforms(layout: Layout, total_nodes: int) -> np.ndarray:
    """One uniform in [0, 1) per tree node (float32; numpy stream 4), the
    random input of the sampling draws."""
    u = _rng(layout.seed, 4).random(total_nodes, dtype=np.float32)
    return np.minimum(u, np.float32(np.nextafter(np.float32(1.0), np.float32(0.0))))


def torch_dtype(name: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def draw_tensors(layout: Layout, total_nodes: int, device="cpu", dtype: Optional[str] = None,
                 poison_slack: bool = False, chunk_elems: int = 1 << 28) -> dict:
    """Q, paged K/V cache and tree K/V, all N(0, 1), drawn in fp32 from a torch
    generator seeded with the layout seed and rounded to the element type
    (round-to-nearest-even for bf16). With poison_slack, cache slots past a
    request's context length inside its last page hold +1e4 in K and V (they
    must never be attended to)."""
    import torch

    spec = layout.spec
    dt = torch_dtype(dtype or spec.dtype)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(layout.seed))
    D, Hq, Hkv, P = spec.head_dim, spec.hq, spec.hkv, spec.page_size

    def randn(shape):
        out = torch.empty(shape, dtype=dt, device=device)
        flat = out.view(-1)
        n = flat.numel()
        for s in range(0, n, chunk_elems):
            e = min(n, s + chunk_elems)
            flat[s:e] = torch.randn(e - s, generator=gen, device=device, dtype=torch.float32).to(dt)
        return out

    q = randn((total_nodes, Hq, D))
    k_cache = randn((layout.num_pages, Hkv, P, D))
    v_cache = randn((layout.num_pages, Hkv, P, D))
    k_tree = randn((total_nodes, Hkv, D))
    v_tree = randn((total_nodes, Hkv, D))
    if poison_slack:
        for b in range(layout.batch):
            c = int(layout.ctx_len[b])
            if c % P:
                pg = int(layout.page_table[b, c // P])
                k_cache[pg, :, c % P:, :] = 1.0e4
                v_cache[pg, :, c % P:, :] = 1.0e4
    return dict(q=q, k_cache=k_cache, v_cache=v_cache, k_tree=k_tree, v_tree=v_tree)
