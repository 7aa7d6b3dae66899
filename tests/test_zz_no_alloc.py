"""The allocation-free attention entry point (static device scratch) against
the workspace entry point, both through the C ABI: two calls in a row on one
GPU, the second with a smaller input; a batch whose automatic plan does not
fit the scratch; an explicit split that does not fit."""

import numpy as np
import pytest
import torch

from paper_2606_04446_amd import workload as wl
from tests.gpu_cases import TOL, Case, d2sd, max_abs

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20


def call_both(case, kv_split=0, host_offsets=False):
    """(noalloc out, lse), (workspace out, lse), workspace bytes of the plan.
    host_offsets: both calls plan from the host copy of the node offsets, as
    the benchmark does."""
    m = d2sd()
    x = case.x
    ins = (x["q"], x["k_cache"], x["v_cache"], case.d_pt, case.d_ctx, x["k_tree"], x["v_tree"], case.d_ip,
           case.tree["anc_mask"])
    kw = dict(total_nodes=case.total, max_nodes=case.max_nodes,
              max_ctx_len=int(case.layout.ctx_len.max(initial=0)), kv_split=kv_split,
              node_indptr_host=case.node_indptr if host_offsets else None)
    ws = m.cascade_workspace_size(m.attn_args(*ins, x["q"], None, **kw))
    o_ref, l_ref = m.cascade_verify_attention(*ins, **kw)
    o = torch.full_like(x["q"], float("nan"))
    l = torch.full(x["q"].shape[:2], float("nan"), dtype=torch.float32, device=x["q"].device)
    m.cascade_verify_attention_noalloc(*ins, out=o, lse=l, **kw)
    torch.cuda.synchronize()
    return (o, l), (o_ref, l_ref), ws


def test_two_calls_in_a_row_second_smaller():
    # 8 requests, contexts 1024-8192 tokens, splits of 1024: eight splits of partial states in the scratch
    big = Case(wl.draw_layout(3))
    (o, l), (o_ref, l_ref), ws = call_both(big, kv_split=1024)
    assert 0 < ws <= SCRATCH_BYTES
    assert torch.equal(o, o_ref) and torch.equal(l, l_ref)       # same plan, same kernels: bit for bit
    # then one request of 4096 tokens (automatic split of 256: sixteen splits, fewer rows)
    small = Case(wl.draw_layout(2))
    (o2, l2), (o2_ref, l2_ref), ws2 = call_both(small)
    assert 0 < ws2 < ws
    assert torch.equal(o2, o2_ref) and torch.equal(l2, l2_ref)
    # and the first batch again after the smaller call left its contents in the scratch
    (o3, l3), _, _ = call_both(big, kv_split=1024)
    assert torch.equal(o3, o_ref) and torch.equal(l3, l_ref)


def test_automatic_plan_larger_than_the_scratch():
    """The 64-request, 32k-context batch's automatic plan from the host node
    offsets (the packed shape, two splits of 16384 tokens, 173 MB of partial
    states) does not fit: the entry point takes fewer, longer splits (here one,
    which needs none). Every row matches the workspace entry point within the
    bf16 tolerance, and the requests with the smallest and the largest tree
    match the oracle."""
    case = Case(wl.draw_layout(5))
    (o, l), (o_ref, l_ref), ws = call_both(case, host_offsets=True)
    assert ws > SCRATCH_BYTES
    tol = TOL[case.dtype]
    assert max_abs(o.double().cpu().numpy(), o_ref.double().cpu().numpy()) <= tol
    assert max_abs(l.cpu().numpy(), l_ref.cpu().numpy()) <= tol
    o_h, l_h = o.double().cpu().numpy(), l.cpu().numpy()
    sizes = np.diff(case.node_indptr)
    for b in sorted({int(np.argmin(sizes)), int(np.argmax(sizes))}):
        s, e = int(case.node_indptr[b]), int(case.node_indptr[b + 1])
        ow, lw = case.oracle_attention(b)
        assert max(max_abs(o_h[s:e], ow), max_abs(l_h[s:e], lw)) <= tol, b


def test_explicit_split_larger_than_the_scratch_is_rejected():
    m = d2sd()
    case = Case(wl.draw_layout(3))
    x = case.x
    o = torch.full_like(x["q"], float("nan"))
    with pytest.raises(m.D2SDError) as err:
        m.cascade_verify_attention_noalloc(
            x["q"], x["k_cache"], x["v_cache"], case.d_pt, case.d_ctx, x["k_tree"], x["v_tree"], case.d_ip,
            case.tree["anc_mask"], total_nodes=case.total, max_nodes=case.max_nodes,
            max_ctx_len=int(case.layout.ctx_len.max()), kv_split=256, out=o)
    assert err.value.status == m.ERR_WORKSPACE_TOO_SMALL and "static scratch" in str(err.value)
    torch.cuda.synchronize()
    assert torch.isnan(o.float()).all()                                   # nothing launched


def test_single_split_needs_no_scratch():
    """One split per context (the 32-request workload's shape at 1024 tokens):
    no partial states, results equal to the workspace entry point's."""
    lay = wl.custom_layout(16, [[3, 9], [1, 2, 14], []], [1024, 700, 1], hq=32, hkv=8, dtype="bf16", seed=5)
    case = Case(lay)
    (o, l), (o_ref, l_ref), ws = call_both(case, kv_split=1024)
    assert ws == 0
    assert torch.equal(o, o_ref) and torch.equal(l, l_ref)
