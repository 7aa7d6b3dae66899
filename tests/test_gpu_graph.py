"""A verify step (tree build, cascade attention, accept path) captured in a
HIP graph, in each attention workgroup shape: several replays, with eager work and synchronisations between
them, each checked against the eager result; a replay after an in-place
change of the inputs must see the new values."""

import numpy as np
import pytest
import torch

from paper_2606_04446_amd import workload as wl
from tests.gpu_cases import Case

pytestmark = pytest.mark.gpu


def d2sd():
    from paper_2606_04446_amd import d2sd as m
    return m


def _layout(name):
    """(layout, attention launch options, expected (rows per workgroup, packed))."""
    if name in (2, 3):
        return wl.draw_layout(name), {}, (128, False)
    rng = np.random.default_rng(77)
    rows = [sorted(rng.choice(np.arange(1, 16), int(rng.integers(0, 6)), replace=False).tolist()) for _ in range(6)]
    ctx = [3000, 5000, 17, 2048, 4500, 0]
    if name == "wide":      # one stream per 384-row workgroup, several splits (the merge is captured too)
        lay = wl.custom_layout(16, rows, ctx, hq=32, hkv=8, dtype="bf16", seed=78)
        return lay, dict(kv_split=1024, row_group=384, packed=1), (384, False)
    # workgroups over the sequence of all streams' tiles, planned from the host node offsets
    lay = wl.custom_layout(16, rows, ctx, hq=64, hkv=2, dtype="bf16", seed=79)
    return lay, dict(kv_split=1024, row_group=384, packed=2, host=True), (384, True)


@pytest.mark.parametrize("cfg", [2, 3, "wide", "packed"])
def test_graph_replays_match_eager(cfg):
    m = d2sd()
    lay, opt, want_shape = _layout(cfg)
    case = Case(lay)
    kw = dict(kv_split=opt.get("kv_split", 0), row_group=opt.get("row_group", 0), packed=opt.get("packed", 0),
              node_indptr_host=case.node_indptr if opt.get("host") else None)
    assert case.shape(kw["kv_split"], host_offsets=bool(opt.get("host")), row_group=kw["row_group"],
                      packed=kw["packed"]) == want_shape
    x = case.x
    B, total, W = case.B, case.total, case.W
    dev = torch.device("cuda")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_draft, d_argmax = t(case.draft), t(case.argmax)
    tree = m.tree_build(B, case.d_K, case.d_p, case.d_ip, total, W)
    out = torch.empty_like(x["q"])
    lse = torch.empty(x["q"].shape[:2], dtype=torch.float32, device=dev)
    max_ctx = int(case.layout.ctx_len.max())
    args = m.attn_args(x["q"], x["k_cache"], x["v_cache"], case.d_pt, case.d_ctx, x["k_tree"], x["v_tree"],
                       case.d_ip, tree["anc_mask"], out, lse, total_nodes=total, max_nodes=case.max_nodes,
                       max_ctx_len=max_ctx, **kw)
    ws = torch.empty(max(m.cascade_workspace_size(args), 1), dtype=torch.uint8, device=dev)
    acc = m.accept_path(B, case.d_ip, total, tree["parent"], tree["depth"], tree["path_id"], d_draft, d_argmax)

    def step():
        m.tree_build(B, case.d_K, case.d_p, case.d_ip, total, W, out=tree)
        m.cascade_verify_attention(x["q"], x["k_cache"], x["v_cache"], case.d_pt, case.d_ctx, x["k_tree"],
                                   x["v_tree"], case.d_ip, tree["anc_mask"], total_nodes=total,
                                   max_nodes=case.max_nodes, max_ctx_len=max_ctx, out=out, lse=lse, workspace=ws,
                                   **kw)
        m.accept_path(B, case.d_ip, total, tree["parent"], tree["depth"], tree["path_id"], d_draft, d_argmax,
                      out=acc)

    def snapshot():
        torch.cuda.synchronize()
        return [v.clone() for v in (out, lse, tree["anc_mask"], tree["parent"], *acc.values())]

    step()
    ref = snapshot()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        # clobber every output eagerly, do unrelated eager work, then replay
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        tree["anc_mask"].fill_(-1)
        for v in acc.values():
            v.fill_(-7)
        junk = torch.randn(1 << 20, device=dev).sum()
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        for a, b in zip(got, ref):
            assert torch.equal(a, b), rep
        assert torch.isfinite(junk)
    # the graph reads the live input buffers
    x["q"].mul_(0.5)
    step()
    ref2 = snapshot()
    out.fill_(0.0)
    g.replay()
    got2 = snapshot()
    for a, b in zip(got2, ref2):
        assert torch.equal(a, b)
    assert not torch.equal(ref2[0], ref[0])
