"""GPU parity of the cascade verify attention against the float64 oracle.

Tolerance (max abs over every output element, and over lse): 1e-4 for fp32
inputs, 2e-2 for bf16 inputs, both with fp32 accumulation. The bf16 cases run
in both workgroup shapes (ROW_GROUPS: the automatic choice, which is 128 rows
for these small grids, and 384 rows forced)."""

import numpy as np
import pytest
import torch

from paper_2606_04446_amd import workload as wl
from tests.gpu_cases import TOL, Case, d2sd, max_abs

pytestmark = pytest.mark.gpu

ROW_GROUPS = [0, 384]


def check_full(case, stage="cascade", kv_split=0, out=None, lse=None, row_group=0, packed=0, host_offsets=False):
    code = {"cascade": 0, "prefix": 1, "tree": 2}[stage]
    o, l = case.attention(stage=code, kv_split=kv_split, row_group=row_group, packed=packed,
                          host_offsets=host_offsets)
    torch.cuda.synchronize()
    o = o.double().cpu().numpy()
    l = l.cpu().numpy()
    tol = TOL[case.dtype]
    worst = 0.0
    for b in range(case.layout.batch):
        s, e = int(case.node_indptr[b]), int(case.node_indptr[b + 1])
        ow, lw = case.oracle_attention(b, stage)
        worst = max(worst, max_abs(o[s:e], ow), max_abs(l[s:e], lw))
    assert worst <= tol, (stage, kv_split, worst)
    return worst


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_workload_full(cfg, row_group):
    case = Case(wl.draw_layout(cfg))
    check_full(case, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("cfg", [1, 2])
@pytest.mark.parametrize("stage", ["prefix", "tree"])
def test_workload_stages(cfg, stage, row_group):
    check_full(Case(wl.draw_layout(cfg)), stage, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kv_split", [64, 128, 320, 512])
def test_split_reduction(dtype, kv_split, row_group):
    """Many context splits with a ragged last split exercise the LSE reduction
    (four or more splits in the longest context: the four-group merge; two:
    the one-group merge)."""
    lay = wl.custom_layout(16, [[3, 7], [1], [], [2, 5, 9, 15]], [1000, 129, 64, 1], hq=8, hkv=2,
                           dtype=dtype, seed=11)
    check_full(Case(lay), "cascade", kv_split, row_group=row_group)
    check_full(Case(lay), "prefix", kv_split, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edge_shapes(dtype, row_group):
    # empty contexts, contexts not a multiple of the page or tile size, K = 0,
    # K = B-1, single extreme positions, mixed K in one batch
    rows = [[], list(range(1, 16)), [1], [15], [4, 8, 12], [], [2, 3]]
    ctx = [0, 1, 15, 17, 63, 65, 300]
    lay = wl.custom_layout(16, rows, ctx, hq=4, hkv=2, dtype=dtype, seed=12)
    case = Case(lay)
    for stage in ("cascade", "prefix", "tree"):
        check_full(case, stage, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_contexts_longer_than_one_split(dtype, row_group):
    """Contexts past the longest split (32768 tokens) take several splits and
    page ids past the first 2048 of a request; lengths are not multiples of
    the page or tile size. Automatic split and the longest explicit one."""
    lay = wl.custom_layout(16, [[3, 11], [1, 2, 14]], [70001, 33003], hq=8, hkv=2, dtype=dtype, seed=21)
    case = Case(lay, poison_slack=True)
    check_full(case, row_group=row_group)
    check_full(case, "cascade", kv_split=32768, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("seed", range(8))
def test_random_layouts(seed, row_group):
    """Seeded random batches: block length, re-anchor sets, context lengths
    (page- and tile-ragged, some empty), head grouping, dtype and split
    length all drawn, then every output row against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.choice([2, 3, 5, 8, 13, 16, 24, 32]))
    batch = int(rng.integers(1, 6))
    rows = [sorted(rng.choice(np.arange(1, B), int(rng.integers(0, B)), replace=False).tolist())
            for _ in range(batch)]
    ctx = [int(c) for c in rng.choice([0, 1, 15, 16, 17, 31, 33, 100, 257, 1000, 2049, 3000], batch)]
    hq, hkv = [(4, 1), (8, 2), (16, 4), (32, 8), (12, 3), (8, 8)][int(rng.integers(0, 6))]
    dtype = "f32" if seed % 4 == 3 else "bf16"
    kv_split = int(rng.choice([0, 64, 256, 1024]))
    lay = wl.custom_layout(B, rows, ctx, hq=hq, hkv=hkv, dtype=dtype, seed=seed)
    check_full(Case(lay, poison_slack=True), "cascade", kv_split, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("hq,hkv", [(8, 8), (12, 4), (64, 8), (6, 1), (256, 2)])
def test_gqa_groupings(hq, hkv, row_group):
    lay = wl.custom_layout(16, [[2, 9], [5, 6, 7, 8]], [200, 77], hq=hq, hkv=hkv, dtype="bf16", seed=13)
    check_full(Case(lay), row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
def test_poisoned_slack_is_never_read(row_group):
    lay = wl.custom_layout(16, [[4], [1, 2]], [37, 250], hq=8, hkv=2, dtype="bf16", seed=14)
    check_full(Case(lay, poison_slack=True), row_group=row_group)
    check_full(Case(lay, poison_slack=True), "cascade", kv_split=64, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
@pytest.mark.parametrize("kv_split", [0, 64, 128, 192])
def test_whole_tile_counts_around_the_steady_state(kv_split, row_group):
    """Context lengths giving 0-5 whole 32-key tiles per split, with and
    without a ragged tail, so that the steady-state loop (taken while the
    tile consumed and the tile queued are both whole context tiles) hands
    over to the general loop at every count and stage parity."""
    ctx = [0, 1, 31, 32, 33, 63, 64, 65, 95, 96, 97, 127, 128, 129, 160, 161, 192, 200]
    rng = np.random.default_rng(kv_split)
    p_rows = [sorted(rng.choice(np.arange(1, 16), size=int(rng.integers(0, 4)), replace=False).tolist())
              for _ in ctx]
    lay = wl.custom_layout(16, p_rows, ctx, hq=8, hkv=2, dtype="bf16", seed=16)
    check_full(Case(lay, poison_slack=True), "cascade", kv_split=kv_split, row_group=row_group)
    check_full(Case(lay), "prefix", kv_split=kv_split, row_group=row_group)


@pytest.mark.parametrize("row_group", ROW_GROUPS)
def test_large_block_trees(row_group):
    # B = 64: up to 2080 nodes, masks of 65 words, many tree tiles (4160 rows per
    # request and KV head: 33 row groups of 128 or 11 of 384)
    lay = wl.custom_layout(64, [list(range(1, 64)), [10, 30]], [100, 0], hq=4, hkv=2, dtype="bf16", seed=15)
    check_full(Case(lay), row_group=row_group)


@pytest.mark.parametrize("row_group", [128, 384])
def test_forced_shapes_many_requests(row_group):
    """40 requests with ragged contexts, both shapes forced, against the
    oracle on every row."""
    lay = wl.custom_layout(16, [[1 + (b % 15)] for b in range(40)], [700 + 37 * b for b in range(40)], hq=32,
                           hkv=8, dtype="bf16", seed=17)
    check_full(Case(lay, poison_slack=True), row_group=row_group)


def test_merge_state_recombines_stages():
    m = d2sd()
    case = Case(wl.draw_layout(2))
    op, lp = case.attention(stage=1)
    ot, lt = case.attention(stage=2)
    oc, lc = case.attention(stage=0)
    D = op.shape[-1]
    om, lm = m.merge_state(op.float().reshape(-1, D).contiguous(), lp.reshape(-1).contiguous(),
                           ot.float().reshape(-1, D).contiguous(), lt.reshape(-1).contiguous())
    torch.cuda.synchronize()
    assert max_abs(om.cpu().numpy(), oc.float().reshape(-1, D).cpu().numpy()) <= TOL["bf16"]
    assert max_abs(lm.cpu().numpy(), lc.reshape(-1).cpu().numpy()) <= 1e-4


def test_merge_state_against_oracle():
    from oracle.attention import merge_states
    m = d2sd()
    g = torch.Generator().manual_seed(3)
    rows, D = 300, 128
    o_a, o_b = torch.randn(rows, D, generator=g), torch.randn(rows, D, generator=g)
    l_a, l_b = torch.randn(rows, generator=g) * 3, torch.randn(rows, generator=g) * 3
    l_a[:5] = -float("inf"); l_b[3:8] = -float("inf")
    om, lm = m.merge_state(o_a.cuda(), l_a.cuda(), o_b.cuda(), l_b.cuda())
    ow, lw = merge_states(o_a.double().numpy(), l_a.double().numpy(), o_b.double().numpy(), l_b.double().numpy())
    torch.cuda.synchronize()
    assert max_abs(om.cpu().numpy(), ow) <= 1e-5
    assert max_abs(lm.cpu().numpy(), lw) <= 1e-5


@pytest.mark.parametrize("cfg", [3, 4, 5])
def test_deterministic(cfg):
    """Two calls give the same bits, in the launch the benchmark makes (planned
    from the host node offsets): four-wave groups with twelve splits, one
    384-row workgroup per request and KV head, and the packed kernel with two
    splits and the merge."""
    case = Case(wl.draw_layout(cfg))
    o1, l1 = case.attention(host_offsets=True)
    o2, l2 = case.attention(host_offsets=True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert case.shape(host_offsets=True) == {3: (128, False), 4: (384, False), 5: (384, True)}[cfg]


def test_kernel_timing_per_launch():
    """The library's launch-stream events: one duration per attention launch,
    in launch order, cleared by the read; nothing is recorded while off."""
    m = d2sd()
    case = Case(wl.draw_layout(2))
    case.attention()
    torch.cuda.synchronize()
    m.kernel_timing_collect_each()
    m.kernel_timing_enable(True)
    for _ in range(3):
        case.attention()
    torch.cuda.synchronize()
    m.kernel_timing_enable(False)
    each = m.kernel_timing_collect_each()
    assert len(each) == 3 and all(0.0 < ms < 1000.0 for ms in each)
    assert m.kernel_timing_collect_each() == []
    case.attention()
    torch.cuda.synchronize()
    assert m.kernel_timing_collect() == (0, 0.0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noncascade_baseline(dtype):
    lay = wl.custom_layout(16, [[3, 7], [], [1, 2, 3, 4]], [500, 64, 33], hq=8, hkv=2, dtype=dtype, seed=16)
    case = Case(lay)
    o, l = case.noncascade()
    torch.cuda.synchronize()
    o = o.double().cpu().numpy(); l = l.cpu().numpy()
    for b in range(lay.batch):
        s, e = int(case.node_indptr[b]), int(case.node_indptr[b + 1])
        ow, lw = case.oracle_attention(b)
        assert max(max_abs(o[s:e], ow), max_abs(l[s:e], lw)) <= TOL[dtype]


def sampled_rows(case, n_samples, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n_samples):
        b = int(rng.integers(0, case.layout.batch))
        N = int(case.node_indptr[b + 1] - case.node_indptr[b])
        nodes = sorted({0, N - 1, int(rng.integers(0, N))})
        heads = sorted({0, case.spec.hq - 1, int(rng.integers(0, case.spec.hq))})
        out.append((b, nodes, heads))
    return out


@pytest.mark.parametrize("cfg", [4, 5])
def test_full_size_sampled(cfg):
    """The benchmark's workloads at full size, in the launch configuration the
    benchmark uses (automatic split), checked on sampled rows."""
    case = Case(wl.draw_layout(cfg))
    o, l = case.attention()
    torch.cuda.synchronize()
    tol = TOL[case.dtype]
    for b, nodes, heads in sampled_rows(case, 3, cfg):
        s = int(case.node_indptr[b])
        ow, lw = case.oracle_attention(b, nodes=nodes, heads=heads)
        og = o[[s + n for n in nodes]][:, heads].double().cpu().numpy()
        lg = l[[s + n for n in nodes]][:, heads].cpu().numpy()
        assert max(max_abs(og, ow), max_abs(lg, lw)) <= tol, (cfg, b)
    # properties that hold everywhere: finite outputs, |o| bounded by max |v|
    assert torch.isfinite(o.float()).all() and torch.isfinite(l).all()


# ---- the packed twelve-wave kernel (workgroups over the sequence of all streams' query tiles) ----

def check_packed(lay, kv_split=0, stages=("cascade",), poison=True):
    case = Case(lay, poison_slack=poison)
    for stage in stages:
        code = {"cascade": 0, "prefix": 1, "tree": 2}[stage]
        assert case.shape(kv_split, host_offsets=True, row_group=384, packed=2, stage=code) == (384, True)
        check_full(case, stage, kv_split, row_group=384, packed=2, host_offsets=True)


@pytest.mark.parametrize("seed", range(8))
def test_packed_random_layouts(seed):
    """Random batches with 32 query heads per KV head (a node is a whole
    tile, so every stream holds >= B >= 8 tiles), ragged and empty contexts,
    poisoned page slack, contexts past one split, several split lengths;
    every row against the oracle."""
    rng = np.random.default_rng(3000 + seed)
    batch = int(rng.integers(1, 9))
    B = int(rng.choice([8, 16, 24]))
    rows = [sorted(rng.choice(np.arange(1, B), int(rng.integers(0, B)), replace=False).tolist())
            for _ in range(batch)]
    ctx = [int(c) for c in rng.choice([0, 1, 15, 17, 33, 100, 1000, 3000, 17000, 40000], batch)]
    kv_split = int(rng.choice([0, 64, 256, 1024, 16384])) if max(ctx) <= 3000 else int(rng.choice([0, 16384]))
    lay = wl.custom_layout(B, rows, ctx, hq=64, hkv=2, dtype="bf16", seed=seed)
    check_packed(lay, kv_split)


def test_packed_three_streams_per_workgroup():
    """Exactly six tiles per stream (48 nodes x 4 query heads per KV head):
    twelve consecutive tiles span two or three streams."""
    p = [2, 5, 11, 14]                                  # 16 + 14 + 11 + 5 + 2 = 48 nodes: 192 rows, 6 tiles
    lay = wl.custom_layout(16, [p] * 7, [700, 31, 0, 2000, 64, 333, 1500], hq=8, hkv=2, dtype="bf16", seed=31)
    check_packed(lay, 0, stages=("cascade", "prefix", "tree"))
    check_packed(lay, 256)


def test_packed_largest_batch():
    """The largest batch the packed kernel takes (2048 requests: the block
    scan of the requests' tile counts holds three requests per thread, and the
    binary search over them runs its full depth), small ragged contexts and
    one- to four-node branches; every row against the oracle."""
    rng = np.random.default_rng(2048)
    rows = [sorted(rng.choice(np.arange(1, 8), int(rng.integers(0, 3)), replace=False).tolist())
            for _ in range(2048)]
    ctx = [int(c) for c in rng.choice([0, 1, 16, 17, 40, 64, 100], 2048)]
    lay = wl.custom_layout(8, rows, ctx, hq=64, hkv=2, dtype="bf16", seed=2048)
    check_packed(lay, 0, stages=("cascade", "prefix"))


@pytest.mark.parametrize("kv_split", [0, 1024])
def test_packed_stages_and_tree_tiles(kv_split):
    """Large trees (B = 32, up to 4 tree tiles after the context) in every stage."""
    lay = wl.custom_layout(32, [[1, 5, 9, 20, 31], [], [3, 4, 5, 6, 7, 8], [30]], [4000, 0, 77, 1025], hq=32, hkv=4,
                           dtype="bf16", seed=32)
    check_packed(lay, kv_split, stages=("cascade", "prefix", "tree"))
