"""C ABI on the CPU: the library loads, exports the header, and its host logic
(planning, sizing, validation) behaves as documented. No call here reaches a
kernel launch: every device entry point is exercised only on paths that fail
validation before any HIP call."""

import ctypes
import math

import numpy as np
import pytest

from oracle.tree import build_tree, mask_words as oracle_mask_words

d2sd = pytest.importorskip("paper_2606_04446_amd.d2sd")
lib = d2sd._lib

FAKE = 0x1000  # never dereferenced: validation fails before any launch


def test_exports_every_header_function():
    names = d2sd.header_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    assert d2sd.status_string(0) == "ok"
    for s in range(1, 5):
        assert d2sd.status_string(s) not in ("ok", "unknown status")
    assert d2sd.status_string(99) == "unknown status"
    assert d2sd.version() >= 100


def test_mask_words_matches_oracle():
    for B in range(2, 65):
        assert d2sd.mask_words(B) == oracle_mask_words(B)
    assert d2sd.mask_words(1) == 0 and d2sd.mask_words(65) == 0


def test_tree_plan_matches_oracle_node_counts():
    rng = np.random.default_rng(0)
    for _ in range(40):
        B = int(rng.integers(2, 65))
        batch = int(rng.integers(1, 9))
        K = rng.integers(0, B, size=batch)
        kmax = max(1, int(K.max()))
        p = np.zeros((batch, kmax), np.int32)
        for b in range(batch):
            p[b, :K[b]] = rng.permutation(np.arange(1, B))[:K[b]]   # unsorted on purpose
        ip, w = d2sd.tree_plan(B, K, p)
        expect = np.concatenate([[0], np.cumsum([build_tree(B, p[b, :K[b]]).N for b in range(batch)])])
        assert np.array_equal(ip, expect)
        assert w == oracle_mask_words(B)


@pytest.mark.parametrize("B,K,p,msg", [
    (1, [0], [[0]], "B = 1"),
    (65, [0], [[0]], "B = 65"),
    (16, [2], [[3, 3]], "repeated"),
    (16, [1], [[0]], "outside"),
    (16, [1], [[16]], "outside"),
    (4, [4], [[1, 2, 3, 1]], "K = 4"),
])
def test_tree_plan_rejects(B, K, p, msg):
    K = np.asarray(K, np.int32)
    p = np.asarray(p, np.int32)
    out = np.full(len(K) + 1, -7, np.int32)
    st = lib.d2sd_tree_plan(len(K), B, K.ctypes.data, p.ctypes.data, p.shape[1], out.ctypes.data, None)
    assert st == d2sd.ERR_INVALID_ARG
    assert msg in d2sd.last_error()
    assert (out == -7).all()          # outputs untouched on error


def test_tree_plan_validation_agrees_with_oracle():
    """Random (B, K, p), valid or not: the host plan accepts exactly the inputs
    the oracle's validation accepts (B <= 64 on top), with its node counts."""
    from oracle.tree import validate
    rng = np.random.default_rng(21)
    accepted = rejected = 0
    for _ in range(400):
        B = int(rng.integers(0, 68))
        batch = int(rng.integers(1, 5))
        kmax = int(rng.integers(1, 8))
        K = rng.integers(-1, kmax + 2, size=batch).astype(np.int32)
        p = rng.integers(-1, max(B, 1) + 2, size=(batch, kmax)).astype(np.int32)
        ok = 2 <= B <= 64 and all(0 <= K[b] <= kmax for b in range(batch))
        counts = []
        for b in range(batch):
            if not ok:
                break
            try:
                counts.append(build_tree(B, validate(B, p[b, :K[b]].tolist())).N)
            except ValueError:
                ok = False
        out = np.full(batch + 1, -7, np.int32)
        st = lib.d2sd_tree_plan(batch, B, K.ctypes.data, p.ctypes.data, kmax, out.ctypes.data, None)
        if ok:
            accepted += 1
            assert st == d2sd.OK, (B, K, p, d2sd.last_error())
            assert out.tolist() == np.concatenate([[0], np.cumsum(counts)]).tolist()
        else:
            rejected += 1
            assert st == d2sd.ERR_INVALID_ARG, (B, K, p)
            assert (out == -7).all()
    assert accepted > 40 and rejected > 40


def test_tree_plan_null_pointer():
    K = np.zeros(1, np.int32)
    assert lib.d2sd_tree_plan(1, 4, K.ctypes.data, None, 0, None, None) == d2sd.ERR_INVALID_ARG


def test_tree_build_and_accept_validation():
    f = ctypes.c_void_p(FAKE)
    assert lib.d2sd_tree_build(0, 16, 1, f, f, f, 10, 5, f, f, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert lib.d2sd_tree_build(1, 16, 1, f, f, f, 10, 4, f, f, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert "mask_words" in d2sd.last_error()
    assert lib.d2sd_tree_build(1, 16, 1, f, f, f, 10, 5, None, f, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert lib.d2sd_accept_path(1, 1, f, 10, f, f, f, f, f, f, f, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert lib.d2sd_accept_path(1, 16, f, 10, f, f, f, f, f, None, f, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert lib.d2sd_merge_state(4, 0, f, f, f, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert lib.d2sd_merge_state(4, 128, f, None, f, f, f, f, None) == d2sd.ERR_INVALID_ARG


def test_select_reanchor_and_indptr_validation():
    f = FAKE
    sel = d2sd._select
    assert sel(0, 16, 4, f, f, f, None, None) == d2sd.ERR_INVALID_ARG        # batch
    assert sel(1, 1, 4, f, f, f, None, None) == d2sd.ERR_INVALID_ARG         # B < 2
    assert sel(1, 65, 4, f, f, f, None, None) == d2sd.ERR_INVALID_ARG        # B > 64
    assert sel(1, 16, 0, f, f, f, None, None) == d2sd.ERR_INVALID_ARG        # Kmax
    assert sel(1, 16, 4, None, f, f, None, None) == d2sd.ERR_INVALID_ARG     # conf
    assert sel(1, 16, 4, f, f, None, None, None) == d2sd.ERR_INVALID_ARG     # p_out
    ind = d2sd._indptr
    assert ind(0, 16, 4, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert ind(1, 65, 4, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert ind(1, 16, -1, f, f, f, None) == d2sd.ERR_INVALID_ARG
    assert ind(1, 16, 4, f, None, f, None) == d2sd.ERR_INVALID_ARG
    assert ind(1, 16, 4, f, f, None, None) == d2sd.ERR_INVALID_ARG
    assert "NULL" in d2sd.last_error()


def test_commit_validation():
    f = FAKE
    c = d2sd._commit
    ok = dict(batch=1, B=16, hkv=8, D=128, P=16, dt=d2sd.BF16, npages=64, maxp=64, maxc=1000)
    def call(**kw):
        a = {**ok, **kw}
        return c(a["batch"], a["B"], a["hkv"], a["D"], a["P"], a["dt"], a["npages"], a["maxp"], a["maxc"],
                 f, 10, f, f, f, f, f, f, f, f, None)
    assert call(batch=0) == d2sd.ERR_INVALID_ARG
    assert call(B=1) == d2sd.ERR_INVALID_ARG
    assert call(D=64) == d2sd.ERR_UNSUPPORTED
    assert call(P=32) == d2sd.ERR_UNSUPPORTED
    assert call(dt=5) == d2sd.ERR_INVALID_ARG
    assert call(maxc=64 * 16 - 15) == d2sd.ERR_INVALID_ARG     # positions up to C + B must have pages
    assert call(hkv=1 << 26) == d2sd.ERR_UNSUPPORTED             # chunk index of a path past 2^31
    assert "exceeds" in d2sd.last_error()
    assert c(1, 16, 8, 128, 16, d2sd.BF16, 64, 64, 100, f, 10, f, f, f, f, f, None, f, f, None) == d2sd.ERR_INVALID_ARG
    # K/V rows move in 16-byte chunks: every K/V pointer must be 16-byte aligned
    for pos, name in ((13, "k_tree"), (14, "v_tree"), (17, "k_cache"), (18, "v_cache")):
        args = [1, 16, 8, 128, 16, d2sd.BF16, 64, 64, 100, f, 10, f, f, f, f, f, f, f, f, None]
        args[pos] = f + 8
        assert c(*args) == d2sd.ERR_INVALID_ARG, name
        assert name in d2sd.last_error() and "aligned" in d2sd.last_error()


def test_sample_targets_validation():
    f = FAKE
    ok = dict(batch=1, total=10, maxn=10, V=32000, dt=d2sd.BF16, logits=f, T=1.0, u=f)

    def call(**kw):
        a = {**ok, **kw}
        return d2sd._sample(a["batch"], f, a["total"], a["maxn"], f, f, a["V"], a["dt"], a["logits"], a["T"],
                            a["u"], None, f, None)
    assert call(batch=0) == d2sd.ERR_INVALID_ARG
    assert call(total=-1) == d2sd.ERR_INVALID_ARG
    assert call(maxn=0) == d2sd.ERR_INVALID_ARG
    assert call(maxn=2081) == d2sd.ERR_INVALID_ARG
    assert call(batch=2 ** 20, maxn=2080) == d2sd.ERR_INVALID_ARG          # grid beyond 2^31 - 1
    assert call(V=0) == d2sd.ERR_INVALID_ARG
    assert call(V=(1 << 20) + 1) == d2sd.ERR_INVALID_ARG
    assert call(dt=7) == d2sd.ERR_INVALID_ARG
    for T in (-1.0, 1e-7, 2e6, math.inf, math.nan):
        assert call(T=T) == d2sd.ERR_INVALID_ARG, T
    assert call(u=None) == d2sd.ERR_INVALID_ARG                            # T > 0 needs uniforms
    assert call(logits=None) == d2sd.ERR_INVALID_ARG
    assert call(logits=f + 8) == d2sd.ERR_INVALID_ARG                      # alignment
    assert "aligned" in d2sd.last_error()
    assert d2sd._sample(1, f, 10, 10, f, f, 100, d2sd.F32, f, 1.0, f, None, None, None) == d2sd.ERR_INVALID_ARG


def good_args(**kw):
    a = d2sd.AttnArgs()
    a.batch, a.num_qo_heads, a.num_kv_heads, a.head_dim, a.page_size = 32, 32, 8, 128, 16
    a.dtype, a.stage, a.sm_scale = d2sd.BF16, d2sd.STAGE_CASCADE, 0.0
    a.total_nodes, a.max_nodes, a.max_ctx_len = 32 * 80, 108, 16384
    a.num_pages, a.max_pages, a.mask_words, a.kv_split = 32 * 1024, 1024, 5, 0
    for name in ("q", "k_cache", "v_cache", "page_table", "ctx_len", "k_tree", "v_tree", "node_indptr",
                 "anc_mask", "out"):
        setattr(a, name, FAKE)
    a.lse = None
    for k, v in kw.items():
        setattr(a, k, v)
    return a


def ws_size(a):
    n = ctypes.c_size_t(123)
    st = d2sd._ws_size(ctypes.byref(a), ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("field,value,status", [
    ("batch", 0, d2sd.ERR_INVALID_ARG),
    ("num_kv_heads", 5, d2sd.ERR_INVALID_ARG),
    ("head_dim", 64, d2sd.ERR_UNSUPPORTED),
    ("page_size", 32, d2sd.ERR_UNSUPPORTED),
    ("dtype", 7, d2sd.ERR_INVALID_ARG),
    ("stage", 3, d2sd.ERR_INVALID_ARG),
    ("max_nodes", 5000, d2sd.ERR_INVALID_ARG),
    ("max_ctx_len", 16385 + 1024 * 16, d2sd.ERR_INVALID_ARG),
    ("kv_split", 100, d2sd.ERR_INVALID_ARG),
    ("kv_split", 32768 + 64, d2sd.ERR_INVALID_ARG),
    ("mask_words", 3, d2sd.ERR_INVALID_ARG),
    ("num_pages", 0, d2sd.ERR_INVALID_ARG),
])
def test_attention_validation(field, value, status):
    a = good_args(**{field: value})
    assert ws_size(a)[0] == status
    assert d2sd._cascade(ctypes.byref(a), None, 0, None) == status
    assert d2sd.last_error()


def test_attention_null_pointers():
    for name in ("q", "k_cache", "page_table", "ctx_len", "k_tree", "node_indptr", "anc_mask", "out"):
        a = good_args(**{name: None})
        assert d2sd._cascade(ctypes.byref(a), None, 0, None) == d2sd.ERR_INVALID_ARG, name
    # the context-only state does not read the mask
    a = good_args(anc_mask=None, stage=d2sd.STAGE_PREFIX, kv_split=64)
    assert d2sd._cascade(ctypes.byref(a), None, 0, None) == d2sd.ERR_WORKSPACE_TOO_SMALL


def test_attention_alignment():
    """Q, K/V and the output move in 16-byte chunks: a pointer off a 16-byte
    boundary is rejected before any launch (the mask, page table and lse are
    read in 4-byte units and need no more)."""
    for name in ("q", "k_cache", "v_cache", "k_tree", "v_tree", "out"):
        a = good_args(**{name: FAKE + 8})
        assert d2sd._cascade(ctypes.byref(a), None, 0, None) == d2sd.ERR_INVALID_ARG, name
        assert name in d2sd.last_error() and "aligned" in d2sd.last_error()
        assert d2sd._noncascade(ctypes.byref(a), None) == d2sd.ERR_INVALID_ARG, name
    # 4-byte aligned int arrays pass validation (the call stops at the missing workspace, before any launch)
    a = good_args(page_table=FAKE + 4, ctx_len=FAKE + 4, anc_mask=FAKE + 4, node_indptr=FAKE + 4, kv_split=4096)
    assert d2sd._cascade(ctypes.byref(a), None, 0, None) == d2sd.ERR_WORKSPACE_TOO_SMALL


def _with_host_indptr(a, ip):
    ip = np.ascontiguousarray(np.asarray(ip, np.int32))
    a.node_indptr_host = ip.ctypes.data
    a.keep(ip)
    return a


def test_node_indptr_host_validation():
    ip = np.arange(33, dtype=np.int32) * 80            # 32 requests of 80 nodes
    ok = _with_host_indptr(good_args(), ip)
    assert ws_size(ok)[0] == d2sd.OK
    for bad in (ip + 1, np.where(np.arange(33) == 32, 2559, ip), np.where(np.arange(33) == 5, 2000, ip)):
        a = _with_host_indptr(good_args(), bad)
        assert ws_size(a)[0] == d2sd.ERR_INVALID_ARG
        assert "node_indptr_host" in d2sd.last_error()
    big = np.concatenate([[0], np.cumsum([109] + [79] * 31)]).astype(np.int32)   # a request above max_nodes
    assert ws_size(_with_host_indptr(good_args(total_nodes=int(big[-1])), big))[0] == d2sd.ERR_INVALID_ARG


def _best_splits(g, R, s_lo, s_hi):
    """The split count minimising ceil(g s / R) / s, more splits only for >= 3%."""
    best_s, best = s_lo, -(-g * s_lo // R) / s_lo
    for s in range(s_lo + 1, min(s_hi, 4 * s_lo) + 1):
        t = -(-g * s // R) / s
        if t < 0.97 * best:
            best_s, best = s, t
    return best_s, best


def _documented_plan(g4, g12, tiles1, ctx, min_split=256, gain=1.08):
    """(split, rows per workgroup, packed) the planner documents for grids that
    fill the chip with one split: each shape's best split count, and the shape
    with the shorter time, the 384-row shapes counted 8% faster; the packed
    shape (tiles1 query tiles per split, twelve per workgroup, splits of at
    most 16384 tokens) when it is at least as fast as the one-stream one."""
    s_lo = max(1, -(-ctx // 32768))
    s_hi = max(s_lo, ctx // min_split)
    s4, t4 = _best_splits(g4, 768, s_lo, s_hi)
    s12, t12 = _best_splits(g12, 256, s_lo, s_hi)
    s_lo_p = max(s_lo, -(-ctx // 16384))
    ptime = lambda s: -(-(-(-tiles1 * s // 12)) // 256) / s
    sp, tp = s_lo_p, ptime(s_lo_p)
    for s in range(s_lo_p + 1, min(s_hi, 4 * s_lo_p) + 1):
        if ptime(s) < 0.97 * tp:
            sp, tp = s, ptime(s)
    if tiles1 and tp / gain < 0.97 * t12 / gain and tp / gain < t4:
        s, rows, packed = sp, 384, True
    elif t12 / gain < t4:
        s, rows, packed = s12, 384, False
    else:
        s, rows, packed = s4, 128, False
    per = -(-ctx // s)
    return -(-per // 64) * 64, rows, packed


@pytest.mark.parametrize("cfg", [4, 5])
def test_automatic_split_counts_rounds(cfg):
    """Large grids: split count and workgroup shape come from the resident
    rounds of the exact work-item counts (node offsets given on the host)."""
    from paper_2606_04446_amd import workload as wl
    lay = wl.draw_layout(cfg)
    ip, W = d2sd.tree_plan(lay.spec.B, lay.K, lay.p)
    n = np.diff(ip)
    G = lay.spec.hq // lay.spec.hkv
    g4 = int((-(-(n * G) // 128)).sum()) * lay.spec.hkv
    g12 = int((-(-(n * G) // 384)).sum()) * lay.spec.hkv
    t = -(-(n * G) // 32)
    tiles1 = int(t.sum()) * lay.spec.hkv if t.min() >= 6 else 0
    ctx = int(lay.ctx_len.max())
    a = good_args(batch=lay.batch, num_qo_heads=lay.spec.hq, num_kv_heads=lay.spec.hkv, total_nodes=int(ip[-1]),
                  max_nodes=int(n.max()), max_ctx_len=ctx, num_pages=lay.num_pages, max_pages=lay.max_pages,
                  mask_words=W)
    _with_host_indptr(a, ip)
    split = d2sd.cascade_kv_split(a)
    rows, packed = d2sd.cascade_shape(a)
    assert (split, rows, packed) == _documented_plan(g4, g12, tiles1, ctx)
    # 32 requests: 768 four-wave groups (one round), 256 one-stream twelve-wave groups (one round, each
    # context read once) or 224 packed workgroups (also one round: no gain) -> one-stream 384-row
    # workgroups, one split; 64 requests with 64 query heads: 2800 four-wave groups (three splits: 10.9
    # rounds) against 1740 packed workgroups at two splits (6.8 rounds of 256) -> packed, two splits
    assert (g4, -(-ctx // split), rows, packed) == {4: (768, 1, 384, False), 5: (2800, 2, 384, True)}[cfg]
    a.packed = 1                                     # one stream per workgroup: the plans without packing
    assert (d2sd.cascade_kv_split(a), *d2sd.cascade_shape(a)) == _documented_plan(g4, g12, 0, ctx)


def test_row_group_is_validated_and_can_be_forced():
    for bad in (64, 256, 512, -128):
        a = good_args(row_group=bad)
        assert ws_size(a)[0] == d2sd.ERR_INVALID_ARG and "row_group" in d2sd.last_error()
    small = dict(batch=2, total_nodes=100, max_nodes=50, max_ctx_len=1000, num_pages=200, max_pages=100)
    assert d2sd.cascade_row_group(good_args(**small)) == 128          # a small grid: four-wave groups
    assert d2sd.cascade_row_group(good_args(row_group=384, **small)) == 384
    assert d2sd.cascade_row_group(good_args(row_group=128)) == 128
    assert d2sd.cascade_row_group(good_args(row_group=384, dtype=d2sd.F32, **small)) == 128   # fp32: one shape
    for bad in (-1, 3):
        assert ws_size(good_args(packed=bad))[0] == d2sd.ERR_INVALID_ARG and "packed" in d2sd.last_error()
    # packed needs the host node offsets and >= 6 tiles per stream; otherwise one stream per workgroup
    assert d2sd.cascade_shape(good_args(row_group=384, packed=2)) == (384, False)
    ip = np.arange(33, dtype=np.int32) * 80                              # 80 nodes x 4 heads = 10 tiles
    assert d2sd.cascade_shape(_with_host_indptr(good_args(row_group=384, packed=2), ip)) == (384, True)
    ip = np.concatenate([[0], np.cumsum([80] * 31 + [40])]).astype(np.int32)   # one request of 5 tiles
    assert d2sd.cascade_shape(_with_host_indptr(good_args(row_group=384, packed=2, total_nodes=int(ip[-1])),
                                                ip)) == (384, False)
    # the packed kernel stages the tile counts of at most 2048 requests in LDS
    for batch, packed in ((2048, True), (2049, False)):
        ip = np.arange(batch + 1, dtype=np.int32) * 8                      # 8 nodes x 32 heads = 8 tiles
        a = good_args(row_group=384, packed=2, batch=batch, num_qo_heads=64, num_kv_heads=2,
                      total_nodes=8 * batch, max_nodes=8, max_ctx_len=64, num_pages=4 * batch, max_pages=4,
                      mask_words=1)
        assert d2sd.cascade_shape(_with_host_indptr(a, ip)) == (384, packed), batch


def test_workspace_sizing_and_too_small():
    a = good_args(kv_split=4096)
    st, n = ws_size(a)
    assert st == 0
    rows = a.total_nodes * a.num_qo_heads
    assert n == 4 * rows * (128 * 2 + 2 * 4)      # 4 splits: bf16 normalised outputs, fp32 m and l
    a32 = good_args(kv_split=4096, dtype=d2sd.F32)
    assert ws_size(a32) == (0, 4 * rows * (128 * 4 + 2 * 4))   # fp32 inputs keep fp32 partial outputs
    assert d2sd._cascade(ctypes.byref(a), ctypes.c_void_p(FAKE), n - 1, None) == d2sd.ERR_WORKSPACE_TOO_SMALL
    assert "need" in d2sd.last_error()
    a = good_args(kv_split=16384)                  # one split: finalised in place
    assert ws_size(a) == (0, 0)
    a = good_args(stage=d2sd.STAGE_TREE, kv_split=64)
    assert ws_size(a) == (0, 0)


def test_automatic_split():
    a = good_args()
    s = d2sd.cascade_kv_split(a)
    assert s % 64 == 0 and 256 <= s <= 16384
    small = good_args(batch=1, total_nodes=48, max_nodes=48, max_ctx_len=4096, num_pages=256, max_pages=256)
    s2 = d2sd.cascade_kv_split(small)
    assert s2 % 64 == 0 and s2 >= 256 and math.ceil(4096 / s2) > 1


def test_noncascade_validation():
    a = good_args(stage=d2sd.STAGE_PREFIX)
    assert d2sd._noncascade(ctypes.byref(a), None) == d2sd.ERR_INVALID_ARG
    a = good_args(num_qo_heads=8 * 300, num_kv_heads=8)
    assert d2sd._noncascade(ctypes.byref(a), None) == d2sd.ERR_UNSUPPORTED
    a = good_args(max_ctx_len=32768 + 16, max_pages=4096)
    assert d2sd._noncascade(ctypes.byref(a), None) == d2sd.ERR_UNSUPPORTED


def test_timing_collect_empty():
    d2sd.kernel_timing_enable(False)
    assert d2sd.kernel_timing_collect() == (0, 0.0)
    assert d2sd.kernel_timing_collect_each() == []
    assert d2sd.kernel_timing_collect_parts() == ([], [])
    n = ctypes.c_int(-1)
    assert d2sd._timing_parts(0, None, None, ctypes.byref(n)) == d2sd.OK and n.value == 0
    assert d2sd._timing_parts(2, None, None, ctypes.byref(n)) == d2sd.ERR_INVALID_ARG
    n = ctypes.c_int(-1)
    assert d2sd._timing_each(0, None, ctypes.byref(n)) == d2sd.OK and n.value == 0
    assert d2sd._timing_each(-1, None, ctypes.byref(n)) == d2sd.ERR_INVALID_ARG
    assert d2sd._timing_each(4, None, ctypes.byref(n)) == d2sd.ERR_INVALID_ARG
    assert d2sd._timing_each(0, None, None) == d2sd.ERR_INVALID_ARG
