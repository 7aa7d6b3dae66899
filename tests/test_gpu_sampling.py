"""GPU parity of the target-token draws for sampling verification (T > 0) and
their argmax form (T = 0) against the oracle, then the whole sampled verify
(draws + accept path) against the oracle's.

Bars: representatives and argmax tokens bit for bit. Drawn tokens bit for bit
wherever the uniform lies farther than CDF_TOL from every cumulative-probability
boundary of its row (the oracle measures this in float64 and moves such
uniforms before the call, or the check falls back to validity). CDF_TOL bounds
how far the kernel's float32 running sums can sit from the float64 ones:
per-lane sums of at most 32 terms, a 6-level lane reduction, the step scan and
the in-step scan give at most ~128 roundings of 2^-24 relative to the total
(7.6e-6), and rounding log2(e)/T and the exponent offsets moves each weight
by at most ~2e-6 relative for the weights that matter; 3e-5 leaves a 3x
margin. Where the uniform is within CDF_TOL of a boundary, the drawn token
must be one whose interval reaches within CDF_TOL of it."""

import numpy as np
import pytest
import torch

from oracle.accept import accept_by_alive
from oracle.sampling import context_reps, sample_targets, sample_token, token_cdf, uniform_margin
from oracle.tree import build_tree, resample_parents, third_level_parents, tree_from_parents
from paper_2606_04446_amd import workload as wl

pytestmark = pytest.mark.gpu

CDF_TOL = 3e-5


def d2sd():
    from paper_2606_04446_amd import d2sd as m
    return m


def flat(trees, drafts):
    ip = np.concatenate([[0], np.cumsum([t.N for t in trees])]).astype(np.int32)
    parent = np.concatenate([t.parent for t in trees]).astype(np.int32)
    draft = np.concatenate(drafts).astype(np.int32)
    return ip, parent, draft


def run_device(trees, drafts, logits, T, u):
    """logits: torch tensor [ΣN, V] (host or device), u: float32 [ΣN]."""
    m = d2sd()
    dev = torch.device("cuda")
    ip, parent, draft = flat(trees, drafts)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    max_nodes = max(t_.N for t_ in trees)
    print(f"sample_targets: batch {len(trees)} nodes {ip[-1]} vocab {logits.shape[1]} T {T} "
          f"dtype {logits.dtype}", flush=True)
    toks, reps = m.sample_targets(t(ip), int(ip[-1]), max_nodes, t(parent), t(draft), logits.to(dev), T,
                                  t(np.asarray(u, np.float32)), want_rep=True)
    torch.cuda.synchronize()
    return toks.cpu().numpy(), reps.cpu().numpy()


def as64(logits):
    return logits.float().cpu().numpy().astype(np.float64)


def settle(trees, drafts, l64, T, u):
    """Move the uniforms of representative nodes that lie within CDF_TOL of a
    boundary of their row (oracle-side; the step is the same for every run)."""
    u = np.array(u, np.float32)
    if T == 0:
        return u
    off = 0
    for t, d in zip(trees, drafts):
        for r in set(context_reps(t.parent, d)):
            g = off + r
            while uniform_margin(l64[g], T, float(u[g])) < CDF_TOL:
                u[g] = np.float32((float(u[g]) + 0.377) % 1.0)
        off += t.N
    return u


def oracle(trees, drafts, l64, T, u):
    reps, toks, off = [], [], 0
    for t, d in zip(trees, drafts):
        r, k = sample_targets(t.parent, d, l64[off:off + t.N], T, u[off:off + t.N])
        reps += r
        toks += k
        off += t.N
    return np.array(reps, np.int32), np.array(toks, np.int32)


def valid_draw(row64, T, u, j):
    """j is a token whose cumulative interval comes within CDF_TOL of u."""
    if not 0 <= j < len(row64) or row64[j] == -np.inf:
        return False
    cdf = token_cdf(row64, T)
    lo = cdf[j - 1] if j > 0 else 0.0
    return lo <= u + CDF_TOL and cdf[j] >= u - CDF_TOL


def small_alphabet_trees(rng, count, B=8, shape="canonical"):
    trees, drafts = [], []
    for _ in range(count):
        if shape == "canonical":
            K = int(rng.integers(0, B))
            t = build_tree(B, sorted(rng.choice(np.arange(1, B), K, replace=False)))
        elif shape == "third":
            p = sorted(rng.choice(np.arange(1, B - 1), int(rng.integers(1, B - 2)), replace=False))
            t = tree_from_parents(third_level_parents(B, p, [int(rng.integers(pk + 1, B)) for pk in p]))
        else:
            t = tree_from_parents(resample_parents(B, int(rng.integers(1, 6))))
        trees.append(t)
        drafts.append(rng.integers(0, 3, t.N).tolist())   # three token ids force repeated contexts
    if shape == "canonical":                     # and one planted repeat of a whole branch tail
        trees.append(build_tree(4, [1, 2]))
        drafts.append([100, 5, 6, 7, 5, 9, 7, 6, 7])
    return trees, drafts


def host_logits(n, V, dtype, seed, sigma=2.0):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((n, V), generator=g) * sigma
    return x.to(wl.torch_dtype(dtype))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V", [1, 7, 1000, 2048, 2049, 4097, 9000])
@pytest.mark.parametrize("T", [0.0, 0.7, 1.0])
def test_draws_match_oracle(dtype, V, T):
    rng = np.random.default_rng(V * 7 + int(T * 10))
    trees, drafts = small_alphabet_trees(rng, 5)
    n = sum(t.N for t in trees)
    logits = host_logits(n, V, dtype, seed=V)
    l64 = as64(logits)
    u = settle(trees, drafts, l64, T, rng.random(n, dtype=np.float32))
    toks, reps = run_device(trees, drafts, logits, T, u)
    want_reps, want_toks = oracle(trees, drafts, l64, T, u)
    assert np.array_equal(reps, want_reps)
    assert (want_reps != np.concatenate([np.arange(t.N) for t in trees])).any()   # repeats were exercised
    assert np.array_equal(toks, want_toks)


@pytest.mark.parametrize("shape", ["third", "resample"])
def test_general_tree_representatives(shape):
    rng = np.random.default_rng(17)
    trees, drafts = small_alphabet_trees(rng, 6, B=10, shape=shape)
    n = sum(t.N for t in trees)
    logits = host_logits(n, 500, "bf16", seed=3)
    l64 = as64(logits)
    u = settle(trees, drafts, l64, 1.0, rng.random(n, dtype=np.float32))
    toks, reps = run_device(trees, drafts, logits, 1.0, u)
    want_reps, want_toks = oracle(trees, drafts, l64, 1.0, u)
    assert np.array_equal(reps, want_reps)
    assert np.array_equal(toks, want_toks)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_uniforms_on_boundaries_give_valid_draws(dtype):
    """Uniforms placed on the float64 boundaries themselves: the kernel may
    land on either side, and must land on a token adjacent to the boundary."""
    rng = np.random.default_rng(9)
    V = 3000
    trees = [build_tree(4, [])] * 8
    drafts = [[0, 1, 2, 3]] * 8                 # no repeats: every node draws its own row
    n = sum(t.N for t in trees)
    logits = host_logits(n, V, dtype, seed=11, sigma=1.0)
    l64 = as64(logits)
    u = np.empty(n, np.float32)
    for g in range(n):
        cdf = token_cdf(l64[g], 1.0)
        u[g] = np.float32(cdf[int(rng.integers(0, V - 1))])
    toks, _ = run_device(trees, drafts, logits, 1.0, u)
    for g in range(n):
        assert valid_draw(l64[g], 1.0, float(u[g]), int(toks[g])), g


def test_edge_rows():
    """One-token rows, -inf entries, u = 0, u just below 1, ties at T = 0 and a
    row with no finite logit."""
    V = 2100                                    # three fp32 steps of 1024, the last one ragged
    rows = np.zeros((8, V), np.float32)
    rows[0, :] = -np.inf
    rows[0, 1234] = 0.5                         # only token 1234 can be drawn
    rows[1, :] = -np.inf                        # no finite logit: -1
    rows[2, :] = 0.0                            # uniform row, u = 0 -> token 0
    rows[3, :] = 0.0
    rows[3, 2050:] = -np.inf                    # u just below 1 -> last finite token 2049
    rows[4, :] = -1.0
    rows[4, [17, 900, 2099]] = 3.0              # T = 0 ties -> first index
    rows[5, :] = np.linspace(-3, 3, V)
    rows[6, ::2] = -np.inf                      # masked even tokens
    rows[6, 1::2] = np.linspace(0, 1, V // 2)
    rows[7, :] = -np.inf
    rows[7, V - 1] = 1.0                        # only the last token of a ragged tail
    u = np.array([0.5, 0.5, 0.0, np.nextafter(np.float32(1), np.float32(0)), 0.5, 0.25, 0.6, 0.9], np.float32)
    trees = [build_tree(2, [])] * 4
    drafts = [[0, 1]] * 4
    logits = torch.from_numpy(rows)
    l64 = rows.astype(np.float64)
    for T in (1.0, 0.0):
        toks, _ = run_device(trees, drafts, logits, T, u)
        for g in range(8):
            if g == 1 or T == 0 or uniform_margin(l64[g], T, float(u[g])) >= CDF_TOL:
                assert toks[g] == sample_token(l64[g], T, float(u[g])), (T, g)
            else:
                assert valid_draw(l64[g], T, float(u[g]), int(toks[g])), (T, g)
        if T > 0:
            assert (toks[0], toks[2], toks[3], toks[7]) == (1234, 0, 2049, V - 1)
    assert (toks[0], toks[3], toks[4], toks[7]) == (1234, 0, 17, V - 1)      # T = 0: first maxima


def test_full_vocabulary_sampled_rows():
    """Workload ctx16k-b32 tree shape (32 requests, B = 16, K = 8) with a
    151,936-entry vocabulary in bf16 at T = 1 and T = 0, launched as the
    benchmark launches it; the oracle checks 48 sampled nodes."""
    layout = wl.draw_layout(4)
    m = d2sd()
    ip, W = m.tree_plan(16, layout.K, layout.p)
    trees = [build_tree(16, layout.p[b, :layout.K[b]]) for b in range(layout.batch)]
    parent = np.concatenate([t.parent for t in trees]).astype(np.int32)
    draft, argmax = wl.draw_tokens(layout, ip, parent)
    drafts = [draft[ip[b]:ip[b + 1]].tolist() for b in range(layout.batch)]
    V = 151_936
    logits = wl.draw_logits(layout, argmax, vocab=V, device="cuda", dtype="bf16")
    u = wl.draw_uniforms(layout, int(ip[-1]))
    rng = np.random.default_rng(4)
    picks = np.sort(rng.choice(int(ip[-1]), 48, replace=False))
    for T in (1.0, 0.0):
        toks, reps = run_device(trees, drafts, logits, T, u)
        want_reps = np.concatenate([context_reps(t.parent, d) for t, d in zip(trees, drafts)])
        assert np.array_equal(reps, want_reps)
        exact = 0
        for g in picks:
            r = int(ip[np.searchsorted(ip, g, side="right") - 1]) + int(reps[g])
            row = logits[r].float().cpu().numpy().astype(np.float64)
            want = sample_token(row, T, float(u[r]))
            if T == 0 or uniform_margin(row, T, float(u[r])) >= CDF_TOL:
                assert toks[g] == want, (T, g)
                exact += 1
            else:
                assert valid_draw(row, T, float(u[r]), int(toks[g])), (T, g)
        # at T = 1 about 30% of the mass sits in intervals ~2e-6 wide, closer
        # than CDF_TOL to a boundary: those draws can only be checked for validity
        assert exact >= (48 if T == 0 else 24)


@pytest.mark.parametrize("cfg", [2, 3])
def test_sampled_verify_matches_oracle(cfg):
    """Tree build -> draws at T = 1 -> accept path, against the oracle's
    sampled verify of every request (vocabulary 32,000)."""
    m = d2sd()
    dev = torch.device("cuda")
    layout = wl.draw_layout(cfg)
    B = layout.spec.B
    ip, W = m.tree_plan(B, layout.K, layout.p)
    total = int(ip[-1])
    trees = [build_tree(B, layout.p[b, :layout.K[b]]) for b in range(layout.batch)]
    parent = np.concatenate([t.parent for t in trees]).astype(np.int32)
    draft, argmax = wl.draw_tokens(layout, ip, parent)
    drafts = [draft[ip[b]:ip[b + 1]].tolist() for b in range(layout.batch)]
    logits = wl.draw_logits(layout, argmax, vocab=wl.VOCAB, device="cpu", dtype="bf16")
    l64 = as64(logits)
    u = settle(trees, drafts, l64, 1.0, wl.draw_uniforms(layout, total))
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    d_ip = t(ip)
    print(f"sampled verify: workload {cfg} nodes {total}", flush=True)
    tree = m.tree_build(B, t(layout.K), t(layout.p), d_ip, total, W)
    max_nodes = int(np.diff(ip).max())
    toks, _ = m.sample_targets(d_ip, total, max_nodes, tree["parent"], t(draft), logits.to(dev), 1.0, t(u))
    res = m.accept_path(B, d_ip, total, tree["parent"], tree["depth"], tree["path_id"], t(draft), toks)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in res.items()}
    off = 0
    accepted = 0
    for b, tr in enumerate(trees):
        _, ref_toks = sample_targets(tr.parent, drafts[b], l64[off:off + tr.N], 1.0, u[off:off + tr.N])
        assert np.array_equal(toks[off:off + tr.N].cpu().numpy(), ref_toks), b
        ref = accept_by_alive(tr, drafts[b], ref_toks)
        pn, tk = ref.padded(B)
        assert got["accept_len"][b] == ref.L and got["accept_node"][b] == ref.node, b
        assert list(got["path_nodes"][b]) == pn and list(got["out_tokens"][b]) == tk, b
        accepted += ref.L
        off += tr.N
    if layout.batch >= 8:                      # one request may reject at its first draft
        assert accepted > 0
