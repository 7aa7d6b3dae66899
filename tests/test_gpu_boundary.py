"""GPU parity of device re-anchor selection (Eq. 4-5) and device tree offsets.

r(i) and the kept positions must equal the oracle's bit for bit: both sides
evaluate r in float64 with the same operation order, from the same float32
confidences, and break ties the same way (smaller prefix length first)."""

import numpy as np
import pytest
import torch

from oracle.boundary import rejection_posterior, reanchor_positions
from oracle.tree import build_tree
from tests.gpu_cases import oracle_tree_arrays

pytestmark = pytest.mark.gpu


def d2sd():
    from paper_2606_04446_amd import d2sd as m
    return m


def draw_conf(rng, kind, batch, n):
    if kind == "uniform":
        c = rng.random((batch, n))
    elif kind == "beta52":
        c = rng.beta(5.0, 2.0, (batch, n))
    elif kind == "constant":
        c = np.repeat(rng.random((batch, 1)), n, axis=1)
    elif kind == "quantized":     # many exact ties, exact 0 and 1
        c = rng.choice([0.0, 0.25, 0.5, 0.75, 1.0], size=(batch, n))
    elif kind == "extreme":
        c = rng.choice([0.0, 1.0, 1e-30, 1.0 - 2 ** -24], size=(batch, n))
    elif kind == "invalid":       # outside [0, 1]: NaN and +-inf posteriors
        c = rng.choice([np.nan, np.inf, -np.inf, -0.5, 1.5, 0.0, 0.3, 0.7, 1.0], size=(batch, n))
    else:
        raise ValueError(kind)
    return c.astype(np.float32)


def check_select(B, Kmax, kind, seed, batch=64):
    m = d2sd()
    rng = np.random.default_rng([seed, B, Kmax])
    n = B - 1
    conf = draw_conf(rng, kind, batch, n)
    K = rng.integers(0, min(Kmax, n) + 1, size=batch).astype(np.int32)
    K[0] = min(Kmax, n)                       # always one full selection
    dev = torch.device("cuda")
    p, r = m.select_reanchor(B, torch.from_numpy(conf).to(dev), torch.from_numpy(K).to(dev), Kmax, want_r=True)
    torch.cuda.synchronize()
    p, r = p.cpu().numpy(), r.cpu().numpy()
    for b in range(batch):
        r_or = np.array(rejection_posterior(conf[b]), dtype=np.float64)
        assert np.array_equal(r[b], r_or, equal_nan=True), (B, kind, b, r[b], r_or)
        want = reanchor_positions(conf[b], int(K[b]))
        got = p[b].tolist()
        assert got == want + [-1] * (Kmax - len(want)), (B, kind, b, got, want)


@pytest.mark.parametrize("kind", ["uniform", "beta52", "constant", "quantized", "extreme", "invalid"])
@pytest.mark.parametrize("B", [2, 3, 4, 16, 33, 64])
def test_select_reanchor_matches_oracle(B, kind):
    check_select(B, max(1, min(8, B - 1)), kind, seed=7)


def test_select_reanchor_full_and_wide_kmax():
    check_select(16, 15, "beta52", seed=1)      # K up to B - 1 (every position)
    check_select(16, 40, "uniform", seed=2)     # Kmax above B - 1: rows padded with -1
    check_select(64, 63, "quantized", seed=3)


@pytest.mark.parametrize("B", [4, 16, 64])
def test_select_reanchor_invalid_confidences_stay_in_bounds(B):
    """NaN posteriors rank last (the oracle's reading), so exactly K positions
    are written per request: a guard region after p_out stays untouched."""
    m = d2sd()
    rng = np.random.default_rng([11, B])
    batch, Kmax, guard = 32, 3, 256
    conf = draw_conf(rng, "invalid", batch, B - 1)
    K = np.full(batch, min(Kmax, B - 1), dtype=np.int32)
    dev = torch.device("cuda")
    buf = torch.full((batch * Kmax + guard,), -7, dtype=torch.int32, device=dev)
    p_out = buf[:batch * Kmax].view(batch, Kmax)
    p, _ = m.select_reanchor(B, torch.from_numpy(conf).to(dev), torch.from_numpy(K).to(dev), Kmax, p_out=p_out)
    torch.cuda.synchronize()
    assert (buf[batch * Kmax:] == -7).all().item()
    got = p.cpu().numpy()
    for b in range(batch):
        assert got[b].tolist() == reanchor_positions(conf[b], int(K[b])), (B, b, conf[b], got[b])


def test_select_reanchor_clamps_k():
    m = d2sd()
    dev = torch.device("cuda")
    conf = torch.full((3, 15), 0.5, dtype=torch.float32, device=dev)
    K = torch.tensor([-3, 99, 2], dtype=torch.int32, device=dev)
    p, _ = m.select_reanchor(16, conf, K, 4)
    torch.cuda.synchronize()
    assert p.cpu().tolist() == [[-1, -1, -1, -1], [1, 2, 3, 4], [1, 2, -1, -1]]


@pytest.mark.parametrize("batch", [1, 255, 256, 257, 1000])
def test_tree_indptr_matches_host_plan(batch):
    m = d2sd()
    rng = np.random.default_rng(batch)
    B, Kmax = 16, 8
    K = rng.integers(0, Kmax + 1, size=batch).astype(np.int32)
    p = np.zeros((batch, Kmax), np.int32)
    for b in range(batch):
        p[b, :K[b]] = rng.choice(np.arange(1, B), size=K[b], replace=False)
    ip_host, _ = m.tree_plan(B, K, p)
    dev = torch.device("cuda")
    ip = m.tree_indptr(B, torch.from_numpy(K).to(dev), torch.from_numpy(p).to(dev))
    torch.cuda.synchronize()
    assert np.array_equal(ip.cpu().numpy(), ip_host)


def test_select_then_tree_on_device_matches_oracle():
    """Confidences -> re-anchor positions -> node offsets -> tree, all on the
    device, against the oracle's selection and tree built from it."""
    m = d2sd()
    rng = np.random.default_rng(11)
    B, Kmax, batch = 16, 4, 48
    conf = draw_conf(rng, "beta52", batch, B - 1)
    K = np.full(batch, Kmax, np.int32)
    dev = torch.device("cuda")
    dK = torch.from_numpy(K).to(dev)
    p, _ = m.select_reanchor(B, torch.from_numpy(conf).to(dev), dK, Kmax)
    ip = m.tree_indptr(B, dK, p)
    trees = [build_tree(B, reanchor_positions(conf[b], Kmax)) for b in range(batch)]
    total = sum(t.N for t in trees)
    W = m.mask_words(B)
    tree = m.tree_build(B, dK, p, ip, total, W)
    torch.cuda.synchronize()
    ip_or = np.concatenate([[0], np.cumsum([t.N for t in trees])]).astype(np.int32)
    assert np.array_equal(ip.cpu().numpy(), ip_or)
    parent, depth, path, mask, leaf = oracle_tree_arrays(trees, W, Kmax)
    assert np.array_equal(tree["parent"].cpu().numpy(), parent)
    assert np.array_equal(tree["depth"].cpu().numpy(), depth)
    assert np.array_equal(tree["path_id"].cpu().numpy(), path)
    assert np.array_equal(tree["anc_mask"].cpu().numpy(), mask)
    assert np.array_equal(tree["path_leaf"].cpu().numpy(), leaf)
