"""Pins of the sampling-verification oracle: closed-form distributions, a
library softmax, the greedy limit, a second derivation of the context
representatives, and exactness of the emitted-token distribution by full
enumeration on small trees."""

import itertools
import math

import numpy as np
import pytest
import scipy.special

from oracle.accept import accept_by_alive
from oracle.sampling import context_reps, sample_token, sample_targets, token_cdf, uniform_margin, verify_sampled
from oracle.tree import build_tree, resample_parents, third_level_parents, tree_from_parents


def test_uniform_logits_closed_form():
    """Equal logits: every token has probability 1/V, so u draws floor(u V)."""
    V = 97
    rng = np.random.default_rng(0)
    for T in (0.5, 1.0, 3.0):
        for u in rng.random(200):
            if min(abs(u * V - round(u * V)), 1.0) < 1e-9:
                continue
            assert sample_token(np.full(V, 2.5), T, u) == math.floor(u * V)


def test_two_tokens_closed_form():
    """Logits (0, d): P(token 0) = 1 / (1 + exp(d / T))."""
    for d, T in ((1.0, 1.0), (-2.0, 0.7), (5.0, 2.0)):
        p0 = 1.0 / (1.0 + math.exp(d / T))
        for u in np.linspace(0.0, 0.999, 400):
            if abs(u - p0) < 1e-12:
                continue
            assert sample_token([0.0, d], T, u) == (0 if u < p0 else 1)


def test_alternating_logits_closed_form_pins_vocabulary_order():
    """Even tokens have logit 0, odd tokens -a, so r = exp(-a / T) and
    F(j) = (#even <= j + r * #odd <= j) / (n (1 + r)) for V = 2n. The weights
    are not monotone in the index, so an inversion over sorted probabilities,
    or over a shuffled order, draws other tokens."""
    n, a, T = 50, 1.3, 0.8
    r = math.exp(-a / T)
    logits = np.array([0.0 if i % 2 == 0 else -a for i in range(2 * n)])

    def F(j):
        ev = j // 2 + 1
        od = (j + 1) // 2
        return (ev + r * od) / (n * (1 + r))

    bounds = [F(j) for j in range(2 * n)]
    np.testing.assert_allclose(token_cdf(logits, T), bounds, rtol=0, atol=1e-14)
    rng = np.random.default_rng(1)
    for u in rng.random(500):
        expect = next(j for j in range(2 * n) if bounds[j] > u)
        if min(abs(u - b) for b in bounds) < 1e-12:
            continue
        assert sample_token(logits, T, u) == expect


def test_interval_lengths_match_library_softmax():
    """The set of u drawing token j has length softmax(l / T)_j: checked on a
    fine midpoint grid of u against scipy's softmax."""
    rng = np.random.default_rng(2)
    V, M = 12, 200_000
    logits = rng.normal(0.0, 2.0, V)
    logits[3] = -np.inf                       # a masked token is never drawn
    for T in (0.6, 1.0, 1.7):
        counts = np.zeros(V)
        us = (np.arange(M) + 0.5) / M
        cdf = token_cdf(logits, T)
        for j in np.searchsorted(cdf, us, side="right"):
            counts[j] += 1
        p = scipy.special.softmax(logits / T)
        np.testing.assert_allclose(counts / M, p, rtol=0, atol=2.0 / M)
        assert counts[3] == 0
        # the vectorised count above and the per-draw definition agree
        for u in us[::4001]:
            assert sample_token(logits, T, u) == int(np.searchsorted(cdf, u, side="right"))


def test_greedy_and_small_temperature_limit():
    """T = 0 is the argmax with the lowest index on ties; a small T with a
    unique maximum ahead by >= 1 draws the argmax for every u."""
    rng = np.random.default_rng(3)
    for _ in range(50):
        logits = rng.integers(-5, 5, 40).astype(float)
        top = int(np.argmax(logits))
        assert sample_token(logits, 0.0, 0.3) == top
        assert all(logits[i] < logits[top] for i in range(top))
        logits[top] += 1.0
        for u in (0.0, 0.5, 0.999999):
            assert sample_token(logits, 1e-3, u) == top


def test_edges():
    assert sample_token([4.0], 1.0, 0.99) == 0                    # one token
    assert sample_token([-np.inf, 0.0, -np.inf, 0.0], 1.0, 0.0) == 1
    assert sample_token([-np.inf, 0.0, -np.inf, 0.0], 1.0, np.nextafter(1.0, 0.0)) == 3
    assert sample_token([0.0, 0.0, 0.0, -np.inf], 1.0, np.nextafter(1.0, 0.0)) == 2
    for T in (0.0, 1.0):
        assert sample_token([-np.inf] * 5, T, 0.5) == -1                # no distribution


def test_temperature_is_a_logit_scale():
    """softmax(l / T) at temperature T equals softmax(l / T) at temperature 1."""
    rng = np.random.default_rng(4)
    logits = rng.normal(0, 3, 64)
    for T in (0.25, 2.0):
        for u in rng.random(100):
            if uniform_margin(logits, T, u) < 1e-9:
                continue
            assert sample_token(logits, T, u) == sample_token(logits / T, 1.0, u)


# ---------------------------------------------------------------- reps --

def reps_by_recursion(parent, draft):
    """Second derivation: two nodes share a context iff their parents share one
    and their tokens are equal; parents precede children, so one pass in
    index order resolves every node."""
    reps = []
    for n in range(len(parent)):
        if parent[n] == -1:
            reps.append(n)
            continue
        pr = reps[parent[n]]
        reps.append(next(m for m in range(n + 1)
                         if parent[m] != -1 and reps[parent[m]] == pr and draft[m] == draft[n]))
    return reps


def test_context_reps_hand_case():
    """B = 4, p = (1, 2): main chain 0-1-2-3 (tokens 5 6 7), branch 1 = nodes
    4 5 6 under the anchor (tokens 5 9 7), branch 2 = nodes 7 8 under node 1
    (tokens 6 7). Node 4 repeats node 1's context (5); node 7 repeats node 2's
    (5 6) and node 8 node 3's (5 6 7). Node 5 (5 9) is new, and so is node 6."""
    t = build_tree(4, [1, 2])
    draft = [100, 5, 6, 7, 5, 9, 7, 6, 7]
    assert t.parent == [-1, 0, 1, 2, 0, 4, 5, 1, 7]
    assert context_reps(t.parent, draft) == [0, 1, 2, 3, 1, 5, 6, 2, 3]


@pytest.mark.parametrize("shape", ["canonical", "third", "resample"])
def test_context_reps_two_derivations(shape):
    rng = np.random.default_rng(5)
    for _ in range(200):
        B = int(rng.integers(2, 9))
        if shape == "canonical":
            K = int(rng.integers(0, B))
            parent = build_tree(B, sorted(rng.choice(np.arange(1, B), K, replace=False))).parent
        elif shape == "third":
            if B < 3:
                continue
            p = sorted(rng.choice(np.arange(1, B - 1), int(rng.integers(0, B - 2)), replace=False))
            q = [int(rng.integers(pk + 1, B)) for pk in p]
            parent = third_level_parents(B, p, q)
        else:
            parent = resample_parents(B, int(rng.integers(1, 5)))
        draft = rng.integers(0, 3, len(parent)).tolist()   # a 3-token alphabet forces repeats
        assert context_reps(parent, draft) == reps_by_recursion(parent, draft)


# ---------------------------------------------------- exactness by enumeration --

def target_logits(context, V, seed):
    """A fixed, context-dependent target model for the enumeration tests."""
    h = seed
    for tok in context:
        h = (h * 1_000_003 + 7919 * (tok + 1)) % (2 ** 61 - 1)
    return np.random.default_rng(h).normal(0.0, 0.7, V)


def path_context(parent, draft, n):
    ctx = []
    while parent[n] != -1:
        ctx.append(int(draft[n]))
        n = parent[n]
    return tuple(ctx[::-1])


def emitted_distribution(tree, draft, V, T, seed, dedup=True):
    """Exact distribution of the emitted tokens (accepted drafts, then the
    bonus), padded to B tokens by the target's own continuation: enumerate the
    token drawn at every representative node, drawing it through the oracle
    with u at the midpoint of that token's interval, weighted by the interval
    length."""
    B = tree.B
    ctx = [path_context(tree.parent, draft, n) for n in range(tree.N)]
    logits = np.array([target_logits(c, V, seed) for c in ctx])
    reps = context_reps(tree.parent, draft) if dedup else list(range(tree.N))
    uniq = sorted(set(reps))
    cdfs = {r: token_cdf(logits[r], T) for r in uniq}
    dist = {}
    for choice in itertools.product(range(V), repeat=len(uniq)):
        u = np.zeros(tree.N)
        w = 1.0
        for r, j in zip(uniq, choice):
            lo = cdfs[r][j - 1] if j else 0.0
            hi = cdfs[r][j]
            w *= hi - lo
            u[r] = 0.5 * (lo + hi)
        if w == 0.0:
            continue
        _, _, acc = verify_sampled(tree, draft, logits, T, u, dedup=dedup)
        seqs = {tuple(acc.tokens): w}
        while len(next(iter(seqs))) < B:          # continue with the target itself
            nxt = {}
            for s, ws in seqs.items():
                p = scipy.special.softmax(target_logits(s, V, seed) / T)
                for j in range(V):
                    nxt[s + (j,)] = nxt.get(s + (j,), 0.0) + ws * p[j]
            seqs = nxt
        for s, ws in seqs.items():
            dist[s] = dist.get(s, 0.0) + ws
    return dist


def autoregressive_distribution(B, V, T, seed):
    dist = {}
    for s in itertools.product(range(V), repeat=B):
        pr = 1.0
        for k in range(B):
            pr *= scipy.special.softmax(target_logits(s[:k], V, seed) / T)[s[k]]
        dist[s] = pr
    return dist


def tree_cases():
    # canonical tree, re-drafted branch repeating the first draft's position-1 token
    yield build_tree(3, [1]), [9, 0, 1, 0, 2]
    # canonical tree, no repeated context
    yield build_tree(3, [1, 2]), [9, 0, 1, 2, 0, 1]
    # three resampled chains, two of them identical
    yield tree_from_parents(resample_parents(3, 3)), [9, 1, 2, 1, 2, 0, 1]


@pytest.mark.parametrize("case", range(3))
@pytest.mark.parametrize("T", [1.0, 0.6])
def test_emitted_tokens_follow_the_target_exactly(case, T):
    tree, draft = list(tree_cases())[case]
    V, seed = 3, 11 + case
    got = emitted_distribution(tree, draft, V, T, seed)
    want = autoregressive_distribution(tree.B, V, T, seed)
    assert set(got) <= set(want)
    for s, pw in want.items():
        assert got.get(s, 0.0) == pytest.approx(pw, abs=1e-12), s


@pytest.mark.parametrize("case", [0, 2])
def test_independent_draws_at_repeated_contexts_are_biased(case):
    """Planted mistake: drawing at every node separately. On the trees that
    repeat a context the emitted distribution then leaves the target's."""
    tree, draft = list(tree_cases())[case]
    V, seed, T = 3, 11 + case, 1.0
    got = emitted_distribution(tree, draft, V, T, seed, dedup=False)
    want = autoregressive_distribution(tree.B, V, T, seed)
    assert max(abs(got.get(s, 0.0) - pw) for s, pw in want.items()) > 1e-3


def test_greedy_rule_is_the_zero_temperature_case():
    """At T = 0 the sampled path equals the greedy accept on argmax tokens."""
    rng = np.random.default_rng(6)
    for _ in range(100):
        B = int(rng.integers(2, 8))
        K = int(rng.integers(0, B))
        t = build_tree(B, sorted(rng.choice(np.arange(1, B), K, replace=False)))
        draft = rng.integers(0, 4, t.N).tolist()
        logits = rng.integers(-3, 3, (t.N, 4)).astype(float)
        # repeated contexts must see equal rows for argmax to be consistent
        reps = context_reps(t.parent, draft)
        logits = logits[reps]
        _, toks, acc = verify_sampled(t, draft, logits, 0.0, rng.random(t.N))
        ref = accept_by_alive(t, draft, [int(np.argmax(r)) for r in logits])
        assert (acc.L, acc.node, acc.tokens) == (ref.L, ref.node, ref.tokens)


def test_representatives_use_their_own_row_and_uniform():
    t = build_tree(3, [1])
    draft = [9, 0, 1, 0, 2]                    # node 3 repeats node 1
    logits = np.zeros((5, 4))
    u = np.array([0.1, 0.3, 0.6, 0.9, 0.95])
    reps, toks = sample_targets(t.parent, draft, logits, 1.0, u)
    assert reps == [0, 1, 2, 1, 4]
    assert toks == [0, 1, 2, 1, 3]             # uniform logits: floor(4 u) of the representative
