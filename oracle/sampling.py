"""Sampling verification of the candidate tree (T > 0) (oracle; test infrastructure).

Tables 3-4 report D^2SD under sampling (T = 1) as well as greedy decoding, and
sec. 5 relies on speculative decoding being lossless through rejection
sampling, but the paper states no acceptance rule for a tree at T > 0.

Reading (the rule this oracle and the device path implement):
  * At every tree node the target's next-token distribution is
    softmax(logits / T) over the vocabulary; one token is drawn from it by
    inversion with a uniform u in [0, 1): the smallest token index j whose
    cumulative probability (in vocabulary order) exceeds u. T = 0 is the
    greedy case: the argmax, lowest index on ties.
  * A non-root node is accepted when its draft token equals the token drawn at
    its parent and its parent is accepted; the accepted length, chosen node and
    bonus token then follow the greedy rule unchanged (deepest accepted node,
    lowest canonical index on ties; bonus = the token drawn at that node).
  * Nodes whose root paths carry the same draft tokens (the same context) share
    one draw: the draw of the lowest-index such node, its representative. Two
    branches can repeat a context when a re-drafted token equals the
    first-draft token at the same position.

This is the rejection-sampling rule of speculative sampling with every drafted
token taken as a point-mass proposal: a child with token x is accepted with
probability p(x); after it is rejected, the residual distribution excludes x
and the next distinct child is tried. Drawing one token per context and
following the child that carries it is the same procedure. The emitted tokens
(accepted drafts, then the bonus) then follow the target's distribution
exactly. The sharing of draws is what keeps this exact on trees that repeat a
context: independent draws at two equal contexts would let the deeper of two
outcomes be chosen, which biases the result.
"""

from __future__ import annotations

import math

import numpy as np

from oracle.accept import accept_by_alive


def context_reps(parent, draft) -> list:
    """Representative of every node of one request: the lowest-index node whose
    root path has the same length and the same draft tokens (the root's own
    token, the anchor, is shared by all and not compared)."""
    first = {}
    reps = []
    for n in range(len(parent)):
        toks, c = [], n
        while parent[c] != -1:
            toks.append(int(draft[c]))
            c = parent[c]
        key = (c, tuple(toks))                 # (root, path tokens leaf to root)
        reps.append(first.setdefault(key, n))
    return reps


def token_cdf(logits, T: float) -> np.ndarray:
    """Cumulative next-token probabilities in vocabulary order (float64), T > 0."""
    x = np.asarray(logits, dtype=np.float64)
    m = np.max(x)
    w = np.exp((x - m) / T)
    return np.cumsum(w) / np.sum(w)


def sample_token(logits, T: float, u: float) -> int:
    """Token drawn from softmax(logits / T) by inversion with uniform u.

    T = 0: argmax, lowest index on ties. T > 0: the smallest j with
    sum_{i <= j} w_i > u * sum_i w_i, where w_i = exp((l_i - max l) / T). If
    rounding leaves no such j, the last token of positive weight is taken.
    A row with no finite logit defines no distribution and gives -1."""
    x = np.asarray(logits, dtype=np.float64)
    if not np.isfinite(np.max(x)):
        return -1
    if T == 0:
        return int(np.argmax(x))               # first maximum
    m = np.max(x)
    w = np.exp((x - m) / T)
    target = float(u) * float(np.sum(w))
    cum = np.cumsum(w)                         # running sums in vocabulary order
    j = int(np.searchsorted(cum, target, side="right"))   # first cum > target
    return j if j < len(w) else int(np.nonzero(w > 0)[0][-1])


def sample_targets(parent, draft, logits, T: float, uniform, dedup: bool = True):
    """(reps, tokens) of one request: the token drawn at every node, each node
    using its representative's logits row and uniform. dedup=False draws at
    every node independently (not the rule; used to show why sharing matters)."""
    reps = context_reps(parent, draft) if dedup else list(range(len(parent)))
    drawn = {}
    tokens = []
    for n, r in enumerate(reps):
        if r not in drawn:
            drawn[r] = sample_token(logits[r], T, uniform[r])
        tokens.append(drawn[r])
    return reps, tokens


def verify_sampled(tree, draft, logits, T: float, uniform, dedup: bool = True):
    """Accepted result of one request under the sampling rule above."""
    reps, tokens = sample_targets(tree.parent, draft, logits, T, uniform, dedup)
    return reps, tokens, accept_by_alive(tree, draft, tokens)


def uniform_margin(logits, T: float, u: float) -> float:
    """Distance from u to the nearest cumulative-probability boundary (T > 0):
    how far rounding in the sums may move before the drawn token can change."""
    cdf = token_cdf(logits, T)
    j = int(np.searchsorted(cdf, u, side="right"))
    lo = cdf[j - 1] if j > 0 else 0.0
    hi = cdf[min(j, len(cdf) - 1)]
    return min(abs(u - lo), abs(hi - u)) if math.isfinite(hi) else 0.0
