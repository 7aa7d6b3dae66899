"""Rejection-boundary posterior and top-K prefix selection (oracle; test infrastructure).

Eq. 3: c_k is the first drafter's confidence at block position k = 1..gamma-1.
Eq. 4: r(i) = (prod_{k=1..i} c_k) * (1 - c_{i+1}), i = 0..gamma-2, the chance
that exactly i drafts are accepted. Eq. 5: the K prefix lengths with the
largest r(i) are kept; sec. 3.3 (ii): each becomes a re-anchoring point.

Readings: ties in r(i) go to the smaller i; a kept prefix length i gives the
re-anchor block position p = i + 1.
"""

from __future__ import annotations

import math


def rejection_posterior(conf) -> list:
    """r(0..gamma-2) from confidences c_1..c_{gamma-1} (conf[0] is c_1)."""
    conf = [float(x) for x in conf]
    r = []
    for i in range(len(conf)):
        prod = 1.0
        for k in range(1, i + 1):
            prod *= conf[k - 1]
        r.append(prod * (1.0 - conf[i]))      # (1 - c_{i+1}), conf[i] = c_{i+1}
    return r


def top_k_prefixes(r, K: int) -> list:
    """Indices i of the K largest r(i); ties go to the smaller i.

    The paper assumes confidences in [0, 1]. Outside that range r(i) can be
    NaN; such an r(i) is read as the least likely prefix length (it ranks
    below every number, -inf included, ties again by index)."""
    def rank_key(i):
        return (math.inf if math.isnan(r[i]) else -r[i], i)
    order = sorted(range(len(r)), key=rank_key)
    return sorted(order[:K])


def reanchor_positions(conf, K: int) -> list:
    """Re-anchor block positions p = i + 1 for the top-K prefix lengths."""
    return [i + 1 for i in top_k_prefixes(rejection_posterior(conf), K)]
