"""Closed forms used to pin the oracle (derived independently of its code).

Acceptance under the synthetic token model: every non-root node matches its
parent's target prediction independently with probability q. Let m be the
number of consecutive matches on the main chain from depth 1 (0 <= m <= B-1):
P(m) = q^m (1-q) for m < B-1 and q^(B-1) for m = B-1. Branch k (re-anchor
position p_k, first node at depth p_k under main node p_k - 1) is reachable
iff m >= p_k - 1, and reaches depth j >= p_k iff its j - p_k + 1 nodes all
match. So for j > m:
    P(L >= j | m) = 1 - prod_{k: p_k <= m+1} (1 - q^(j - p_k + 1)),
P(L >= j | m) = 1 for j <= m, and E[L] = sum_{j=1}^{B-1} P(L >= j).
"""


def expected_accept_len(B, p, q):
    total = 0.0
    for j in range(1, B):
        pj = 0.0
        for m in range(B):
            pm = q ** m * (1.0 - q) if m < B - 1 else q ** (B - 1)
            if m >= j:
                pj += pm
                continue
            miss_all = 1.0
            for pk in p:
                if pk <= m + 1:
                    miss_all *= 1.0 - q ** (j - pk + 1)
            pj += pm * (1.0 - miss_all)
        total += pj
    return total
