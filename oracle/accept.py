"""Longest accepted prefix across the candidate tree (oracle; test infrastructure).

Sec. 2 ("DFlash"): the target verifies a drafted block by prefix matching,
accepting tokens up to but not including the first mismatch, and its
prediction at the rejection boundary becomes the next anchor (bonus token).
Sec. 3.3 (iv): with K+1 candidates the longest accepted prefix across branches
is committed. Greedy decoding (T = 0): a draft token matches when it equals
the target's argmax prediction after its parent.

Readings:
  * the anchor (root) is already committed; accepted length L counts drafts,
    0 <= L <= B-1, and L+1 tokens are committed (drafts + bonus);
  * equal-length candidates: the first path in canonical order wins (main
    chain, then branches by ascending re-anchor position), which is the
    accepted node of depth L with the lowest canonical index;
  * bonus token = target argmax at the last accepted node.

Two independent derivations are given; tests require them to agree.
"""

from __future__ import annotations

import dataclasses


@dataclasses.dataclass
class Accepted:
    L: int              # accepted draft tokens
    best_path: int      # path of the chosen node (0 = main chain)
    node: int           # chosen (last accepted) node
    path_nodes: list    # nodes at depths 0..L on the chosen path
    tokens: list        # committed tokens: drafts at depths 1..L, then the bonus

    def padded(self, B: int):
        """Rows as the device API lays them out (-1 padded to length B)."""
        pn = self.path_nodes + [-1] * (B - len(self.path_nodes))
        tk = self.tokens + [-1] * (B - len(self.tokens))
        return pn, tk


def accept_by_paths(tree, draft, argmax) -> Accepted:
    """Walk each root-to-leaf candidate and keep the first longest one."""
    best = None
    for k in range(tree.K + 1):
        nodes = tree.path_nodes(k)
        L = 0
        for d in range(1, len(nodes)):
            if draft[nodes[d]] == argmax[nodes[d - 1]]:
                L = d
            else:
                break
        if best is None or L > best[0]:
            best = (L, k, nodes)
    L, k, nodes = best
    chosen = nodes[L]
    toks = [int(draft[nodes[d]]) for d in range(1, L + 1)] + [int(argmax[chosen])]
    return Accepted(L, k, chosen, list(nodes[:L + 1]), toks)


def accept_by_alive(tree, draft, argmax) -> Accepted:
    """Propagate acceptance from the root in node order (parents come first)."""
    alive = [False] * tree.N
    for c in range(tree.N):
        par = tree.parent[c]
        alive[c] = True if par == -1 else (alive[par] and draft[c] == argmax[par])
    L = max(tree.position[c] for c in range(tree.N) if alive[c])
    chosen = min(c for c in range(tree.N) if alive[c] and tree.position[c] == L)
    path, c = [], chosen
    while c != -1:
        path.append(c)
        c = tree.parent[c]
    path = path[::-1]
    toks = [int(draft[n]) for n in path[1:]] + [int(argmax[chosen])]
    return Accepted(L, tree.path[chosen], chosen, path, toks)
