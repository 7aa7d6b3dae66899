"""Candidate tree of one request (oracle; test infrastructure).

Sec. 3.2 (after Eq. 5): the branch for a selected prefix length i keeps the
anchor and the first i first-draft tokens and re-drafts the remaining
gamma-1-i block positions; sec. 3.3 (iii): every branch agrees with the first
draft on its first i+1 tokens. Fig. 1(b) step 4: the first-draft block and the
K branches form K+1 candidates with shared prefixes.

Readings (the paper gives no node order or mask format):
  * B = gamma counts the anchor at block position 0 (sec. 2, sec. 3.3 (i)).
  * A branch with prefix length i re-anchors at block position p = i + 1 and
    owns one node per position p..B-1; its first node hangs under the
    first-draft node at position p - 1.
  * The anchor is the root (depth 0); a node's depth is its block position.
  * Canonical node order: the main (first-draft) chain 0..B-1, then the
    branches by ascending p, each in position order.
  * No trie merging of equal tokens: the topology depends on (B, p) only.
  * Masks hold ancestor-or-self sets, bit m of a row is word m // 32,
    bit m % 32; a row has ceil((B + B(B-1)/2) / 32) words (the largest tree).
"""

from __future__ import annotations

import dataclasses

import numpy as np


def mask_words(B: int) -> int:
    """Words per mask row: enough bits for the largest tree of block length B."""
    largest = B + B * (B - 1) // 2
    return (largest + 31) // 32


def validate(B: int, p) -> list[int]:
    """Check a branch set; return it sorted ascending."""
    if not isinstance(B, (int, np.integer)) or B < 2:
        raise ValueError(f"block length B must be an integer >= 2, got {B!r}")
    p = [int(x) for x in p]
    if len(p) > B - 1:
        raise ValueError(f"at most B-1 = {B - 1} branches, got {len(p)}")
    if len(set(p)) != len(p):
        raise ValueError(f"re-anchor positions must be distinct, got {p}")
    for x in p:
        if not 1 <= x <= B - 1:
            raise ValueError(f"re-anchor position {x} outside [1, {B - 1}]")
    return sorted(p)


@dataclasses.dataclass
class Tree:
    B: int
    p: list            # re-anchor positions, ascending
    position: list     # block position (= depth) of each node
    path: list         # 0 for the main chain, k for the k-th branch (1-based)
    parent: list       # parent node index, -1 for the root
    ancestors: list    # ancestor-or-self index set of each node

    @property
    def N(self) -> int:
        return len(self.parent)

    @property
    def K(self) -> int:
        return len(self.p)

    @property
    def depth(self) -> list:
        return list(self.position)

    def path_leaf(self) -> list:
        """Last node of each root-to-leaf path: main chain first, then branches."""
        leaf = [None] * (self.K + 1)
        for n in range(self.N):
            leaf[self.path[n]] = n            # nodes of a path appear in position order
        return leaf

    def path_nodes(self, k: int) -> list:
        """Nodes of path k from the root to its leaf, found by walking parents."""
        out = []
        n = self.path_leaf()[k]
        while n != -1:
            out.append(n)
            n = self.parent[n]
        return out[::-1]

    def visible(self) -> np.ndarray:
        """[N, N] bool: entry (n, m) is True iff m is an ancestor-or-self of n."""
        v = np.zeros((self.N, self.N), bool)
        for n, anc in enumerate(self.ancestors):
            for m in anc:
                v[n, m] = True
        return v

    def packed_mask(self, words: int | None = None) -> np.ndarray:
        """[N, words] uint32 ancestor-or-self bits, LSB first."""
        W = mask_words(self.B) if words is None else words
        out = np.zeros((self.N, W), np.uint64)
        for n, anc in enumerate(self.ancestors):
            for m in anc:
                out[n, m // 32] |= np.uint64(1) << np.uint64(m % 32)
        return out.astype(np.uint32)


def build_tree(B: int, p) -> Tree:
    """Tree of one request from block length B and re-anchor positions p."""
    ps = validate(B, p)
    position, path, parent = [], [], []
    for j in range(B):                         # first-draft block: anchor + B-1 drafts
        position.append(j)
        path.append(0)
        parent.append(j - 1)
    for k, pk in enumerate(ps, start=1):       # one branch per selected prefix
        prev = pk - 1                          # main-chain node holding position pk-1
        for j in range(pk, B):
            position.append(j)
            path.append(k)
            parent.append(prev)
            prev = len(parent) - 1
    ancestors = []
    for n in range(len(parent)):               # walk parent pointers into a set
        s, c = set(), n
        while c != -1:
            s.add(c)
            c = parent[c]
        ancestors.append(s)
    return Tree(B, ps, position, path, parent, ancestors)


def tree_from_parents(parent, B: int | None = None) -> Tree:
    """Tree of one request from an arbitrary parent array: the general trees
    of the third-level cascade (sec. 4.3, up to 2K+1 candidates sharing
    prefixes) and of independent resampling (K+1 chains under the anchor).

    Readings (generalising the canonical tree):
      * node 0 is the anchor (root, parent -1); every other node's parent
        precedes it (0 <= parent[n] < n), i.e. nodes are topologically ordered;
      * depth = number of edges to the root;
      * node n starts a new path when its parent is not node n - 1, and
        path[n] counts the path-starting nodes among 1..n (on a canonical tree
        this is the branch number); p lists the depth at which each extra path
        starts (the re-anchor position, for a canonical tree);
      * ancestor-or-self sets by walking parents, as for the canonical tree.
    B defaults to the largest depth + 1."""
    parent = [int(x) for x in parent]
    if not parent or parent[0] != -1:
        raise ValueError("node 0 must be the root (parent -1)")
    for n in range(1, len(parent)):
        if not 0 <= parent[n] < n:
            raise ValueError(f"node {n}: parent {parent[n]} must lie in [0, {n})")
    position, ancestors = [], []
    for n in range(len(parent)):
        s, c = set(), n
        while c != -1:
            s.add(c)
            c = parent[c]
        ancestors.append(s)
        position.append(len(s) - 1)
    path, starts = [], 0
    p = []
    for n in range(len(parent)):
        if n > 0 and parent[n] != n - 1:
            starts += 1
            p.append(position[n])
        path.append(starts)
    if B is None:
        B = max(position) + 1
    return Tree(B, p, position, path, parent, ancestors)


def third_level_parents(B: int, p, q) -> list:
    """Parent array of the third-level cascade tree (sec. 4.3): the canonical
    tree of (B, p) plus, for branch k (ascending p), a sub-branch re-anchored
    at position q[k] (p[k] < q[k] <= B-1) inside that branch's tail: it keeps
    the branch up to q[k] - 1 and owns positions q[k]..B-1. Sub-branches come
    after all branches, in branch order."""
    t = build_tree(B, p)
    parent = list(t.parent)
    for k, pk in enumerate(t.p, start=1):
        qk = int(q[k - 1])
        if not pk < qk <= B - 1:
            raise ValueError(f"sub-branch position {qk} outside ({pk}, {B - 1}]")
        # branch node holding position qk - 1 (the branch itself when qk - 1 >= pk)
        prev = [n for n in range(t.N) if t.path[n] == k and t.position[n] == qk - 1][0]
        for _ in range(qk, B):
            parent.append(prev)
            prev = len(parent) - 1
    return parent


def resample_parents(B: int, chains: int) -> list:
    """Parent array of `chains` independent draft chains of B-1 tokens under
    one anchor (the naive resampling baseline of sec. 1 / sec. 4.3)."""
    parent = [-1]
    for _ in range(chains):
        prev = 0
        for _ in range(1, B):
            parent.append(prev)
            prev = len(parent) - 1
    return parent
