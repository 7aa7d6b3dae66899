"""Committing the accepted path into the paged KV cache (oracle; test infrastructure).

Sec. 3.3: a decoding cycle consumes the verified KV cache of the target and
the bonus token of the previous cycle; after joint verification (iv) the
longest accepted prefix is committed and the target's prediction at the
rejection point becomes the next anchor. So after the accept step of request
b, the tokens at depths 0..L of the chosen path (the anchor, then the L
accepted drafts) join the verified context: their keys and values, computed
in this pass as tree-node K/V, are written at absolute positions C_b .. C_b+L
of the request's paged cache, and the context length becomes C_b + L + 1. The
bonus token is not written: it is the next cycle's anchor, whose K/V that
cycle computes as the root of its tree.

Readings: position C_b + d lives in page page_table[b, (C_b + d) // page_size]
at row (C_b + d) % page_size (the same paging as the context read); the
caller has already placed pages in the table for every position below
C_b + B; nothing else of the cache changes.
"""

from __future__ import annotations

import numpy as np


def commit_accepted(k_cache, v_cache, page_table, ctx_len, node_indptr, path_nodes, accept_len,
                    k_tree, v_tree, page_size: int = 16):
    """Return (k_cache', v_cache', ctx_len') after committing every request's
    accepted path. Inputs are numpy arrays and are not modified:
      k_cache, v_cache [num_pages, Hkv, page_size, D]; page_table [batch, max_pages];
      ctx_len [batch]; node_indptr [batch+1]; path_nodes [batch, B] (local node
      of depth d, -1 past the accepted depth); accept_len [batch] (L);
      k_tree, v_tree [sum N, Hkv, D]."""
    kc = np.array(k_cache, copy=True)
    vc = np.array(v_cache, copy=True)
    ctx = np.array(ctx_len, copy=True)
    for b in range(len(ctx_len)):
        C, L = int(ctx_len[b]), int(accept_len[b])
        for d in range(L + 1):
            node = int(node_indptr[b]) + int(path_nodes[b, d])
            pos = C + d
            page = int(page_table[b, pos // page_size])
            row = pos % page_size
            for h in range(kc.shape[1]):
                kc[page, h, row, :] = k_tree[node, h, :]
                vc[page, h, row, :] = v_tree[node, h, :]
        ctx[b] = C + L + 1
    return kc, vc, ctx
