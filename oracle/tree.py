"""Tree verification: acceptance and cache commit (oracle).  Test infrastructure only.

The paper's strongest configurations draft a tree of candidates rather than one chain
(DDTree, Sec. 4.3 and Table 2; Appendix B gives node budgets of 64 to 512).  The target
scores every node in one forward pass -- ``forward.verify_block`` with ``parents`` --
where node r sits at position C + depth(r), is stored at cache slot C + r and attends to
the cached context and to its ancestors' slots.  The paper states no tree acceptance
procedure; under greedy decoding (temperature 0) the plain one is the longest accepted
root-to-node path:

* a node r > 0 is accepted with its parent when its token is the token the target ranks
  first at the parent (argmax of the parent's row, first index of the maximum); a node is
  reachable when it and every ancestor below the root are accepted (the root always is);
* the last node of the path is the deepest reachable node, the smallest index among equally
  deep ones; its ancestors form the path, and a = its depth is the number of drafts kept;
* the emitted tokens are the path's tokens below the root followed by the argmax of the last
  node's row (a correction, or the bonus token at a leaf);
* commit: the accepted nodes' K/V move from their tree slots C + path[k] to the positions
  C + k they hold in the sequence (k = 1..a; the root stays at C), and the cached length
  becomes C + a + 1.  Their rotary positions C + depth = C + k are already right, so the
  move is a copy.

On every root-to-leaf path the chain rule (``accept.accept_greedy``) keeps the path's
reachable prefix, so the tree keeps the longest of those.
"""
import numpy as np

from .accept import argmax_first
from .forward import LSV_ERR_INVALID_ARG, LSV_OK, ancestors, tree_depths


def accept_tree_greedy(logits, row_offsets, tokens, parents, width):
    """Per sequence: (accept_len, emitted tokens padded with -1 to `width`, path of node
    indices padded with -1, status).  A tree whose parents are invalid, or whose accepted
    path would not fit `width` entries, gets LSV_ERR_INVALID_ARG and emits nothing."""
    off = [int(x) for x in row_offsets]
    B = len(off) - 1
    acc = np.zeros(B, np.int32)
    out = np.full((B, width), -1, np.int32)
    path = np.full((B, width), -1, np.int32)
    status = np.zeros(B, np.int32)
    for b in range(B):
        r0, n = off[b], off[b + 1] - off[b]
        par = [int(p) for p in parents[r0:r0 + n]]
        if n < 1 or tree_depths(par) is None:
            status[b] = LSV_ERR_INVALID_ARG
            continue
        if not np.all(np.isfinite(logits[r0:r0 + n])):
            status[b] = -5  # LSV_ERR_NONFINITE
            continue
        depth = tree_depths(par)
        top = [argmax_first(logits[r0 + u]) for u in range(n)]
        reach = [True] + [False] * (n - 1)
        for c in range(1, n):  # parents precede children
            reach[c] = reach[par[c]] and int(tokens[r0 + c]) == top[par[c]]
        last = 0
        for c in range(1, n):
            if reach[c] and depth[c] > depth[last]:
                last = c
        walk = [int(x) for x in ancestors(par, last)]
        a = len(walk) - 1
        if a + 1 > width:
            status[b] = LSV_ERR_INVALID_ARG
            continue
        acc[b] = a
        for k in range(1, a + 1):
            out[b, k - 1] = int(tokens[r0 + walk[k]])
        out[b, a] = argmax_first(logits[r0 + walk[-1]])
        path[b, :a + 1] = walk
        status[b] = LSV_OK
    return {"accept_len": acc, "out_tokens": out, "path": path, "status": status}


def compact(cache, seq_len, result):
    """Move every accepted node's K/V from slot C + path[k] to position C + k (in increasing
    k), then commit seq_len[b] = C + a + 1; sequences whose status is not OK are left alone.
    seq_len is the length before the round (C)."""
    new = np.array(seq_len, dtype=np.int64).copy()
    for b in range(len(new)):
        if result["status"][b] != LSV_OK:
            continue
        C, a = int(new[b]), int(result["accept_len"][b])
        for l in range(len(cache.k)):
            for k in range(1, a + 1):
                src = C + int(result["path"][b, k])
                cache.k[l][b, :, C + k, :] = cache.k[l][b, :, src, :]
                cache.v[l][b, :, C + k, :] = cache.v[l][b, :, src, :]
        new[b] = C + a + 1
    return new
