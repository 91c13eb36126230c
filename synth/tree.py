"""Seeded draft trees (input generation only; none of the method's arithmetic).

A tree of n nodes is a parent array: node 0 is the root (parent -1) and every other node's
parent has a smaller index.  ``ddtree_like`` mimics a tree drafter (Sec. 4.3, DDTree): one
drafting pass proposes, at each of D depths, a few candidate tokens with probabilities, and
the tree keeps the n most probable prefixes (best-first by the product of their
candidates' probabilities), so that shallow, likely branches are dense and deep ones thin."""
import heapq

import numpy as np


def ddtree_like(seed, n_nodes, depth, branch, vocab):
    """(parents int32 [n], tokens int32 [n] with tokens[0] = -1 for the caller's root, depth of
    every node).  Candidate tokens per depth: `branch` distinct ids with Dirichlet(0.5)
    probabilities; the children of a node at depth d are the candidates of depth d + 1."""
    rng = np.random.default_rng([seed, 0x7EE])
    cand = [rng.choice(vocab, size=branch, replace=False) for _ in range(depth)]
    prob = [np.sort(rng.dirichlet(np.full(branch, 0.5)))[::-1] for _ in range(depth)]
    parents, tokens, depths = [-1], [-1], [0]
    heap = [(-prob[0][j], 0, 0, j) for j in range(branch)]  # (-score, parent node, depth of parent, candidate)
    heapq.heapify(heap)
    while len(parents) < n_nodes and heap:
        neg, par, d, j = heapq.heappop(heap)
        node = len(parents)
        parents.append(par)
        tokens.append(int(cand[d][j]))
        depths.append(d + 1)
        if d + 1 < depth:
            for jj in range(branch):
                heapq.heappush(heap, (neg * prob[d + 1][jj], node, d + 1, jj))
    return np.array(parents, np.int32), np.array(tokens, np.int32), np.array(depths, np.int32)


def random_tree(seed, n_nodes, max_depth):
    """Parents of a random tree: each node hangs under a uniformly drawn earlier node whose depth
    is below max_depth."""
    rng = np.random.default_rng([seed, 0x7EF])
    parents, depths = [-1], [0]
    for r in range(1, n_nodes):
        ok = [i for i in range(r) if depths[i] < max_depth]
        p = int(ok[rng.integers(0, len(ok))])
        parents.append(p)
        depths.append(depths[p] + 1)
    return np.array(parents, np.int32), np.array(depths, np.int32)
