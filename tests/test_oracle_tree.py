"""Pins of the tree-verification oracle (oracle/forward.py with parents, oracle/tree.py).

* A chain tree (parent r - 1) is the plain causal block: identical logits and cache.
* Every node's logits and K/V equal those of a plain verify of its root-to-node path, which
  is the definition of tree attention (ancestors only, rotary position = depth); this is
  checked node by node on random trees (fp32 and bf16 shapes).
* Tree acceptance against brute force: the chain rule (accept.accept_greedy) applied to
  every root-to-leaf path; the tree result is the longest of them, with its tokens.
* Commit: after moving the accepted nodes' K/V, the cache holds exactly what verifying the
  accepted path as a chain writes, and decoding on from it gives the same logits.
* Invalid parent arrays are refused."""
import copy

import numpy as np
import pytest

from oracle import accept as OA
from oracle import forward as OF
from oracle import tree as OT
from synth import configs, gen
from synth import tree as ST


def _model(shape, seed, ctx):
    w = gen.model_weights(shape, seed, "random")
    om = OF.Model(shape, w)
    cache = OF.KVCache(shape, 1, ctx + 80)
    for l in range(shape.n_layers):
        k, v = gen.synthetic_kv(shape, seed, l, 1, ctx)
        cache.k[l][0, :, :ctx] = OF.stored_to_f64(k[0], shape.dtype)
        cache.v[l][0, :, :ctx] = OF.stored_to_f64(v[0], shape.dtype)
    return om, cache


@pytest.mark.parametrize("shape", [configs.TINY_F32, configs.TINY_BF16])
def test_chain_tree_is_the_causal_block(synth_built, shape):
    om, cache = _model(shape, 3, 40)
    toks = gen.randint(3, 5, 9, shape.vocab)
    c1, c2 = copy.deepcopy(cache), copy.deepcopy(cache)
    l1, s1 = OF.verify_block(om, c1, [40], toks, [0, 9])
    l2, s2 = OF.verify_block(om, c2, [40], toks, [0, 9], parents=np.arange(-1, 8))
    assert list(s1) == list(s2) == [0]
    assert np.array_equal(l1, l2)
    for l in range(shape.n_layers):
        assert np.array_equal(c1.k[l], c2.k[l]) and np.array_equal(c1.v[l], c2.v[l])


@pytest.mark.parametrize("shape,n,depth", [(configs.TINY_F32, 24, 6), (configs.TINY_BF16, 18, 4)])
def test_every_node_equals_its_path(synth_built, shape, n, depth):
    C = 37
    om, cache = _model(shape, 4, C)
    par, dep = ST.random_tree(4, n, depth)
    toks = gen.randint(4, 6, n, shape.vocab)
    tc = copy.deepcopy(cache)
    lt, st = OF.verify_block(om, tc, [C], toks, [0, n], parents=par)
    assert st[0] == 0
    scale = np.abs(lt).max()
    for r in range(n):
        path = OF.ancestors(list(par), r)
        assert len(path) == dep[r] + 1
        pc = copy.deepcopy(cache)
        lp, _ = OF.verify_block(om, pc, [C], toks[path], [0, len(path)])
        assert np.abs(lp[-1] - lt[r]).max() <= 1e-12 * scale, r
        for l in range(shape.n_layers):  # the node's K/V at its tree slot = the path's last entry
            assert np.abs(tc.k[l][0, :, C + r] - pc.k[l][0, :, C + dep[r]]).max() <= 1e-12
            assert np.abs(tc.v[l][0, :, C + r] - pc.v[l][0, :, C + dep[r]]).max() <= 1e-12


def _leaf_paths(par):
    n = len(par)
    kids = [[c for c in range(1, n) if par[c] == u] for u in range(n)]
    return [OF.ancestors(list(par), r) for r in range(n) if not kids[r]]


def test_tree_acceptance_against_every_path():
    rng = np.random.default_rng(11)
    V = 50
    for trial in range(300):
        n = int(rng.integers(1, 40))
        par, dep = ST.random_tree(100 + trial, n, int(rng.integers(1, 8)))
        logits = rng.normal(size=(n, V))
        if trial % 7 == 0:
            logits = rng.integers(-2, 3, size=(n, V)).astype(np.float64)  # exact ties: first index wins
        tokens = rng.integers(0, V, size=n)
        tokens[0] = 0
        for c in range(1, n):  # plant: a child often carries its parent's argmax
            if rng.random() < 0.5:
                tokens[c] = OA.argmax_first(logits[par[c]])
        res = OT.accept_tree_greedy(logits, [0, n], tokens, par, 64)
        assert res["status"][0] == 0
        best = None
        for p in _leaf_paths(par):
            ch = OA.accept_greedy(logits[p], [0, len(p)], tokens[p], out_width=64)
            a = int(ch["accept_len"][0])
            if best is None or a > best[0]:
                best = (a, ch["out_tokens"][0], p[:a + 1])
        a = int(res["accept_len"][0])
        assert a == best[0], trial
        # the chosen path is one the chain rule accepts in full, ending at the smallest node
        # index among the paths of that length
        p = list(res["path"][0, :a + 1])
        ends = [q[a] for q in _leaf_paths(par) if len(q) > a and
                int(OA.accept_greedy(logits[q], [0, len(q)], tokens[q], out_width=64)["accept_len"][0]) >= a]
        assert p[-1] == min(ends) and p == OF.ancestors(list(par), p[-1]), trial
        ch = OA.accept_greedy(logits[p], [0, a + 1], tokens[p], out_width=64)
        assert int(ch["accept_len"][0]) == a and np.array_equal(res["out_tokens"][0], ch["out_tokens"][0]), trial


def test_duplicate_siblings_keep_the_longer_branch():
    """Two children carry the root's argmax; only the second one's subtree goes on, so the
    path runs through it (longest accepted path, not the first matching child)."""
    par = np.array([-1, 0, 0, 1, 2], np.int32)
    tokens = np.array([0, 7, 7, 3, 4], np.int32)
    logits = np.zeros((5, 10))
    logits[0, 7] = 1.0   # root -> 7 (children 1 and 2 both carry it)
    logits[1, 5] = 1.0   # node 1 -> 5: its child 3 carries 3, rejected
    logits[2, 4] = 1.0   # node 2 -> 4: child 4 accepted
    logits[4, 9] = 1.0
    res = OT.accept_tree_greedy(logits, [0, 5], tokens, par, 8)
    assert list(res["path"][0, :3]) == [0, 2, 4] and res["accept_len"][0] == 2
    assert list(res["out_tokens"][0, :3]) == [7, 4, 9]
    logits[1, 3] = 2.0   # now both branches reach depth 2: the smaller final index (3) wins
    res = OT.accept_tree_greedy(logits, [0, 5], tokens, par, 8)
    assert list(res["path"][0, :3]) == [0, 1, 3]


@pytest.mark.parametrize("shape", [configs.TINY_F32, configs.TINY_BF16])
def test_commit_moves_the_path_to_the_chain_positions(synth_built, shape):
    C = 29
    om, cache = _model(shape, 8, C)
    par, _, _ = ST.ddtree_like(8, 20, 5, 3, shape.vocab)
    toks = gen.randint(8, 9, 20, shape.vocab)
    toks[0] = 5
    tc = copy.deepcopy(cache)
    lt, _ = OF.verify_block(om, tc, [C], toks, [0, 20], parents=par)
    # plant a three-step accepted path
    node = 0
    for _ in range(3):
        kids = [c for c in range(1, 20) if par[c] == node]
        if not kids:
            break
        toks_needed = OA.argmax_first(lt[node])
        toks[kids[-1]] = toks_needed
        node = kids[-1]
    tc = copy.deepcopy(cache)
    lt, _ = OF.verify_block(om, tc, [C], toks, [0, 20], parents=par)
    res = OT.accept_tree_greedy(lt, [0, 20], toks, par, 16)
    a = int(res["accept_len"][0])
    assert a >= 1
    new_len = OT.compact(tc, [C], res)
    assert int(new_len[0]) == C + a + 1
    path = list(res["path"][0, :a + 1])
    pc = copy.deepcopy(cache)
    OF.verify_block(om, pc, [C], toks[path], [0, a + 1])
    # equal up to the summation order of products over blocks of different row counts
    for l in range(shape.n_layers):
        assert np.abs(tc.k[l][0, :, :C + a + 1] - pc.k[l][0, :, :C + a + 1]).max() <= 1e-12
        assert np.abs(tc.v[l][0, :, :C + a + 1] - pc.v[l][0, :, :C + a + 1]).max() <= 1e-12
    # decoding on from the committed cache: the next token's logits are the chain's
    nxt = [int(res["out_tokens"][0, a])]
    l1, _ = OF.verify_block(om, tc, [C + a + 1], nxt, [0, 1])
    l2, _ = OF.verify_block(om, pc, [C + a + 1], nxt, [0, 1])
    assert np.abs(l1 - l2).max() <= 1e-12 * np.abs(l2).max()


def test_invalid_trees_are_refused(synth_built):
    shape = configs.TINY_F32
    om, cache = _model(shape, 2, 10)
    for par in ([0, 0, 1], [-1, 1, 0], [-1, 0, 3], [-1, -1, 0]):
        _, st = OF.verify_block(om, copy.deepcopy(cache), [10], [1, 2, 3], [0, 3], parents=par)
        assert st[0] == OF.LSV_ERR_INVALID_ARG, par
        res = OT.accept_tree_greedy(np.zeros((3, 5)), [0, 3], [1, 2, 3], par, 4)
        assert res["status"][0] == OF.LSV_ERR_INVALID_ARG
    # a path longer than the output width is refused too
    res = OT.accept_tree_greedy(np.eye(5, k=1), [0, 5], [0, 1, 2, 3, 4], [-1, 0, 1, 2, 3], 3)
    assert res["status"][0] == OF.LSV_ERR_INVALID_ARG
