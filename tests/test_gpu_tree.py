"""Tree verification on the GPU (lsv_verify_tree, lsv_accept_tree, lsv_commit_tree) against the
oracle (oracle/forward.py with parents, oracle/tree.py):

* fp32 tiny model: tree logits within 1e-5 of each row's largest logit and the K/V each node
  appends at its tree slot, for a drafter-like tree of 64 nodes and a random tree;
* bf16 (head_dim 128, four query heads per kv head): node budgets of 64 (two sequences) and
  512 (one sequence, 128 query tiles), logits within 2e-2 and greedy decisions per row;
* acceptance on the GPU's own logits, bit for bit against the oracle's rule on the same logits,
  with planted paths (accepted length, emitted tokens, path, committed length, status);
* the commit: every accepted node's K row and V column land at position C + depth, bit for bit
  the values the verify step stored at its tree slot; on the fp32 model the next decoding step
  from the committed cache matches the oracle's;
* invalid parent arrays give LSV_ERR_INVALID_ARG."""
import copy

import numpy as np
import pytest
import torch

from oracle import accept as OA
from oracle import forward as OF
from oracle import tree as OT
from paper_2608_08721_amd import lsv, runtime
from synth import configs, gen
from synth import tree as ST
from tests.lsv_testing import GpuModel, greedy_decisions, i32, note, row_rel_err

pytestmark = pytest.mark.gpu


def _setup(shape, seed, contexts, max_rows, cap_extra=16):
    w = gen.model_weights(shape, seed, "random")
    B = len(contexts)
    cap = runtime.kv_capacity(max(contexts) + max_rows + cap_extra)
    gm = GpuModel(shape, w, B, cap, max_rows=max(64, max_rows))
    om = OF.Model(shape, w)
    oc = OF.KVCache(shape, B, cap)
    for l in range(shape.n_layers):
        for b in range(B):
            k, v = gen.synthetic_kv(shape, seed + 31 * b, l, 1, contexts[b])
            gm.kv.write(l, b, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
            oc.k[l][b, :, :contexts[b]] = OF.stored_to_f64(k[0], shape.dtype)
            oc.v[l][b, :, :contexts[b]] = OF.stored_to_f64(v[0], shape.dtype)
    return gm, om, oc


def _plant(om, oc, contexts, toks, off, parents, levels):
    """Set, level by level, one child of each planted node to the oracle's argmax of its parent's
    row, so that acceptance walks down some branches."""
    toks = toks.copy()
    B = len(contexts)
    for _ in range(levels):
        lg, _ = OF.verify_block(om, copy.deepcopy(oc), contexts, toks, off, parents=parents)
        for b in range(B):
            r0, n = off[b], off[b + 1] - off[b]
            par = parents[r0:r0 + n]
            dep = OF.tree_depths(list(par))
            for u in range(n):
                kids = [c for c in range(1, n) if par[c] == u]
                if kids and dep[u] < levels:
                    toks[r0 + kids[len(kids) // 2]] = OA.argmax_first(lg[r0 + u])
    return toks


def _trees(specs, seed, vocab):
    """specs: list of ("dd", n, depth, branch) or ("rand", n, depth); returns parents, tokens, off."""
    par, tok = [], []
    for i, sp in enumerate(specs):
        if sp[0] == "dd":
            p, t, _ = ST.ddtree_like(seed + i, sp[1], sp[2], sp[3], vocab)
        else:
            p, _ = ST.random_tree(seed + i, sp[1], sp[2])
            t = gen.randint(seed + i, 77, sp[1], vocab)
        t = t.copy()
        t[0] = int(gen.randint(seed + i, 78, 1, vocab)[0])  # the root: the pending token
        par.append(p)
        tok.append(t)
    off = runtime.row_offsets_of([len(p) for p in par])
    return np.concatenate(par).astype(np.int32), np.concatenate(tok).astype(np.int32), off


def _accept_both(g_logits, off, toks, parents, width, seq_len):
    B, V = len(off) - 1, g_logits.shape[1]
    M = int(off[-1])
    lg = torch.tensor(g_logits.astype(np.float32), device="cuda")
    ws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, M, V))
    acc = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((B, width), -9, dtype=torch.int32, device="cuda")
    path = torch.full((B, width), -9, dtype=torch.int32, device="cuda")
    sl = i32(seq_len)
    st = i32([0] * B)
    lsv.lsv_accept_tree(B, V, lg, i32(off), i32(parents), i32(toks), M, width, acc, out, path, sl, st, ws.buf,
                        ws.nbytes)
    torch.cuda.synchronize()
    want = OT.accept_tree_greedy(g_logits.astype(np.float32).astype(np.float64), off, toks, parents, width)
    got = {"accept_len": acc.cpu().numpy(), "out_tokens": out.cpu().numpy(), "path": path.cpu().numpy(),
           "status": st.cpu().numpy()}
    for k in ("accept_len", "out_tokens", "path", "status"):
        assert np.array_equal(got[k], want[k]), (k, got[k], want[k])
    committed = np.asarray(seq_len) + np.where(want["status"] == 0, want["accept_len"] + 1, 0)
    assert np.array_equal(sl.cpu().numpy(), committed)
    return got, sl, st


def test_tree_fp32_logits_and_kv():
    shape = configs.TINY_F32
    contexts = [40, 75]
    parents, toks, off = _trees([("dd", 64, 6, 4), ("rand", 37, 9)], 5, shape.vocab)
    gm, om, oc = _setup(shape, 5, contexts, int(off[-1]))
    g, st = gm.verify_tree(contexts, toks, off, parents)
    assert list(st) == [0, 0]
    o, ost = OF.verify_block(om, oc, contexts, toks, off, parents=parents)
    err = row_rel_err(g, o)
    note(f"  fp32 trees of {list(np.diff(off))} nodes: max row rel err {err.max():.2e}")
    assert err.max() <= 1e-5
    for b in range(2):
        n = off[b + 1] - off[b]
        for l in range(shape.n_layers):
            gk, gv = (t.float().cpu().numpy() for t in gm.kv.read(l, b, contexts[b], n))
            ok_, ov_ = oc.k[l][b, :, contexts[b]:contexts[b] + n], oc.v[l][b, :, contexts[b]:contexts[b] + n]
            assert np.abs(gk - ok_).max() <= 1e-5 * np.abs(ok_).max()
            assert np.abs(gv - ov_).max() <= 1e-5 * np.abs(ov_).max()


@pytest.mark.parametrize("budget", [64, 512])
def test_tree_bf16_node_budgets(budget):
    shape = configs.SMALL_BF16
    specs = [("dd", 64, 8, 4), ("dd", 64, 6, 6)] if budget == 64 else [("dd", 512, 16, 8)]
    contexts = [300, 129][:len(specs)]
    parents, toks, off = _trees(specs, 40 + budget, shape.vocab)
    gm, om, oc = _setup(shape, 40 + budget, contexts, int(off[-1]))
    g, st = gm.verify_tree(contexts, toks, off, parents)
    assert np.all(st == 0)
    o, _ = OF.verify_block(om, oc, contexts, toks, off, parents=parents)
    err = row_rel_err(g, o)
    note(f"  bf16 trees of {list(np.diff(off))} nodes (budget {budget}): max row rel err {err.max():.2e}")
    assert err.max() <= 2e-2
    greedy_decisions(g, o, 0.5)


def test_tree_acceptance_and_commit_fp32():
    """Planted trees on the fp32 model: GPU acceptance on its own logits equals the oracle's rule
    bit for bit; the commit moves the accepted nodes' K/V; the next decoding step from the
    committed cache matches the oracle's, decoded from its own committed cache."""
    shape = configs.TINY_F32
    contexts = [40, 75]
    parents, toks, off = _trees([("dd", 48, 6, 4), ("rand", 30, 7)], 9, shape.vocab)
    gm, om, oc = _setup(shape, 9, contexts, int(off[-1]))
    toks = _plant(om, oc, contexts, toks, off, parents, 4)
    g, st = gm.verify_tree(contexts, toks, off, parents)
    assert list(st) == [0, 0]
    width = 17
    before = [[tuple(t.float().cpu().numpy() for t in gm.kv.read(l, b, 0, gm.capacity)) for l in range(shape.n_layers)]
              for b in range(2)]
    got, sl, stt = _accept_both(g, off, toks, parents, width, contexts)
    a = list(got["accept_len"])
    note(f"  accepted {a} drafts along paths {[list(got['path'][b, :a[b] + 1]) for b in range(2)]}")
    assert max(a) >= 2
    lsv.lsv_commit_tree(gm.cfg, gm.kv.buf, gm.capacity, 2, sl, i32(a), i32(got["path"]), width, stt)
    torch.cuda.synchronize()
    for b in range(2):
        C = contexts[b]
        for l in range(shape.n_layers):
            k1, v1 = (t.float().cpu().numpy() for t in gm.kv.read(l, b, 0, gm.capacity))
            k0, v0 = before[b][l]
            for k in range(1, a[b] + 1):
                src = C + int(got["path"][b, k])
                assert np.array_equal(k1[:, C + k], k0[:, src]) and np.array_equal(v1[:, C + k], v0[:, src])
            assert np.array_equal(k1[:, :C + 1], k0[:, :C + 1])
    # the oracle's own round: verify, accept on its logits, commit; then one plain step each
    oc2 = copy.deepcopy(oc)
    o, _ = OF.verify_block(om, oc2, contexts, toks, off, parents=parents)
    ores = OT.accept_tree_greedy(o, off, toks, parents, width)
    assert np.array_equal(ores["accept_len"], got["accept_len"])  # fp32: decisions far from ties
    new_len = OT.compact(oc2, contexts, ores)
    nxt = [int(got["out_tokens"][b, a[b]]) for b in range(2)]
    g2, st2 = gm.verify(list(new_len), nxt, [0, 1, 2])
    o2, _ = OF.verify_block(om, oc2, list(new_len), nxt, [0, 1, 2])
    assert list(st2) == [0, 0]
    assert row_rel_err(g2, o2).max() <= 1e-5


def test_tree_acceptance_bf16_parity():
    shape = configs.SMALL_BF16
    contexts = [200, 90, 150]
    parents, toks, off = _trees([("dd", 64, 8, 4), ("dd", 40, 5, 5), ("rand", 50, 10)], 21, shape.vocab)
    gm, om, oc = _setup(shape, 21, contexts, int(off[-1]))
    toks = _plant(om, oc, contexts, toks, off, parents, 5)
    g, st = gm.verify_tree(contexts, toks, off, parents)
    assert np.all(st == 0)
    got, _, _ = _accept_both(g, off, toks, parents, 16, contexts)
    note(f"  bf16 trees: accepted {list(got['accept_len'])}")


def test_invalid_trees():
    shape = configs.TINY_F32
    gm, _, _ = _setup(shape, 3, [20, 20], 8)
    toks = np.arange(8, dtype=np.int32)
    off = [0, 4, 8]
    for bad in ([-1, 0, 1, 2, 0, -1, 0, 1], [-1, 0, 3, 1, -1, 0, 0, 0], [-1, 0, 0, 1, -1, 2, 0, 1]):
        _, st = gm.verify_tree([20, 20], toks, off, bad)
        assert st[0] == (0 if bad[0] == -1 and all(0 <= bad[i] < i for i in range(1, 4)) else lsv.LSV_ERR_INVALID_ARG)
        assert st[1] == (0 if bad[4] == -1 and all(0 <= bad[4 + i] < i for i in range(1, 4)) else lsv.LSV_ERR_INVALID_ARG)
