"""Paged KV cache (lsv_verify_paged, lsv_commit_tree_paged): a pool of 64-position pages shared by
the batch, each sequence's blocks mapped through a scattered page table.

* Verify over the paged cache gives logits and appended K/V bit-identical to the slab cache
  (the same arithmetic; only the addresses differ), and within the bf16 / fp32 bars of the
  oracle -- for chain blocks and for tree blocks, over the fp32 model and two bf16 shapes;
* a tree round commits its accepted path inside the pages (lsv_commit_tree_paged) exactly as
  in a slab cache;
* multi-round decoding with the joint batched length rule (lsv_select_joint) on the paged cache
  emits the same tokens as on the slab cache, and the plain greedy stream."""
import numpy as np
import pytest
import torch

from oracle import forward as OF
from paper_2608_08721_amd import decode, lsv, runtime
from synth import configs, drafter, gen
from synth import tree as ST
from tests.lsv_testing import GpuModel, greedy_decisions, i32, note, row_rel_err

pytestmark = pytest.mark.gpu


def _scattered_table(B, max_pages, seed):
    """Every sequence gets max_pages pages of a shared pool, in a random order (plus unused ones)."""
    rng = np.random.default_rng(seed)
    n_pages = B * max_pages + 3
    perm = rng.permutation(n_pages)[:B * max_pages]
    return perm.reshape(B, max_pages).astype(np.int32), n_pages


def _both(shape, seed, contexts, rows, parents=None, tol=None):
    B = len(contexts)
    w = gen.model_weights(shape, seed, "random")
    cap = runtime.kv_capacity(max(contexts) + max(rows) + 8)
    gm = GpuModel(shape, w, B, cap, max_rows=max(64, int(sum(rows))))
    table, n_pages = _scattered_table(B, cap // lsv.LSV_KV_PAGE, seed)
    pk = runtime.PagedKVCache(gm.cfg, n_pages, table)
    om = OF.Model(shape, w)
    oc = OF.KVCache(shape, B, cap)
    for l in range(shape.n_layers):
        for b in range(B):
            k, v = gen.synthetic_kv(shape, seed + 31 * b, l, 1, contexts[b])
            kd, vd = runtime.to_device(k[0]), runtime.to_device(v[0])
            gm.kv.write(l, b, 0, kd, vd)
            pk.write(l, b, 0, kd, vd)
            oc.k[l][b, :, :contexts[b]] = OF.stored_to_f64(k[0], shape.dtype)
            oc.v[l][b, :, :contexts[b]] = OF.stored_to_f64(v[0], shape.dtype)
    off = runtime.row_offsets_of(rows)
    toks = gen.randint(seed, 900, int(off[-1]), shape.vocab)
    if parents is None:
        g_slab, st = gm.verify(contexts, toks, off)
    else:
        g_slab, st = gm.verify_tree(contexts, toks, off, parents)
    assert np.all(st == 0)
    M = int(off[-1])
    logits = torch.full((gm.max_rows, shape.vocab), float("nan"), device="cuda")
    status = torch.full((B,), 99, dtype=torch.int32, device="cuda")
    lsv.lsv_verify_paged(gm.cfg, gm.dm.buf, pk.buf, n_pages, pk.table, pk.max_pages, B, i32(contexts), i32(toks),
                         i32(off), i32(parents) if parents is not None else None, gm.max_rows, cap, logits, status,
                         gm.ws.buf, gm.ws.nbytes)
    torch.cuda.synchronize()
    g_paged = logits[:M].double().cpu().numpy()
    assert np.all(status.cpu().numpy() == 0)
    assert np.array_equal(g_paged, g_slab)
    for l in range(shape.n_layers):
        for b in range(B):
            ks, vs = gm.kv.read(l, b, 0, contexts[b] + rows[b])
            kp, vp = pk.read(l, b, 0, contexts[b] + rows[b])
            assert torch.equal(ks, kp) and torch.equal(vs, vp), (l, b)
    o, _ = OF.verify_block(om, oc, contexts, toks, off, parents=parents)
    err = row_rel_err(g_paged, o)
    bar = tol if tol is not None else (1e-5 if shape.dtype == "f32" else 2e-2)
    note(f"  {shape.name} paged ({n_pages} pages, table {table.shape}): bit-identical to the slab cache; "
         f"max row rel err {err.max():.2e} vs the oracle")
    assert err.max() <= bar
    if shape.dtype == "bf16":
        greedy_decisions(g_paged, o, 0.5)
    return gm, pk, toks, off, g_paged


def test_paged_chain_blocks():
    _both(configs.TINY_F32, 61, [100, 7, 150], [17, 5, 9])
    _both(configs.TINY_BF16, 62, [200, 77, 1, 130], [17, 5, 1, 33])
    _both(configs.SMALL_BF16, 63, [300, 129], [17, 9])


def test_paged_tree_blocks_and_commit():
    shape = configs.SMALL_BF16
    parents, tokens_unused, _ = ST.ddtree_like(64, 40, 6, 4, shape.vocab)
    p2, _ = ST.random_tree(65, 24, 8)
    par = np.concatenate([parents, p2]).astype(np.int32)
    gm, pk, toks, off, g = _both(shape, 64, [250, 61], [40, 24], parents=par)
    # acceptance on the GPU's logits, then the commit in both caches: bit-identical contents
    B, V, width = 2, shape.vocab, 12
    ws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, int(off[-1]), V))
    acc = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, width), dtype=torch.int32, device="cuda")
    path = torch.zeros((B, width), dtype=torch.int32, device="cuda")
    sl, st = i32([250, 61]), i32([0, 0])
    lg = torch.tensor(g.astype(np.float32), device="cuda")
    # plant: make the first child of the root carry the root's argmax
    kids = [c for c in range(1, 40) if par[c] == 0]
    toks = toks.copy()
    toks[kids[0]] = int(np.argmax(g[0]))
    lsv.lsv_accept_tree(B, V, lg, i32(off), i32(par), i32(toks), int(off[-1]), width, acc, out, path, sl, st, ws.buf,
                        ws.nbytes)
    lsv.lsv_commit_tree(gm.cfg, gm.kv.buf, gm.capacity, B, sl, acc, path, width, st)
    lsv.lsv_commit_tree_paged(gm.cfg, pk.buf, pk.n_pages, pk.table, pk.max_pages, B, sl, acc, path, width, st)
    torch.cuda.synchronize()
    assert int(acc[0]) >= 1
    for l in range(shape.n_layers):
        for b in range(B):
            n = int(sl[b])
            ks, vs = gm.kv.read(l, b, 0, n)
            kp, vp = pk.read(l, b, 0, n)
            assert torch.equal(ks, kp) and torch.equal(vs, vp)
    note(f"  tree commit in pages: accepted {acc.cpu().tolist()}, caches identical")


def test_joint_selection_rounds_on_paged_cache():
    """Serving-style decoding: the joint batched rule allocates each round's lengths over the
    batch; the paged cache gives the same emitted tokens as the slab cache and as plain decoding."""
    m, G, seed, n = configs.SMALL_BF16, 12, 66, 40
    contexts = [130, 70, 200]
    B = len(contexts)
    w = gen.model_weights(m, seed, "random")
    cfg = runtime.model_config(m)
    dm = runtime.DeviceModel.from_weights(cfg, w)
    cap = runtime.kv_capacity(max(contexts) + 2 * n * (G + 1) + G + 2)
    table, n_pages = _scattered_table(B, cap // lsv.LSV_KV_PAGE, seed)

    def caches():
        kv = runtime.KVCache(cfg, B, cap)
        pk = runtime.PagedKVCache(cfg, n_pages, table)
        for b, C in enumerate(contexts):
            for l in range(m.n_layers):
                k, v = gen.synthetic_kv(m, seed + 31 * b, l, 1, C)
                kd, vd = runtime.to_device(k[0]), runtime.to_device(v[0])
                kv.write(l, b, 0, kd, vd)
                pk.write(l, b, 0, kd, vd)
        return kv, pk
    roots = [int(x) for x in gen.randint(seed, 7, B, m.vocab)]

    def run(kv, policy, dr, cost=None, gamma0=None):
        loop = decode.DecodeLoop(cfg, dm, kv, cap, B, G, policy, dr, cost=cost, gamma0=gamma0)
        loop.reset(contexts, roots)
        loop.round()
        got = [list(e) for e in loop.emitted()]
        loop.capture()
        while min(len(x) for x in got) < n:
            loop.replay()
            for b, e in enumerate(loop.emitted()):
                got[b] += e
        assert bool((loop.status == 0).all())
        return [x[:n] for x in got]

    kv, pk = caches()
    plain = run(kv, "static", None, gamma0=0)
    stream = np.zeros((B, cap), np.int64)
    for b, C in enumerate(contexts):
        stream[b, C] = roots[b]
        stream[b, C + 1:C + 1 + n] = plain[b]
    dr = drafter.PlantedDrafter(stream, drafter.confidences(seed, B, cap), seed, m.vocab, G)
    cost_total = np.array([1.0 + 0.01 * r for r in range(B * G + 1)])
    kv, pk = caches()
    joint_slab = run(kv, "joint", dr, cost_total)
    joint_paged = run(pk, "joint", dr, cost_total)
    assert joint_paged == joint_slab == plain
    note(f"  joint rule on {n_pages} scattered pages: {n} tokens per sequence, identical to the slab cache and plain "
         f"decoding")
