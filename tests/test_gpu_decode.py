"""Multi-round decoding on the GPU (DecodeLoop: drafter -> length -> pack -> verify -> accept
-> next roots, one captured graph per round):

* the round plumbing kernels (lsv_pack_block, lsv_next_roots) against the oracle's plain
  definitions, bit for bit, including rows that are empty, too long or past the bound;
* the lossless property (Sec. 3.1): with greedy acceptance the emitted stream of every
  length policy -- static 0 (plain decoding), static 4, the marginal rule, Algorithm 1 and the
  G4-style rule -- equals the oracle's greedy continuation, on the fp32 tiny model (bar 1e-5)
  where every step's top-2 logit gap is far above that bar.  The drafter is the planted,
  calibrated stand-in of synth/drafter.py, fed the oracle's continuation."""
import copy

import numpy as np
import pytest
import torch

from oracle import forward as OF
from oracle import rounds as OR
from paper_2608_08721_amd import decode, lsv, runtime
from synth import configs, drafter, gen
from tests.lsv_testing import i32, note

pytestmark = pytest.mark.gpu


def test_pack_block_and_next_roots_parity():
    rng = np.random.default_rng(3)
    for trial in range(20):
        B = int(rng.integers(1, lsv.LSV_MAX_BATCH + 1))
        G = int(rng.integers(0, 20))
        rows = rng.integers(1, G + 2, size=B)
        bad = rng.random(B) < 0.15
        rows[bad] = np.where(rng.random(bad.sum()) < 0.5, 0, G + 2)  # empty or one too many
        off = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
        # the bound: the rows' end, a little short of it (the last rows are refused), or LSV_MAX_ROWS
        max_rows = int(min(max(1, off[-1] - (rng.integers(0, 3) if trial % 4 == 0 else 0)), lsv.LSV_MAX_ROWS))
        roots = rng.integers(0, 1000, size=B).astype(np.int32)
        drafts = rng.integers(0, 1000, size=(B, max(G, 1))).astype(np.int32)
        tok = torch.full((max_rows,), -5, dtype=torch.int32, device="cuda")
        st = torch.full((B,), 99, dtype=torch.int32, device="cuda")
        lsv.lsv_pack_block(B, G, i32(off), max_rows, i32(roots), i32(drafts), tok, st)
        want_tok = [-5] * max_rows
        want_st = OR.pack_block(off, roots, drafts, G, max_rows, want_tok)
        assert tok.cpu().tolist() == want_tok and st.cpu().tolist() == want_st
        # next roots from an accept-shaped record
        width = G + 1
        acc = rng.integers(-1, width + 1, size=B).astype(np.int32)
        out = rng.integers(0, 1000, size=(B, width)).astype(np.int32)
        ast = np.where(rng.random(B) < 0.2, lsv.LSV_ERR_NONFINITE, 0).astype(np.int32)
        r = i32(roots)
        lsv.lsv_next_roots(B, i32(acc), i32(out), width, i32(ast), r)
        assert r.cpu().tolist() == OR.next_roots(acc, out, width, ast, roots)
    torch.cuda.synchronize()


SEED = 51
N = 40  # greedy tokens per sequence that the test checks


def _setup(m, w, contexts, G):
    cfg = runtime.model_config(m)
    dm = runtime.DeviceModel.from_weights(cfg, w)
    # room for every round the test may run (up to 2N rounds of G + 1 rows past the contexts)
    cap = runtime.kv_capacity(max(contexts) + 2 * N * (G + 1) + G + 2)
    kv = runtime.KVCache(cfg, len(contexts), cap)
    om = OF.Model(m, w)
    conts, roots = [], []
    for b, C in enumerate(contexts):
        oc = OF.KVCache(m, 1, cap)
        for l in range(m.n_layers):
            k, v = gen.synthetic_kv(m, SEED + 31 * b, l, 1, C)
            kv.write(l, b, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
            oc.k[l][0, :, :C] = OF.stored_to_f64(k[0], "f32")
            oc.v[l][0, :, :C] = OF.stored_to_f64(v[0], "f32")
        root = int(gen.randint(SEED, 7 + b, 1, m.vocab)[0])
        cont = OF.greedy_continuation(om, copy.deepcopy(oc), C, root, N)
        # every step is decided by a clear margin (the fp32 path is within 1e-5 of the oracle)
        lg, _ = OF.verify_block(om, copy.deepcopy(oc), [C], [root] + cont[:-1], [0, N])
        top2 = np.sort(lg, axis=1)[:, -2:]
        assert np.all(top2[:, 1] - top2[:, 0] > 1e-3 * np.abs(lg).max()), "pick a seed with settled steps"
        assert list(np.argmax(lg, axis=1)) == cont
        conts.append(cont)
        roots.append(root)
    return cfg, dm, kv, cap, conts, roots


@pytest.mark.parametrize("policy,gamma0", [("static", 0), ("static", 4), ("marginal", None), ("alg1", None),
                                           ("g4", 3)])
def test_loop_is_lossless_fp32(policy, gamma0):
    m, G = configs.TINY_F32, 12
    contexts = [40, 75]
    B = len(contexts)
    w = gen.model_weights(m, SEED)
    cfg, dm, kv, cap, conts, roots = _setup(m, w, contexts, G)
    L = cap
    stream = np.zeros((B, L), np.int64)
    for b, C in enumerate(contexts):
        stream[b, C] = roots[b]
        stream[b, C + 1:C + 1 + N] = conts[b]
    q = drafter.confidences(SEED, B, L)
    dr = drafter.PlantedDrafter(stream, q, SEED, m.vocab, G)
    cost = np.array([0.0] + [1.0 + 0.05 * d for d in range(1, G + 1)])
    loop = decode.DecodeLoop(cfg, dm, kv, cap, B, G, policy, dr, cost=cost, block_n=4, gamma0=gamma0)
    loop.reset(contexts, roots)
    loop.round()  # one eager round, then the captured one replays from where it left off
    got = [list(e) for e in loop.emitted()]
    loop.capture()
    rounds = 1
    while min(len(g) for g in got) < N and rounds < 2 * N:
        loop.replay()
        for b, e in enumerate(loop.emitted()):
            got[b] += e
        rounds += 1
    torch.cuda.synchronize()
    assert bool((loop.status == 0).all())
    for b in range(B):
        assert got[b][:N] == conts[b], (b, got[b][:N], conts[b])
        assert int(loop.seq_len[b]) == contexts[b] + len(got[b])
    note(f"  {policy} (gamma0 {gamma0}): {N} tokens per sequence in {rounds} rounds, identical to greedy decoding")


def test_bf16_loop_streams_agree_for_every_length():
    """bf16, hd 128 (the eight-wave attention under a 17-row bound): plain decoding (static 0)
    gives the greedy stream; static 16 (17-row blocks), the marginal rule, the G4-style rule
    and the joint rule, fed drafts planted from that stream, must emit it token for token -- a row's
    logits do not depend on the block it is verified in."""
    m, G, seed, n = configs.SMALL_BF16, 16, 71, 48
    contexts = [130, 200]
    B = len(contexts)
    w = gen.model_weights(m, seed)
    cfg = runtime.model_config(m)
    dm = runtime.DeviceModel.from_weights(cfg, w)
    cap = runtime.kv_capacity(max(contexts) + 2 * n * (G + 1) + G + 2)
    kv = runtime.KVCache(cfg, B, cap)
    for b, C in enumerate(contexts):
        for l in range(m.n_layers):
            k, v = gen.synthetic_kv(m, seed + 31 * b, l, 1, C)
            kv.write(l, b, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
    roots = [int(x) for x in gen.randint(seed, 7, B, m.vocab)]

    def run(policy, gamma0, dr, cost=None):
        loop = decode.DecodeLoop(cfg, dm, kv, cap, B, G, policy, dr, cost=cost, gamma0=gamma0)
        loop.reset(contexts, roots)
        loop.round()
        got = [list(e) for e in loop.emitted()]
        loop.capture()
        while min(len(g) for g in got) < n:
            loop.replay()
            for b, e in enumerate(loop.emitted()):
                got[b] += e
        assert bool((loop.status == 0).all())
        return [g[:n] for g in got]

    plain = run("static", 0, None)
    stream = np.zeros((B, cap), np.int64)
    for b, C in enumerate(contexts):
        stream[b, C] = roots[b]
        stream[b, C + 1:C + 1 + n] = plain[b]
    dr = drafter.PlantedDrafter(stream, drafter.confidences(seed, B, cap), seed, m.vocab, G)
    cost = np.array([0.0] + [1.0 + 0.02 * d for d in range(1, G + 1)])
    cost_total = np.array([1.0 + 0.01 * r for r in range(B * G + 1)])  # by the batch's total drafts
    for policy, g0 in (("static", 16), ("marginal", None), ("g4", 8), ("joint", None)):
        assert run(policy, g0, dr, cost_total if policy == "joint" else cost) == plain, policy
    note(f"  small bf16: {n} tokens per sequence identical for static 0 / 16, marginal, G4-style and joint")


def test_loop_stops_a_sequence_at_max_ctx():
    """A block that would run past max_ctx is refused by the verify step (LSV_ERR_CAPACITY); the
    acceptance then skips that sequence -- no tokens, no commit, the status kept -- and the next
    roots keep its pending token, so the sequence stays where it was while the other one decodes
    on.  Everything emitted before is the oracle's greedy continuation."""
    m, G, gamma, max_ctx = configs.TINY_F32, 12, 4, 80
    contexts = [40, 75]
    B = len(contexts)
    w = gen.model_weights(m, SEED)
    cfg, dm, kv, cap, conts, roots = _setup(m, w, contexts, G)
    stream = np.zeros((B, cap), np.int64)
    for b, C in enumerate(contexts):
        stream[b, C] = roots[b]
        stream[b, C + 1:C + 1 + N] = conts[b]
    dr = drafter.PlantedDrafter(stream, drafter.confidences(SEED, B, cap), SEED, m.vocab, G)
    loop = decode.DecodeLoop(cfg, dm, kv, cap, B, G, "static", dr, gamma0=gamma, max_ctx=max_ctx)
    loop.reset(contexts, roots)
    got, frozen = [[] for _ in range(B)], [None] * B
    for r in range(40):
        loop.round()
        st, sl, em = loop.status.cpu().tolist(), loop.seq_len.cpu().tolist(), loop.emitted()
        for b in range(B):
            if st[b] == lsv.LSV_OK:
                assert frozen[b] is None, (r, b)
                got[b] += em[b]
                assert sl[b] == contexts[b] + len(got[b])
            else:
                assert st[b] == lsv.LSV_ERR_CAPACITY and em[b] == [-1], (r, b, st[b], em[b])
                frozen[b] = sl[b] if frozen[b] is None else frozen[b]
                assert sl[b] == frozen[b]
        if all(f is not None for f in frozen):
            break
    for b in range(B):
        assert frozen[b] is not None and max_ctx - (gamma + 1) < frozen[b] <= max_ctx, (b, frozen[b])
        assert got[b] == conts[b][:len(got[b])], b
    note(f"  sequences stopped at {frozen} of max_ctx {max_ctx} after emitting {[len(g) for g in got]} tokens")


def test_alg1_drafts_blocks_on_demand():
    """Algorithm 1's budget drives the drafter (blocks of n only when the budget goes
    negative): each round drafts exactly the blocks the oracle's rule uses over that round's
    confidences, verifies the oracle's length, and the stream stays the greedy one."""
    from oracle import selector as S
    m, G, n = configs.TINY_F32, 16, 4
    contexts = [40, 75]
    B = len(contexts)
    w = gen.model_weights(m, SEED)
    cfg, dm, kv, cap, conts, roots = _setup(m, w, contexts, G)
    L = cap
    stream = np.zeros((B, L), np.int64)
    for b, C in enumerate(contexts):
        stream[b, C] = roots[b]
        stream[b, C + 1:C + 1 + N] = conts[b]
    q = drafter.confidences(SEED + 1, B, L)
    dr = drafter.PlantedDrafter(stream, q, SEED, m.vocab, G, n=n)
    loop = decode.DecodeLoop(cfg, dm, kv, cap, B, G, "alg1", dr, block_n=n, alpha=2.2)
    assert loop.on_demand
    loop.reset(contexts, roots)
    got = [[] for _ in range(B)]
    rounds = blocks_total = 0
    while min(len(g) for g in got) < N and rounds < 2 * N:
        sl = loop.seq_len.cpu().numpy()
        want = [S.select_alg1([float(q[b, min(sl[b] + k, L - 1)]) for k in range(1, G + 1)], G, 2.2, n)
                for b in range(B)]
        before = dr.drafted.clone()
        loop.round()
        for b, e in enumerate(loop.emitted()):
            got[b] += e
        gam, blk = loop.gamma.cpu().tolist(), loop.blocks.cpu().tolist()
        assert [(gam[b], blk[b]) for b in range(B)] == want, (rounds, want, gam, blk)
        assert (dr.drafted - before).cpu().tolist() == [min(bl * n, G) for bl in blk]
        blocks_total += sum(blk)
        rounds += 1
    assert bool((loop.status == 0).all())
    for b in range(B):
        assert got[b][:N] == conts[b]
    note(f"  alg1 with blocks on demand: {rounds} rounds, {blocks_total} blocks of {n} drafted "
         f"(all up front: {rounds * B * (-(-G // n))}), stream identical to greedy decoding")


def test_sampling_round_emits_the_target_distribution():
    """Sec. 3.1's sampling setting, a whole round on the device: with proposals from an
    unrelated distribution, the first emitted token of a round follows the target's
    softmax(logits / T) at the root (chi-square over 64 sequences x 160 rounds); a run of
    rounds keeps every status OK and commits every emitted token."""
    from scipy import stats
    m, G, T = configs.TINY_F32, 4, 0.7
    B, C = 64, 50
    w = gen.model_weights(m, SEED)
    cfg = runtime.model_config(m)
    dm = runtime.DeviceModel.from_weights(cfg, w)
    cap = runtime.kv_capacity(C + 40 * (G + 1) + 8)
    kv = runtime.KVCache(cfg, B, cap)
    om = OF.Model(m, w)
    oc = OF.KVCache(m, 1, cap)
    for l in range(m.n_layers):
        k, v = gen.synthetic_kv(m, SEED, l, 1, C)
        kd, vd = runtime.to_device(k[0]), runtime.to_device(v[0])
        for b in range(B):
            kv.write(l, b, 0, kd, vd)
        oc.k[l][0, :, :C] = OF.stored_to_f64(k[0], "f32")
        oc.v[l][0, :, :C] = OF.stored_to_f64(v[0], "f32")
    root = int(gen.randint(SEED, 5, 1, m.vocab)[0])
    lg, _ = OF.verify_block(om, oc, [C], [root], [0, 1])
    z = lg[0] / T
    p0 = np.exp(z - z.max())
    p0 /= p0.sum()
    dr = drafter.SampledDrafter(SEED, m.vocab)
    loop = decode.DecodeLoop(cfg, dm, kv, cap, B, G, "static", dr, gamma0=G, accept="sample", temperature=T)
    with pytest.raises(RuntimeError):
        loop.capture()
    counts = np.zeros(m.vocab)
    trials = 160
    for t in range(trials):
        loop.reset([C] * B, [root] * B)
        loop.seed = 1000 + t
        loop.round()
        first = loop.out[:, 0].cpu().numpy()
        assert bool((loop.status == 0).all())
        np.add.at(counts, first, 1)
    n_s = B * trials
    exp_ = p0 * n_s
    big = exp_ >= 5
    obs = np.concatenate([counts[big], [counts[~big].sum()]])
    ex = np.concatenate([exp_[big], [exp_[~big].sum()]])
    keep = ex > 0
    chi = stats.chisquare(obs[keep], ex[keep])
    note(f"  sampling round at T {T}: first emitted token over {n_s} draws, {int(big.sum())} bins + rest, "
         f"chi-square p {chi.pvalue:.3f}")
    assert chi.pvalue > 1e-3
    # a run of rounds: statuses OK, every emitted token committed
    loop.reset([C] * B, [root] * B)
    total = np.zeros(B, np.int64)
    for r in range(20):
        loop.seed = 77
        loop.round()
        acc = loop.acc.cpu().numpy()
        assert bool((loop.status == 0).all()) and np.all((acc >= 0) & (acc <= G))
        total += acc + 1
    assert np.array_equal(loop.seq_len.cpu().numpy(), C + total)
