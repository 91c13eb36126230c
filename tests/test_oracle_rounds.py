"""Pins of the round plumbing oracle (Sec. 3.1): hand-checked layouts, and the lossless
property -- an oracle-only multi-round loop (pack -> verify -> greedy accept -> commit ->
next root) emits exactly the plain greedy continuation, whatever the drafts and lengths."""
import copy

import numpy as np
import torch

from oracle import accept as OA
from oracle import forward as OF
from oracle import rounds as OR
from synth import configs, drafter, gen


def test_pack_block_by_hand():
    tok = [-1] * 9
    st = OR.pack_block([0, 3, 4, 4, 9], [7, 8, 9, 5], [[1, 2, 3], [4, 5, 6], [0, 0, 0], [9, 9, 9]], 3, 9, tok)
    # sequence 2 has no rows, sequence 3 asks for 5 rows with G = 3
    assert st == [OR.OK, OR.OK, OR.INVALID_ARG, OR.INVALID_ARG]
    assert tok == [7, 1, 2, 8, -1, -1, -1, -1, -1]
    tok = [-1] * 4
    assert OR.pack_block([0, 2, 5], [1, 2], [[5, 6], [7, 8]], 2, 4, tok) == [OR.OK, OR.INVALID_ARG]  # past the bound
    assert tok == [1, 5, -1, -1]


def test_next_roots_by_hand():
    out = [[4, 5, -1], [6, -1, -1], [1, 2, 3]]
    assert OR.next_roots([1, 0, 2], out, 3, None, [0, 0, 0]) == [5, 6, 3]
    assert OR.next_roots([1, 0, 3], out, 3, [0, -5, 0], [9, 9, 9]) == [5, 9, 9]  # failed, out of range


def test_oracle_loop_is_lossless():
    m, seed, G, N = configs.TINY_F32, 51, 6, 24
    w = gen.model_weights(m, seed)
    om = OF.Model(m, w)
    C = 30
    cap = 128
    oc = OF.KVCache(m, 1, cap)
    for l in range(m.n_layers):
        k, v = gen.synthetic_kv(m, seed, l, 1, C)
        oc.k[l][0, :, :C] = OF.stored_to_f64(k[0], "f32")
        oc.v[l][0, :, :C] = OF.stored_to_f64(v[0], "f32")
    root = int(gen.randint(seed, 7, 1, m.vocab)[0])
    cont = OF.greedy_continuation(om, copy.deepcopy(oc), C, root, N)
    stream = np.zeros((1, cap), np.int64)
    stream[0, C], stream[0, C + 1:C + 1 + N] = root, cont
    dr = drafter.PlantedDrafter(stream, drafter.confidences(seed, 1, cap), seed, m.vocab, G, device="cpu")
    rng = np.random.default_rng(1)
    seq, roots, got = C, [root], []
    while len(got) < N:
        g = int(rng.integers(0, G + 1))  # any length: the stream must not depend on it
        drafts = torch.zeros((1, G), dtype=torch.int32)
        conf = torch.zeros((1, G), dtype=torch.float32)
        dr(torch.tensor([seq], dtype=torch.int32), drafts, conf)
        off = [0, g + 1]
        toks = [0] * (g + 1)
        assert OR.pack_block(off, roots, drafts.numpy(), G, g + 1, toks) == [OR.OK]
        logits, st = OF.verify_block(om, oc, [seq], toks, off)
        res = OA.accept_greedy(logits, off, toks, out_width=G + 1)
        a = int(res["accept_len"][0])
        got += [int(t) for t in res["out_tokens"][0][:a + 1]]
        seq += a + 1
        roots = OR.next_roots(res["accept_len"], res["out_tokens"], G + 1, res["status"], roots)
    assert got[:N] == cont
