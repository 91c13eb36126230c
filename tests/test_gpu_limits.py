"""The C-ABI's maximum sizes on the GPU, against the oracle:

* lsv_verify_block with LSV_MAX_ROWS = 512 block rows: 64 sequences (LSV_MAX_BATCH) of 8 rows
  over ragged contexts, one sequence of 512 rows (128 query tiles of a 4-head group: sixteen
  passes of the eight-wave attention split kernel), and the fp32 model at 512 rows (bar 1e-5);
  bounds of 512 rows take the 64-row-chunk GEMMs (eight chunks);
* lsv_accept, greedy and sampling, with 512 rows as 64 sequences of 8 and as 8 sequences of
  LSV_MAX_SEQ_ROWS = 64 (the widest block one wave decides).

(The selector's limits, 64 sequences and G = 64, are in test_gpu_select.py.)"""
import numpy as np
import pytest

from oracle import accept as OA
from oracle import forward as OF
from paper_2608_08721_amd import lsv, runtime
from synth import configs, gen
from tests.lsv_testing import GpuModel, note, row_rel_err
from tests.test_gpu_accept import draws_from, gpu_accept, unsettled
from tests.test_gpu_forward import _bf16_case

pytestmark = pytest.mark.gpu


def test_verify_64_sequences_of_8_rows():
    rng = np.random.default_rng(31)
    contexts = [int(c) for c in rng.integers(1, 200, size=lsv.LSV_MAX_BATCH)]
    _bf16_case(configs.TINY_BF16, 31, contexts, [8] * lsv.LSV_MAX_BATCH, bound=lsv.LSV_MAX_ROWS)


def test_verify_one_sequence_of_512_rows():
    _bf16_case(configs.SMALL_BF16, 32, [90], [lsv.LSV_MAX_ROWS], bound=lsv.LSV_MAX_ROWS)


def test_verify_fp32_512_rows():
    m, seed = configs.TINY_F32, 33
    w = gen.model_weights(m, seed)
    C, rows = 40, lsv.LSV_MAX_ROWS
    cap = runtime.kv_capacity(C + rows + 8)
    gm = GpuModel(m, w, 1, cap, max_rows=rows)
    om = OF.Model(m, w)
    oc = OF.KVCache(m, 1, cap)
    for l in range(m.n_layers):
        k, v = gen.synthetic_kv(m, seed, l, 1, C)
        gm.kv.write(l, 0, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
        oc.k[l][0, :, :C] = OF.stored_to_f64(k[0], "f32")
        oc.v[l][0, :, :C] = OF.stored_to_f64(v[0], "f32")
    toks = gen.randint(seed, 900, rows, m.vocab)
    off = [0, rows]
    g_logits, st = gm.verify([C], toks, off)
    o_logits, _ = OF.verify_block(om, oc, [C], toks, off)
    assert st[0] == 0
    err = row_rel_err(g_logits, o_logits)
    note(f"  tiny f32, {rows} rows: max row rel err {err.max():.2e}")
    assert err.max() <= 1e-5


@pytest.mark.parametrize("B,rows_per_seq", [(lsv.LSV_MAX_BATCH, 8), (8, lsv.LSV_MAX_SEQ_ROWS)])
def test_accept_at_the_limits(B, rows_per_seq):
    V = 4096
    rows = np.full(B, rows_per_seq)
    off = runtime.row_offsets_of(rows)
    M = int(off[-1])
    assert M == lsv.LSV_MAX_ROWS
    logits = gen.synthetic_logits(40 + B, M, V, std=2.0)
    # greedy: plant a matching prefix of a different length in each sequence
    tokens = gen.randint(41 + B, 5, M, V)
    rng = np.random.default_rng(B)
    for b in range(B):
        for v in range(1, int(rng.integers(0, rows_per_seq)) + 1):
            tokens[off[b] + v] = int(np.argmax(logits[off[b] + v - 1]))
    seq = rng.integers(0, 1000, size=B).astype(np.int32)
    acc, out, st, sl = gpu_accept(lsv.LSV_ACC_GREEDY, logits, off, tokens, rows_per_seq, seq_len=seq)
    want = OA.accept_greedy(logits, off, tokens, out_width=rows_per_seq)
    assert np.array_equal(st, want["status"]) and np.array_equal(acc, want["accept_len"])
    assert np.array_equal(out, want["out_tokens"]) and np.array_equal(sl, OA.commit(seq, want))
    # sampling at T = 1 with drafts drawn from their own distributions
    q = gen.draft_probs(42 + B, M - B, V)
    for b in range(B):
        tokens[off[b] + 1:off[b + 1]] = draws_from(q[off[b] - b:off[b + 1] - b - 1], rng.random(rows_per_seq - 1))
    acc, out, st, _ = gpu_accept(lsv.LSV_ACC_SAMPLE, logits, off, tokens, rows_per_seq, q, 1.0, 777, 3)
    want = OA.accept_sample(logits, off, tokens, q, 1.0, 777, 3, out_width=rows_per_seq)
    assert np.array_equal(st, want["status"])
    settled = 0
    for b in range(B):
        if unsettled(want["diag"][b]):
            continue
        settled += 1
        assert acc[b] == want["accept_len"][b], b
        assert np.array_equal(out[b], want["out_tokens"][b]), b
    note(f"  {B} x {rows_per_seq} rows: greedy bit-exact, sampling {settled}/{B} bit-exact (rest unsettled)")
    assert settled >= B - max(1, B // 20)
