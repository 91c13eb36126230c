"""A row's verify result does not depend on the block it is verified in.

The same 17 rows are verified as one block, then again at their own positions as blocks of
1 (under a one-row bound, which takes the smaller kernel variants), of 5 and of 11 rows; the
logits of every row must be bit-identical.  Every GEMM output accumulates its k-steps in the
same order whatever the row count, and every attention tile walks the context's chunks in the
same order with the same exp2 whether or not its chunk is masked.  This is what makes
multi-round greedy decoding emit exactly the plain greedy stream for every speculative
length (see test_gpu_decode.py)."""
import dataclasses

import numpy as np
import pytest

from paper_2608_08721_amd import runtime
from synth import configs, gen
from tests.lsv_testing import GpuModel, note

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [configs.SMALL_BF16, configs.TINY_BF16])
def test_row_logits_do_not_depend_on_block_size(shape):
    seed, C, R = 61, 150, 17
    w = gen.model_weights(shape, seed)
    cap = runtime.kv_capacity(C + R + 8)
    gm = GpuModel(shape, w, 1, cap, max_rows=R)
    for l in range(shape.n_layers):
        k, v = gen.synthetic_kv(shape, seed, l, 1, C)
        gm.kv.write(l, 0, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
    toks = gen.randint(seed, 900, R, shape.vocab)
    whole, st = gm.verify([C], toks, [0, R])
    assert st[0] == 0 and np.isfinite(whole).all()
    for sizes, bound in (([1] * R, 1), ([5, 5, 5, 2], R), ([11, 6], R)):
        pos = 0
        for n in sizes:
            lg, st = gm.verify([C + pos], toks[pos:pos + n], [0, n], max_rows=bound)
            assert st[0] == 0
            assert np.array_equal(lg, whole[pos:pos + n]), (shape.name, sizes, pos)
            pos += n
    note(f"  {shape.name}: 17 rows bit-identical as one block and as blocks of 1, 5 and 11 rows")


def test_row_logits_do_not_depend_on_block_size_wide_model():
    """Llama-3-70B width, one layer: its O and down products stream two fragment rows per wave
    for one activation tile and its QKV, O and down for two or more (each wave's sums are those
    of one row per wave), so the same 20 rows as one block, as blocks of 9 and 11 under a batched
    bound and as blocks of 5 under a 16-row bound must give bit-identical logits."""
    shape = configs.LLAMA3_70B.with_layers(1)
    seed, C, R = 62, 150, 20
    w = gen.model_weights(shape, seed)
    cap = runtime.kv_capacity(C + R + 8)
    gm = GpuModel(shape, w, 1, cap, max_rows=132)
    k, v = gen.synthetic_kv(shape, seed, 0, 1, C)
    gm.kv.write(0, 0, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
    toks = gen.randint(seed, 900, R, shape.vocab)
    whole, st = gm.verify([C], toks, [0, R], max_rows=132)
    assert st[0] == 0 and np.isfinite(whole).all()
    for sizes, bound in (([9, 11], 132), ([5, 5, 5, 5], 16)):
        pos = 0
        for n in sizes:
            lg, st = gm.verify([C + pos], toks[pos:pos + n], [0, n], max_rows=bound)
            assert st[0] == 0
            assert np.array_equal(lg, whole[pos:pos + n]), (sizes, bound, pos)
            pos += n
    note(f"  {shape.name}: 20 rows bit-identical as one block and as blocks of 9 + 11 and 5")


def test_packed_attention_grid_rows_do_not_depend_on_the_batch():
    """The packed split grid (eight ragged sequences of up to 8,190 positions over eight kv
    heads) takes a workgroup per split that holds keys, so which workgroup computes a split
    depends on the other sequences' lengths and rows; the split boundaries do not.  Sequence 3's
    17 rows verified in one batch, and again as blocks of 9 and 8 in batches whose other
    sequences carry other rows, must give bit-identical logits."""
    shape = dataclasses.replace(configs.SMALL_BF16, n_kv_heads=8, n_layers=1, name="small-bf16-kv8")
    seed = 63
    contexts = [8190, 1200, 4000, 300, 7000, 1, 2500, 6100]
    B = len(contexts)
    w = gen.model_weights(shape, seed)
    cap = runtime.kv_capacity(max(contexts) + 17 + 8)
    gm = GpuModel(shape, w, B, cap, max_rows=64)
    for b in range(B):
        k, v = gen.synthetic_kv(shape, seed + b, 0, 1, contexts[b])
        gm.kv.write(0, b, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
    rows = [3, 5, 1, 17, 2, 4, 9, 1]
    off = runtime.row_offsets_of(rows)
    toks = gen.randint(seed, 900, int(off[-1]), shape.vocab)
    whole, st = gm.verify(contexts, toks, off, max_rows=64)
    assert np.all(st == 0) and np.isfinite(whole).all()
    mine = toks[off[3]:off[4]]
    want = whole[off[3]:off[4]]
    pos = 0
    for n, others in ((9, 1), (8, 2)):
        r = [others] * B
        r[3] = n
        o = runtime.row_offsets_of(r)
        t = gen.randint(seed + n, 901, int(o[-1]), shape.vocab)
        t[o[3]:o[4]] = mine[pos:pos + n]
        ctx = list(contexts)
        ctx[3] += pos
        lg, st = gm.verify(ctx, t, o, max_rows=64)
        assert np.all(st == 0)
        assert np.array_equal(lg[o[3]:o[4]], want[pos:pos + n]), (n, pos)
        pos += n
    note("  packed grid: 17 rows of one sequence bit-identical across batches with other rows")
