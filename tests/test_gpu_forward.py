"""GPU verify forward pass (lsv_verify_block) and the whole step vs the oracle.

* tiny fp32 decoder (2 layers, d 256, 4 x 64 heads, F 688, V 1024, context 128):
  prefill and verify logits within 1e-5 of the largest logit of each row, and the
  greedy accept results bit-exact (argmax margins dwarf that error);
* bf16 decoders (grouped-query attention, head_dim 64 and 128, ragged contexts over
  several 64-key chunks): logits within 2e-2; greedy decisions equal wherever the
  oracle's top-2 margin exceeds twice the row's measured logit error, and at least half
  of the rows decided (tests.lsv_testing.greedy_decisions);
* Llama-3-8B width (d 4096, 32/8 x 128 heads, F 14336, V 128256) with 2 of its 32
  layers, context 2048 from the seeded KV generator, 17 rows: the same bf16 bar.
Unless a test says otherwise the RMSNorm gains are random per column (0.5 + U(0, 1)), so
the attention, FFN and final norms' gains all reach the logits."""
import copy
import dataclasses

import numpy as np
import pytest
import torch

from oracle import accept as OA
from oracle import forward as OF
from paper_2608_08721_amd import lsv, runtime
from synth import configs, gen
from tests.lsv_testing import GpuModel, greedy_decisions, i32, note, row_rel_err, top2_margin

pytestmark = pytest.mark.gpu


def greedy_gpu(logits_t, off, tokens, width):
    B = len(off) - 1
    M, V = logits_t.shape
    ws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, M, V))
    acc = torch.zeros(B, dtype=torch.int32, device="cuda")
    out = torch.zeros((B, width), dtype=torch.int32, device="cuda")
    st = torch.zeros(B, dtype=torch.int32, device="cuda")
    lsv.lsv_accept(lsv.LSV_ACC_GREEDY, B, V, logits_t, i32(off), M, width, i32(tokens), None, 0.0, 0, 0, acc, out,
                   None, st, ws.buf, ws.nbytes)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), out.cpu().numpy(), st.cpu().numpy()


@pytest.mark.parametrize("gains", ["ones", "random"])
def test_tiny_f32_end_to_end(gains):
    wl = configs.WORKLOADS["tiny-f32-b1-c128"]
    m = wl.model
    w = gen.model_weights(m, wl.seed, gains)
    C = int(gen.contexts(wl)[0])
    prompt = gen.prefix_ids(wl.seed, 1, [C], m.vocab)[0]
    note(f"tiny f32, {gains} gains: prefill {C} tokens")
    om = OF.Model(m, w)
    ocache = OF.KVCache(m, 1, 256)
    o_last, o_len = OF.prefill(om, ocache, [prompt])
    gm = GpuModel(m, w, 1, 256)
    g_last, g_len = gm.prefill([prompt])
    assert row_rel_err(g_last, o_last).max() <= 1e-5
    root = int(np.argmax(o_last[0]))
    assert root == int(np.argmax(g_last[0]))
    # plant: first k drafts are the target's greedy continuation, the rest random ids
    for k in (0, 5, 16):
        cont = OF.greedy_continuation(om, copy.deepcopy(ocache), C, root, k) if k else []
        rand = list(gen.randint(wl.seed, 500 + k, wl.G - k, m.vocab))
        drafts = cont + rand
        toks = np.array([root] + drafts, np.int32)
        off = [0, wl.G + 1]
        oc = copy.deepcopy(ocache)
        o_logits, _ = OF.verify_block(om, oc, [C], toks, off)
        g_logits, st = gm.verify([C], toks, off)
        assert st[0] == 0
        err = row_rel_err(g_logits, o_logits)
        note(f"  k={k}: max row rel err {err.max():.2e}")
        assert err.max() <= 1e-5
        want = OA.accept_greedy(o_logits, off, toks)
        margins = [top2_margin(r) / np.abs(r).max() for r in o_logits]
        assert min(margins) > 1e-4   # every decision is far outside the error bound
        acc, out, st = greedy_gpu(gm.logits[:wl.G + 1], off, toks, wl.G + 1)
        assert acc[0] == want["accept_len"][0] and np.array_equal(out[0], want["out_tokens"][0])
        if k == 16:
            assert acc[0] == 16


def _bf16_case(shape, seed, contexts, rows, tol=2e-2, bound=None, gains="random", min_decided=0.5):
    """Verify through the C-ABI against the oracle. bound: the host row bound of the call
    (default: the workspace's, max(64, total rows))."""
    B = len(contexts)
    w = gen.model_weights(shape, seed, gains)
    cap = runtime.kv_capacity(max(contexts) + max(rows) + 8)
    gm = GpuModel(shape, w, B, cap, max_rows=max(64, int(sum(rows)), bound or 0))
    om = OF.Model(shape, w)
    oc = OF.KVCache(shape, B, cap)
    for l in range(shape.n_layers):
        for b in range(B):
            k, v = gen.synthetic_kv(shape, seed + 31 * b, l, 1, contexts[b])
            gm.kv.write(l, b, 0, runtime.to_device(k[0]), runtime.to_device(v[0]))
            oc.k[l][b, :, :contexts[b]] = OF.stored_to_f64(k[0], "bf16")
            oc.v[l][b, :, :contexts[b]] = OF.stored_to_f64(v[0], "bf16")
    off = runtime.row_offsets_of(rows)
    toks = gen.randint(seed, 900, int(off[-1]), shape.vocab)
    g_logits, st = gm.verify(contexts, toks, off, max_rows=bound)
    assert np.all(st == 0)
    o_logits, _ = OF.verify_block(om, oc, contexts, toks, off)
    err = row_rel_err(g_logits, o_logits)
    note(f"  {shape.name}: contexts {list(contexts)} rows {list(rows)}: max row rel err {err.max():.2e}")
    assert err.max() <= tol
    # the K/V the GPU appended match the oracle's block entries, and the cached context is untouched
    for b in range(B):
        for l in range(shape.n_layers):
            gk, gv = (t.float().cpu().numpy() for t in gm.kv.read(l, b, 0, contexts[b] + rows[b]))
            k0, v0 = gen.synthetic_kv(shape, seed + 31 * b, l, 1, contexts[b])
            assert np.array_equal(gk[:, :contexts[b]], OF.stored_to_f64(k0[0], "bf16"))
            assert np.array_equal(gv[:, :contexts[b]], OF.stored_to_f64(v0[0], "bf16"))
            if rows[b] == 0:
                continue
            for got, want in ((gk, oc.k[l]), (gv, oc.v[l])):
                new_g = got[:, contexts[b]:]
                new_o = want[b, :, contexts[b]:contexts[b] + rows[b]]
                assert np.abs(new_g - new_o).max() <= tol * max(np.abs(new_o).max(), 1e-6) * 4
    # greedy decisions agree wherever the oracle's margin clears the row's error
    greedy_decisions(g_logits, o_logits, min_decided)
    return gm, g_logits, o_logits, toks, off


# eight kv heads: with eight sequences, 64 (sequence, kv head) pairs share the split kernel's grid
SMALL_KV8 = dataclasses.replace(configs.SMALL_BF16, n_kv_heads=8, n_layers=1, name="small-bf16-kv8")


def test_bf16_packed_attention_grid_ragged_long_contexts():
    """Eight sequences of 1 to 8,190 cached positions over eight kv heads: one round of splits
    (four per pair) would walk 33 chunks each of the 129-chunk bound, so the split kernel runs
    on the packed grid -- 12 splits of 11 chunks, the splits that hold keys first.  Logits,
    appended K/V and greedy decisions against the oracle."""
    _bf16_case(SMALL_KV8, 17, [8190, 1200, 4000, 300, 7000, 1, 2500, 6100], [3, 5, 1, 17, 2, 4, 9, 1])


def test_bf16_gqa_hd64_ragged():
    _bf16_case(configs.TINY_BF16, 11, [200, 77, 1, 130], [17, 5, 1, 33])


def test_bf16_hd128_ragged():
    _bf16_case(configs.SMALL_BF16, 12, [129, 300], [17, 9])


def test_bf16_hd128_few_tiles_under_loose_bound():
    """9 rows of a 4-query-head group under a 17-row bound: the attention split kernel takes
    eight waves (chosen from the bound) but has three query tiles, so five waves idle while
    both four-wave groups keep loading chunks."""
    _bf16_case(configs.SMALL_BF16, 15, [300], [9], bound=17)


def test_bf16_hd128_eight_waves_with_one_or_two_tiles():
    """Under a 17-rows-per-sequence bound the split kernel runs eight waves; sequences of 1
    and 2 query tiles leave most waves idle (a 30-token context is a single chunk, so the
    second group's buffer stays unused)."""
    _bf16_case(configs.SMALL_BF16, 19, [300, 30, 129], [3, 7, 1], bound=51)


def test_bf16_hd128_four_waves_few_tiles():
    """Under an 8-rows-per-sequence bound the split kernel runs four waves, one query tile
    each; 1 and 2 tiles leave waves idle, over a multi-chunk and a single-chunk context."""
    _bf16_case(configs.SMALL_BF16, 20, [200, 30], [5, 2], bound=16)


def test_bf16_hd128_two_passes_of_eight_waves():
    """40 rows of a 4-query-head group: ten query tiles, two passes of the eight-wave
    attention split kernel over the context."""
    _bf16_case(configs.SMALL_BF16, 16, [200], [40], bound=64)


def test_bf16_hd128_three_passes_beside_a_one_tile_sequence():
    """Rows 70 + 2 under a 72-row bound: the first sequence's 18 query tiles take three passes
    of the eight-wave split kernel (8, 8, then 2 tiles), the second sequence's
    single tile one."""
    _bf16_case(configs.SMALL_BF16, 21, [260, 40], [70, 2], bound=72)


def test_bf16_hd64_wide_block_unsplit_qkv():
    """140 rows at head dim 64 (d 256): the batched GEMMs, whose QKV product is too narrow to
    split K (projection, then the separate rotary-embedding kernel), and 18 query tiles of a
    2-query-head group, three passes of the eight-wave attention split kernel."""
    _bf16_case(configs.TINY_BF16, 18, [100], [140], bound=140)


def test_bf16_single_row_and_empty_sequence():
    _bf16_case(configs.TINY_BF16, 13, [64, 63], [1, 0])


def test_llama8b_width_two_layers():
    shape = configs.LLAMA3_8B.with_layers(2)
    note("llama3-8b width, 2 layers: generating weights")
    _bf16_case(shape, 2, [2048], [17])


def test_bf16_unit_gains():
    """Gains of one (the workloads' setting): the folded gain is the weight itself."""
    _bf16_case(configs.SMALL_BF16, 12, [129, 300], [17, 9], gains="ones")


def test_wide_model_gateup_skinny_blocks():
    """Qwen2.5-32B and Llama-3-70B widths, one layer, blocks of 9 and 9 + 11 rows: their gate/up
    products (3072 or more fragment rows) take the eight-fragment-rows-per-wave configuration,
    with one and with two activation tiles."""
    _bf16_case(configs.QWEN25_32B.with_layers(1), 22, [1000, 333], [9, 11])
    _bf16_case(configs.LLAMA3_70B.with_layers(1), 23, [700], [9])


def test_wide_model_two_fragment_rows_per_wave():
    """Blocks of two to four activation tiles at Llama-3-70B width, one layer: QKV, O and down
    then stream two fragment rows per wave (640 and 512 fragment rows still leave a stream per
    compute unit) -- 22 rows under a 64-row bound (the 64-row kernel) and 50 rows under a
    batched bound (the fused kernel's 64-row body).  With one activation tile O and down still
    take two rows per wave (12 rows under a batched bound)."""
    _bf16_case(configs.LLAMA3_70B.with_layers(1), 24, [500, 300], [13, 9])
    _bf16_case(configs.LLAMA3_70B.with_layers(1), 25, [400], [50], bound=132)
    _bf16_case(configs.LLAMA3_70B.with_layers(1), 26, [300, 200], [5, 7], bound=132)


def test_workspace_reused_across_bounds():
    """One zeroed workspace serves calls with different row and context bounds: prefill with
    the 64-row bound, then verify blocks with the 17-, 64- and 5-row bounds and a smaller
    max_ctx, each against the oracle."""
    shape = configs.TINY_BF16
    w = gen.model_weights(shape, 14, "random")
    cap = 256
    gm = GpuModel(shape, w, 1, cap)
    om = OF.Model(shape, w)
    oc = OF.KVCache(shape, 1, cap)
    prompt = gen.prefix_ids(14, 1, [150], shape.vocab)[0]
    g_last, _ = gm.prefill([prompt])
    o_last, _ = OF.prefill(om, oc, [prompt])
    assert row_rel_err(g_last, o_last).max() <= 2e-2
    for rows, bound, ctx in ((17, 17, None), (9, 64, None), (5, 5, 192)):
        toks = gen.randint(14, 700 + rows, rows, shape.vocab)
        off = [0, rows]
        g, st = gm.verify([150], toks, off, max_ctx=ctx, max_rows=bound)
        o, _ = OF.verify_block(om, copy.deepcopy(oc), [150], toks, off)
        assert st[0] == 0
        err = row_rel_err(g, o).max()
        note(f"  rows {rows} bound {bound} max_ctx {ctx or cap}: max row rel err {err:.2e}")
        assert err <= 2e-2
