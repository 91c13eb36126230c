"""GPU verify at the batched shapes: more than 64 block rows, which the GEMMs process in
64-row chunks and the attention in passes of query tiles.

* small bf16 model (d 1024, 8/2 x 128 heads), 8 sequences x 33 rows = 264 rows over
  ragged contexts;
* Llama-3-8B width with 1 of its layers, 8 sequences x 33 rows, contexts drawn from
  [1024, 8192] (the batched gamma = 32 workload);
* Qwen2.5-32B width with 1 layer, 4 x 17 rows, context 4096, then speculative rejection
  sampling at T = 1 on the GPU's own logits, bit-exact against the oracle rule;
* Llama-3-70B width with 1 layer, 4 x 33 rows, context 8192, greedy and T = 0.7 sampling.

Logits bar: each row within 2e-2 of its largest |logit| (bf16 operands, fp32 accumulation);
greedy decisions equal wherever the oracle's top-2 margin clears twice the error."""
import numpy as np
import pytest

from oracle import accept as OA
from paper_2608_08721_amd import lsv
from synth import configs, gen
from tests.lsv_testing import note
from tests.test_gpu_accept import gpu_accept, unsettled
from tests.test_gpu_forward import _bf16_case

pytestmark = pytest.mark.gpu


def _sampling_matches(g_logits, off, toks, temperature, seed):
    """GPU sampling acceptance on the GPU's logits vs the oracle rule on the same logits."""
    B, M, V = len(off) - 1, int(off[-1]), g_logits.shape[1]
    q = gen.draft_probs(seed, M - B, V)
    logits = g_logits.astype(np.float32)
    width = int(np.diff(off).max())
    acc, out, st, _ = gpu_accept(lsv.LSV_ACC_SAMPLE, logits, off, toks, width, q, temperature, seed, 77)
    want = OA.accept_sample(logits, off, toks, q, temperature, seed, 77, out_width=width)
    assert np.array_equal(st, want["status"])
    settled = 0
    for b in range(B):
        if unsettled(want["diag"][b]):
            continue
        settled += 1
        assert acc[b] == want["accept_len"][b], b
        assert np.array_equal(out[b], want["out_tokens"][b]), b
    note(f"    sampling T={temperature}: {settled}/{B} sequences bit-exact (rest within rounding of a threshold)")
    assert settled >= B - 1


def test_small_bf16_264_rows():
    rng = np.random.default_rng(21)
    contexts = [int(c) for c in rng.integers(1, 300, size=8)]
    _bf16_case(configs.SMALL_BF16, 21, contexts, [33] * 8)


def test_llama8b_width_batched_264_rows():
    shape = configs.LLAMA3_8B.with_layers(1)
    wl = configs.WORKLOADS["llama3-8b-b8-ragged"]
    contexts = [int(c) for c in gen.contexts(wl)]
    note(f"llama3-8b width, 1 layer, contexts {contexts}")
    _bf16_case(shape, 3, contexts, [33] * 8)


def test_qwen32b_width_sampling():
    shape = configs.QWEN25_32B.with_layers(1)
    note("qwen2.5-32b width, 1 layer, 4 x 17 rows, context 4096")
    gm, g_logits, o_logits, toks, off = _bf16_case(shape, 4, [4096] * 4, [17] * 4)
    _sampling_matches(g_logits, off, toks, 1.0, 404)


def test_llama70b_width_greedy_and_sampling():
    shape = configs.LLAMA3_70B.with_layers(1)
    note("llama3-70b width, 1 layer, 4 x 33 rows, context 8192")
    gm, g_logits, o_logits, toks, off = _bf16_case(shape, 5, [8192] * 4, [33] * 4)
    _sampling_matches(g_logits, off, toks, 0.7, 505)


def test_short_blocks_under_a_batched_bound():
    """Blocks of at most 64 rows under a bound above 64 (the selected lengths of a batch whose
    worst case is large): the 64-row GEMM kernel serves them and the batched kernels, launched
    too, return at once; Llama-3-70B width with 28 rows under a 132-row bound, the small model
    with 20 rows under 272."""
    _bf16_case(configs.LLAMA3_70B.with_layers(1), 24, [8192, 8100, 5000, 7000], [8, 8, 6, 6], bound=132)
    _bf16_case(configs.SMALL_BF16, 25, [300, 40, 129], [9, 5, 6], bound=272)
