"""GPU baseline length policy (the G4-style rule of Sec. 4.1 / Appendix B) vs the oracle,
bit for bit: random round records (all accepted, rejected, failed, unusable), batches past one
wave, the in-place form, and a three-round chain in which each round's verify layout comes from
the device-written row offsets and its outcome from lsv_accept."""
import numpy as np
import pytest
import torch

from oracle import accept as OA
from oracle import policies as OP
from paper_2608_08721_amd import lsv
from tests.lsv_testing import i32, note
from tests.test_gpu_accept import gpu_accept

pytestmark = pytest.mark.gpu


def random_records(rng, B, d_max):
    gamma = rng.integers(0, d_max + 1, size=B)
    acc = np.array([rng.integers(0, g + 1) for g in gamma])
    full = rng.random(B) < 0.4
    acc[full] = gamma[full]  # a good share of rounds with no rejection
    status = np.where(rng.random(B) < 0.1, lsv.LSV_ERR_NONFINITE, 0)
    bad = rng.random(B) < 0.05
    acc[bad] = gamma[bad] + 1  # more accepted than drafted: flagged
    big = rng.random(B) < 0.03
    gamma[big] = lsv.LSV_MAX_SEQ_ROWS  # past the one-wave block limit: flagged
    return gamma.astype(np.int32), acc.astype(np.int32), status.astype(np.int32)


def gpu_g4(gamma, acc, status, d_min, d_max, with_offsets, with_err, in_place=False):
    B = len(gamma)
    g = i32(gamma)
    nxt = g if in_place else torch.full((B,), -7, dtype=torch.int32, device="cuda")
    ro = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda") if with_offsets else None
    err = torch.full((B,), 99, dtype=torch.int32, device="cuda") if with_err else None
    st = i32(status) if status is not None else None
    lsv.lsv_next_length_g4(B, g, i32(acc), st, d_min, d_max, nxt, ro, err)
    torch.cuda.synchronize()
    return (nxt.cpu().numpy(), ro.cpu().numpy() if ro is not None else None,
            err.cpu().numpy() if err is not None else None)


@pytest.mark.parametrize("B", [1, 5, 64, 65, 200, 1000])
def test_g4_parity_random(B):
    rng = np.random.default_rng(B)
    for trial in range(6):
        d_min, d_max = (1, 16) if trial % 2 == 0 else (3, 60)
        gamma, acc, status = random_records(rng, B, d_max)
        use_status = trial % 3 != 2
        want_n, want_e, want_o = OP.g4_next_batch(gamma, acc, d_min, d_max, status if use_status else None)
        offs = B <= lsv.LSV_MAX_BATCH
        got_n, got_o, got_e = gpu_g4(gamma, acc, status if use_status else None, d_min, d_max, offs, trial != 1,
                                     in_place=trial == 3)
        assert got_n.tolist() == want_n
        if got_e is not None:
            assert got_e.tolist() == want_e
        if offs:
            assert got_o.tolist() == want_o
    note(f"  batch {B}: 6 record sets bit-exact")


def test_g4_chain_with_accept():
    """Three rounds: lengths from the rule, the verify layout from the device row offsets,
    the outcome from the GPU acceptance on logits with planted matching prefixes."""
    rng = np.random.default_rng(77)
    B, V, d_min, d_max = 6, 256, 1, 12
    gamma = np.array([4, 1, 12, 7, 3, 9], np.int32)
    acc0 = np.array([4, 0, 12, 2, 3, 9], np.int32)
    nxt, ro, _ = gpu_g4(gamma, acc0, None, d_min, d_max, True, True)
    want = OP.g4_next_batch(gamma, acc0, d_min, d_max)
    assert nxt.tolist() == want[0] and ro.tolist() == want[2]
    g = nxt
    for rnd in range(3):
        off = ro
        M = int(off[-1])
        logits = rng.normal(size=(M, V)).astype(np.float32)
        toks = rng.integers(0, V, size=M).astype(np.int32)
        plant = [int(rng.integers(0, g[b] + 1)) if rng.random() < 0.5 else int(g[b]) for b in range(B)]
        for b in range(B):
            for v in range(1, g[b] + 1):
                best = int(np.argmax(logits[off[b] + v - 1]))
                toks[off[b] + v] = best if v <= plant[b] else (best + 1) % V
        a, _, st, _ = gpu_accept(lsv.LSV_ACC_GREEDY, logits, off, toks, d_max + 1)
        ref = OA.accept_greedy(logits, off, toks, out_width=d_max + 1)
        assert a.tolist() == list(ref["accept_len"]) == plant and np.all(st == 0)
        nxt, ro, err = gpu_g4(g, a, st, d_min, d_max, True, True)
        want_n, want_e, want_o = OP.g4_next_batch(g, a, d_min, d_max, st)
        assert nxt.tolist() == want_n and ro.tolist() == want_o and err.tolist() == want_e
        note(f"  round {rnd}: gamma {g.tolist()} accepted {plant} -> {want_n}")
        g = nxt
