"""GPU acceptance vs the oracle on identical synthetic logits (and draft distributions).

Greedy: bit-exact accepted lengths, emitted tokens, committed lengths and status.
Sampling: bit-exact except decisions the two precisions cannot settle alike (the
ratio test or the race winner within the fp32-softmax error of a tie); those are
counted and must stay rare."""
import numpy as np
import pytest
import torch

from oracle import accept as OA
from paper_2608_08721_amd import lsv, runtime
from synth import gen
from tests.lsv_testing import i32, note

pytestmark = pytest.mark.gpu


def gpu_accept(mode, logits, off, tokens, width, q=None, temperature=0.0, seed=0, rnd=0, seq_len=None, status_in=None):
    B = len(off) - 1
    M, V = logits.shape
    ws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, M, V))
    lg = torch.tensor(logits, dtype=torch.float32, device="cuda")
    qq = torch.tensor(q, dtype=torch.float32, device="cuda") if q is not None else None
    acc = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((B, width), -9, dtype=torch.int32, device="cuda")
    st = i32(status_in if status_in is not None else [0] * B)  # in/out: the incoming status
    sl = i32(seq_len) if seq_len is not None else None
    lsv.lsv_accept(mode, B, V, lg, i32(off), M, width, i32(tokens), qq, temperature, seed, rnd, acc, out, sl, st,
                   ws.buf, ws.nbytes)
    torch.cuda.synchronize()
    return (acc.cpu().numpy(), out.cpu().numpy(), st.cpu().numpy(), sl.cpu().numpy() if sl is not None else None)


def make_block(rng, B, max_rows, V, seed, integer_logits=False):
    rows = rng.integers(1, max_rows + 1, size=B)
    off = runtime.row_offsets_of(rows)
    M = int(off[-1])
    if integer_logits:
        logits = rng.integers(-2, 3, size=(M, V)).astype(np.float32)
    else:
        logits = gen.synthetic_logits(seed, M, V, std=2.0)
    tokens = gen.randint(seed, 77, M, V)
    for b in range(B):  # plant a matching prefix
        k = int(rng.integers(0, rows[b]))
        for v in range(1, k + 1):
            tokens[off[b] + v] = int(np.argmax(logits[off[b] + v - 1]))
    return off, logits, tokens, int(rows.max())


def test_greedy_parity():
    rng = np.random.default_rng(5)
    for trial in range(40):
        B = int(rng.integers(1, 9))
        V = int(rng.choice([3, 17, 1000, 4096, 4097, 50000]))
        off, logits, tokens, width = make_block(rng, B, int(rng.choice([2, 17, 33, 64])), V, trial,
                                                integer_logits=(trial % 3 == 0))
        if trial % 5 == 1:
            logits[int(off[0]), int(rng.integers(V))] = np.nan
        if trial % 7 == 2:
            logits[int(off[-1]) - 1, 0] = np.inf
        seq = rng.integers(0, 1000, size=B).astype(np.int32)
        acc, out, st, sl = gpu_accept(lsv.LSV_ACC_GREEDY, logits, off, tokens, width, seq_len=seq)
        want = OA.accept_greedy(logits, off, tokens, out_width=width)
        assert np.array_equal(st, want["status"]), trial
        assert np.array_equal(acc, want["accept_len"]), trial
        assert np.array_equal(out, want["out_tokens"]), trial
        assert np.array_equal(sl, OA.commit(seq, want)), trial
    note("greedy accept parity: 40 batches bit-exact")


def test_greedy_full_vocab_llama():
    rng = np.random.default_rng(6)
    off, logits, tokens, width = make_block(rng, 1, 17, 128256, 99)
    acc, out, st, _ = gpu_accept(lsv.LSV_ACC_GREEDY, logits, off, tokens, width)
    want = OA.accept_greedy(logits, off, tokens, out_width=width)
    assert np.array_equal(acc, want["accept_len"]) and np.array_equal(out, want["out_tokens"])


def draws_from(q_rows, u):
    cdf = np.cumsum(q_rows.astype(np.float64), axis=1)
    return np.array([int(np.searchsorted(cdf[i], u[i] * cdf[i, -1], side="right")) for i in range(len(q_rows))])


def unsettled(diag, tol=1e-5):
    """True when an fp32-vs-fp64 difference could flip a decision of this sequence."""
    for (u, qx, px) in diag["tests"]:
        if abs(u * qx - px) <= tol * max(px, u * qx):
            return True
    keys = diag.get("keys")
    if keys is None:
        return False
    w = diag["weights"]
    p = diag["p"]
    finite = np.isfinite(keys)
    if finite.sum() < 2:
        return False
    rel = np.full(keys.shape, np.inf)
    rel[finite] = 1e-6 + 4e-6 * (p[finite] + np.abs(p[finite] - w[finite])) / w[finite]
    win = int(np.argmin(keys))
    hi = keys[win] * (1 + rel[win])
    lo = keys * (1 - np.minimum(rel, 0.5))
    lo[win] = np.inf
    return bool(np.min(lo) <= hi)


@pytest.mark.parametrize("temperature", [1.0, 0.7])
def test_sampling_parity(temperature):
    rng = np.random.default_rng(int(temperature * 10))
    skipped = total = 0
    for trial in range(24):
        B = int(rng.integers(1, 5))
        V = int(rng.choice([5, 64, 4096, 32000]))
        rows = rng.integers(1, 18, size=B)
        off = runtime.row_offsets_of(rows)
        M = int(off[-1])
        logits = gen.synthetic_logits(1000 + trial, M, V, std=float(rng.choice([0.5, 2.0, 4.0])))
        q = gen.draft_probs(2000 + trial, M - B, V)
        tokens = gen.randint(3000 + trial, 5, M, V)
        for b in range(B):
            d = draws_from(q[off[b] - b:off[b + 1] - b - 1], rng.random(rows[b] - 1))
            tokens[off[b] + 1:off[b + 1]] = d
        width = int(rows.max())
        seed, rnd = 1234567 + trial, 42 + trial
        acc, out, st, _ = gpu_accept(lsv.LSV_ACC_SAMPLE, logits, off, tokens, width, q, temperature, seed, rnd)
        want = OA.accept_sample(logits, off, tokens, q, temperature, seed, rnd, out_width=width)
        assert np.array_equal(st, want["status"])
        for b in range(B):
            total += 1
            if unsettled(want["diag"][b]):
                skipped += 1
                continue
            assert acc[b] == want["accept_len"][b], (trial, b)
            assert np.array_equal(out[b], want["out_tokens"][b]), (trial, b)
    note(f"sampling parity T={temperature}: {total - skipped}/{total} sequences bit-exact, {skipped} unsettled")
    assert skipped <= max(1, total // 20)


def test_sampling_nonfinite_and_one_hot():
    V = 40
    logits = np.zeros((4, V), np.float32)
    am = [3, 7, 11, 13]
    for r in range(4):
        logits[r, am[r]] = 1000.0
    q = gen.draft_probs(1, 3, V)
    tokens = np.array([0, 3, 7, 5], np.int32)   # two drafts match the one-hot target, the third does not
    acc, out, st, _ = gpu_accept(lsv.LSV_ACC_SAMPLE, logits, [0, 4], tokens, 4, q, 1.0, 9, 9)
    assert st[0] == 0 and acc[0] == 2 and list(out[0]) == [3, 7, 11, -1]
    logits[1, 5] = np.nan
    acc, out, st, _ = gpu_accept(lsv.LSV_ACC_SAMPLE, logits, [0, 4], tokens, 4, q, 1.0, 9, 9)
    assert st[0] == lsv.LSV_ERR_NONFINITE and acc[0] == 0 and list(out[0]) == [-1] * 4


@pytest.mark.parametrize("mode", [lsv.LSV_ACC_GREEDY, lsv.LSV_ACC_SAMPLE])
def test_incoming_error_status_skips_the_sequence(mode):
    """A sequence that arrives with an error (as lsv_verify_block reports a block past the cache
    capacity) emits nothing, accepts nothing, is not committed and keeps its status; the others
    are decided as usual."""
    rng = np.random.default_rng(77)
    B, V, width = 3, 300, 6
    rows = [4, 6, 2]
    off = runtime.row_offsets_of(rows)
    M = int(off[-1])
    logits = rng.normal(size=(M, V)).astype(np.float32)
    tokens = rng.integers(0, V, size=M).astype(np.int32)
    q = None
    if mode == lsv.LSV_ACC_SAMPLE:
        q = rng.dirichlet(np.ones(V), size=M - B).astype(np.float32)
    seq_len = [10, 20, 30]
    args = dict(q=q, temperature=0.0 if q is None else 1.0, seed=5, rnd=3, seq_len=seq_len)
    acc0, out0, st0, sl0 = gpu_accept(mode, logits, off, tokens, width, **args)
    assert list(st0) == [0, 0, 0]
    acc, out, st, sl = gpu_accept(mode, logits, off, tokens, width, status_in=[0, lsv.LSV_ERR_CAPACITY, 0], **args)
    assert list(st) == [0, lsv.LSV_ERR_CAPACITY, 0]
    assert acc[1] == 0 and np.all(out[1] == -1) and sl[1] == seq_len[1]
    for b in (0, 2):
        assert acc[b] == acc0[b] and np.array_equal(out[b], out0[b]) and sl[b] == sl0[b]
