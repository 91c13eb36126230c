"""lsv_accept_noalloc (the acceptance for callers that cannot allocate: its scratch is a fixed
array the library owns on each GPU) against lsv_accept with a caller workspace, through the
C-ABI: greedy and sampling, two calls in a row with the second one smaller, bit for bit on
every output (accepted lengths, emitted tokens, committed lengths, status)."""
import numpy as np
import pytest
import torch

from paper_2608_08721_amd import lsv, runtime
from tests.lsv_testing import i32, note

pytestmark = pytest.mark.gpu


def _block(rng, B, rows_hi, V):
    rows = rng.integers(1, rows_hi + 1, size=B)
    off = runtime.row_offsets_of(rows)
    M = int(off[-1])
    logits = rng.normal(size=(M, V)).astype(np.float32) * 3
    tokens = rng.integers(0, V, size=M).astype(np.int32)
    # make some drafts the row argmax so that prefixes get accepted
    for r in range(M - 1):
        if rng.random() < 0.6:
            tokens[r + 1] = int(np.argmax(logits[r]))
    q = rng.dirichlet(np.ones(V) * 0.3, size=M).astype(np.float32)
    return off, logits, tokens, q, int(rows.max())


def _run(fn, mode, off, logits, tokens, q, width, seq_len, status_in, with_ws):
    B = len(off) - 1
    M, V = logits.shape
    acc = torch.full((B,), -9, dtype=torch.int32, device="cuda")
    out = torch.full((B, width), -9, dtype=torch.int32, device="cuda")
    sl = i32(seq_len)
    st = i32(status_in)
    lg = torch.tensor(logits, device="cuda")
    qq = torch.tensor(q, device="cuda") if mode == lsv.LSV_ACC_SAMPLE else None
    T = 0.8 if mode == lsv.LSV_ACC_SAMPLE else 0.0
    args = [mode, B, V, lg, i32(off), M, width, i32(tokens), qq, T, 11, 5, acc, out, sl, st]
    if with_ws:
        ws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, M, V))
        fn(*args, ws.buf, ws.nbytes)
    else:
        fn(*args)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (acc, out, sl, st)]


@pytest.mark.parametrize("mode", [lsv.LSV_ACC_GREEDY, lsv.LSV_ACC_SAMPLE])
def test_noalloc_matches_workspace_acceptance(mode):
    rng = np.random.default_rng(90 + mode)
    # first call: 8 sequences of up to 33 rows over a 128256-entry vocabulary; second: smaller
    for B, rows_hi, V in ((8, 33, 128256), (3, 9, 5000)):
        off, logits, tokens, q, width = _block(rng, B, rows_hi, V)
        seq_len = rng.integers(100, 1000, size=B)
        status_in = np.zeros(B, np.int32)
        status_in[rng.integers(0, B)] = lsv.LSV_ERR_CAPACITY  # one sequence arrives with an error
        want = _run(lsv.lsv_accept, mode, off, logits, tokens, q, width, seq_len, status_in, True)
        got = _run(lsv.lsv_accept_noalloc, mode, off, logits, tokens, q, width, seq_len, status_in, False)
        for w, g, name in zip(want, got, ("accept_len", "out_tokens", "seq_len", "status")):
            assert np.array_equal(w, g), (B, V, name)
        note(f"  mode {mode}: batch {B} x <= {rows_hi} rows, vocab {V}: accept_len {list(got[0])} identical")
