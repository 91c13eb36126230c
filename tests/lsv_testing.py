"""Helpers shared by the GPU tests: device set-up and oracle comparisons."""
import numpy as np
import torch

from oracle import forward as OF
from paper_2608_08721_amd import lsv, runtime

DEV = "cuda"


def i32(x):
    return torch.tensor(np.asarray(x, dtype=np.int32), device=DEV)


def note(msg):
    print(msg, flush=True)


class GpuModel:
    """Packed model + KV cache + verify workspace on the GPU, driven through the C-ABI."""

    def __init__(self, shape, weights, batch, capacity, max_rows=64):
        self.shape = shape
        self.cfg = runtime.model_config(shape)
        self.dm = runtime.DeviceModel.from_weights(self.cfg, weights)
        self.batch, self.capacity, self.max_rows = batch, capacity, max_rows
        self.kv = runtime.KVCache(self.cfg, batch, capacity)
        self.ws = runtime.Workspace(lsv.lsv_verify_workspace_bytes(self.cfg, batch, max_rows, capacity))
        self.logits = torch.full((max_rows, shape.vocab), float("nan"), dtype=torch.float32, device=DEV)
        self.status = torch.full((batch,), 99, dtype=torch.int32, device=DEV)

    def verify(self, seq_len, tokens, row_offsets, max_ctx=None, max_rows=None):
        """One lsv_verify_block call; max_rows / max_ctx default to the buffers' bounds (a
        smaller bound reuses the same workspace)."""
        M = int(row_offsets[-1])
        lsv.lsv_verify_block(self.cfg, self.dm.buf, self.kv.buf, self.capacity, self.batch, i32(seq_len),
                             i32(tokens), i32(row_offsets), max_rows or self.max_rows, max_ctx or self.capacity,
                             self.logits, self.status, self.ws.buf, self.ws.nbytes)
        torch.cuda.synchronize()
        return self.logits[:M].double().cpu().numpy(), self.status.cpu().numpy()

    def verify_tree(self, seq_len, tokens, row_offsets, parents, max_rows=None):
        """One lsv_verify_tree call (each sequence's rows form a tree given by parents)."""
        M = int(row_offsets[-1])
        lsv.lsv_verify_tree(self.cfg, self.dm.buf, self.kv.buf, self.capacity, self.batch, i32(seq_len), i32(tokens),
                            i32(row_offsets), i32(parents), max_rows or self.max_rows, self.capacity, self.logits,
                            self.status, self.ws.buf, self.ws.nbytes)
        torch.cuda.synchronize()
        return self.logits[:M].double().cpu().numpy(), self.status.cpu().numpy()

    def prefill(self, prompts):
        """Chunked prefill of every sequence through lsv_verify_block; returns last-row logits."""
        B = len(prompts)
        filled = [0] * B
        last = [None] * B
        per = max(1, self.max_rows // B)
        while any(filled[b] < len(prompts[b]) for b in range(B)):
            take = [min(per, len(prompts[b]) - filled[b]) for b in range(B)]
            toks = [prompts[b][filled[b]:filled[b] + take[b]] for b in range(B)]
            off = runtime.row_offsets_of(take)
            seq = list(filled)
            lg, st = self.verify(seq, np.concatenate(toks), off)
            for b in range(B):
                if take[b]:
                    assert st[b] == 0, st
                    filled[b] += take[b]
                    if filled[b] == len(prompts[b]):
                        last[b] = lg[off[b + 1] - 1]
        return np.stack(last), np.array(filled, dtype=np.int32)


def row_rel_err(got, want):
    """Per row: max |got - want| / max |want|."""
    den = np.maximum(np.abs(want).max(axis=1), 1e-30)
    return (np.abs(got - want).max(axis=1) / den)


def top2_margin(row):
    s = np.sort(row)
    return s[-1] - s[-2]


def greedy_decisions(got, want, min_decided, label=""):
    """Greedy decisions of GPU logits `got` against oracle logits `want`, row by row.

    e_r = max_j |got_rj - want_rj| is row r's measured error.  Where the oracle's top-1 /
    top-2 margin exceeds 2 e_r the row has a single argmax that any logits within e_r of
    the oracle's share ("decided"): GPU and oracle must pick the same token.  Elsewhere
    both picks are near-maximal: the GPU's pick must lie within 2 e_r of the oracle's
    maximum.  At least `min_decided` of the rows must be decided (checked on blocks of ten
    rows or more; a share of fewer says little).  Returns the decided share."""
    e = np.abs(got - want).max(axis=1)
    am_g, am_o = got.argmax(axis=1), want.argmax(axis=1)
    margin = np.array([top2_margin(r) for r in want])
    decided = margin > 2 * e
    bad = [r for r in np.flatnonzero(decided) if am_g[r] != am_o[r]]
    assert not bad, f"argmax differs on decided rows {bad}"
    rows = np.arange(len(want))
    near = want.max(axis=1) - want[rows, am_g] <= 2 * e
    assert near.all(), f"GPU picks far from the oracle's maximum on rows {np.flatnonzero(~near)}"
    frac = float(decided.mean()) if len(decided) else 1.0
    note(f"    {label}argmax equal on {int(decided.sum())}/{len(decided)} decided rows ({frac:.0%}); "
         f"{int((am_g == am_o).sum())}/{len(am_o)} rows equal in all")
    assert len(decided) < 10 or frac >= min_decided, (frac, min_decided)
    return frac
