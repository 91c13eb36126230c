"""Synthetic calibrated drafter for multi-round decoding (input generation only).

The paper's drafters are trained models (out of scope here).  This stand-in plants
acceptance: for the token at absolute position p of sequence b it proposes the target's
own greedy token stream[b][p] with probability q[b][p] and some other token otherwise,
and reports q[b][p] as its confidence.  Under greedy acceptance draft k is then accepted,
given that drafts 1..k-1 were, with probability exactly its confidence: the drafter is
calibrated in the sense the selector assumes (Assumption 3.7).

Everything the drafter draws (q, the uniforms, the wrong tokens) is drawn here on the
host from a seed; a round only gathers on the device, so it can sit inside a captured
graph.  The greedy stream comes from the caller (the oracle's or the target's own)."""
import numpy as np
import torch


def confidences(seed, B, L, kind="beta"):
    """Per-position confidences in [0, 1]: 'beta' draws Beta(6, 1.5) (mostly high, a few
    hard tokens), 'uniform' draws U(0, 1)."""
    rng = np.random.default_rng([seed, 0xD7])
    if kind == "uniform":
        return rng.random((B, L))
    return rng.beta(6.0, 1.5, (B, L))


class PlantedDrafter:
    def __init__(self, stream, q, seed, vocab, G, device="cuda"):
        stream = np.asarray(stream, dtype=np.int64)
        q = np.asarray(q, dtype=np.float32)
        B, L = stream.shape
        rng = np.random.default_rng([seed, 0xD8])
        u = rng.random((B, L))
        wrong = (stream + 1 + rng.integers(0, vocab - 1, size=(B, L))) % vocab  # never the stream token
        pick = np.where(u < q, stream, wrong)
        self.G, self.L = G, L
        self.pick = torch.tensor(pick, dtype=torch.int32, device=device)
        self.q = torch.tensor(q, dtype=torch.float32, device=device)
        self.k = torch.arange(1, G + 1, dtype=torch.int64, device=device)

    def __call__(self, seq_len, drafts, conf):
        """Drafts and confidences of the round whose root sits at position seq_len[b]:
        draft k is the proposal for position seq_len[b] + k (device ops only)."""
        idx = (seq_len.to(torch.int64)[:, None] + self.k[None, :]).clamp_(max=self.L - 1)
        drafts.copy_(torch.gather(self.pick, 1, idx))
        conf.copy_(torch.gather(self.q, 1, idx))


def plant_block(continuation, conf, seed, vocab):
    """Drafts for one verify block per sequence, planted like PlantedDrafter: draft v is the
    target's own greedy token continuation[b][v] with probability conf[b][v] and another token
    otherwise, so under greedy acceptance it is accepted (given drafts before it were) with
    exactly its confidence.  continuation, conf: [B, G]; returns int64 [B, G]."""
    cont = np.asarray(continuation, dtype=np.int64)
    q = np.asarray(conf, dtype=np.float64)
    rng = np.random.default_rng([seed, 0xD9])
    u = rng.random(cont.shape)
    wrong = (cont + 1 + rng.integers(0, vocab - 1, size=cont.shape)) % vocab
    return np.where(u < q, cont, wrong)
