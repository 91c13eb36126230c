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
    def __init__(self, stream, q, seed, vocab, G, device="cuda", n=8):
        stream = np.asarray(stream, dtype=np.int64)
        q = np.asarray(q, dtype=np.float32)
        B, L = stream.shape
        rng = np.random.default_rng([seed, 0xD8])
        u = rng.random((B, L))
        wrong = (stream + 1 + rng.integers(0, vocab - 1, size=(B, L))) % vocab  # never the stream token
        pick = np.where(u < q, stream, wrong)
        self.G, self.L, self.n = G, L, n
        self.drafted = torch.zeros(B, dtype=torch.int64, device=device)  # drafts produced, per sequence
        self.pick = torch.tensor(pick, dtype=torch.int32, device=device)
        self.q = torch.tensor(q, dtype=torch.float32, device=device)
        self.k = torch.arange(1, G + 1, dtype=torch.int64, device=device)

    def __call__(self, seq_len, drafts, conf):
        """Drafts and confidences of the round whose root sits at position seq_len[b]:
        draft k is the proposal for position seq_len[b] + k (device ops only)."""
        idx = (seq_len.to(torch.int64)[:, None] + self.k[None, :]).clamp_(max=self.L - 1)
        drafts.copy_(torch.gather(self.pick, 1, idx))
        conf.copy_(torch.gather(self.q, 1, idx))

    def fill_blocks(self, seq_len, have, want, drafts, conf, n=None):
        """Blocks on demand: drafts and confidences k in [have_b * n, want_b * n) of each
        sequence (the other entries keep what they hold).  Device ops only."""
        n = n or self.n
        idx = (seq_len.to(torch.int64)[:, None] + self.k[None, :]).clamp_(max=self.L - 1)
        blk = (self.k - 1) // n
        mask = (blk[None, :] >= have.to(torch.int64)[:, None]) & (blk[None, :] < want.to(torch.int64)[:, None])
        drafts.copy_(torch.where(mask, torch.gather(self.pick, 1, idx).to(drafts.dtype), drafts))
        conf.copy_(torch.where(mask, torch.gather(self.q, 1, idx), conf))
        self.drafted += mask.sum(dim=1, dtype=torch.int64)


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


class SampledDrafter:
    """A proposal distribution per draft for the sampling setting: q = softmax(scale * z),
    z standard normal, drawn on the device from a generator seeded per call, and the draft
    drawn from q; its confidence is q(draft).  Any proposal keeps speculative rejection
    sampling lossless (the emitted tokens follow the target's distribution); this one is
    only there to be one."""

    def __init__(self, seed, vocab, scale=3.0, device="cuda"):
        self.seed, self.vocab, self.scale, self.calls = seed, vocab, scale, 0
        self.gen = torch.Generator(device=device)

    def __call__(self, seq_len, drafts, conf, probs):
        self.gen.manual_seed(self.seed * 1000003 + self.calls)
        self.calls += 1
        B, G, V = probs.shape
        z = torch.randn((B, G, V), generator=self.gen, device=probs.device) * self.scale
        probs.copy_(torch.softmax(z, dim=-1))
        x = torch.multinomial(probs.reshape(-1, V), 1, generator=self.gen).reshape(B, G)
        drafts.copy_(x.to(drafts.dtype))
        conf.copy_(torch.gather(probs, 2, x[:, :, None])[:, :, 0])
