"""Multi-round speculative decoding on the device (Sec. 3.1 rounds, Sec. 3.2-3.4 length
selection, and the baseline policies of Sec. 4.1 / Appendix B).

A round is, on one stream and without a host round trip:
  drafter -> length (lsv_select_length | lsv_select_joint | lsv_next_length_g4 | a static length)
          -> lsv_pack_block -> lsv_verify_block -> lsv_accept (greedy, commits seq_len)
          -> lsv_next_roots.
``kv`` is a slab cache (runtime.KVCache, ``capacity`` positions per sequence) or a paged one
(runtime.PagedKVCache, ``capacity`` = its pages per sequence x 64).  The drafter is the caller's: a callable (seq_len, drafts, conf) that fills the round's
drafts [B, G] and confidences [B, G] on the device.  ``cost`` is indexed by gamma (cost[0]
unused) for the per-sequence rules, and by the batch's total drafts (B * G + 1 entries) for
the joint rule.  The status array is shared by verify and accept: the acceptance skips a
sequence whose verify step failed (for instance a block past ``max_ctx``), so nothing is
committed for it and its root is kept.  ``capture()`` records one round in a
graph; ``replay()`` runs it.  This module only marshals buffers: every step runs in the
library's kernels.

Blocks on demand (Algorithm 1's budget): with the 'alg1' policy and a drafter that has
``fill_blocks(seq_len, have, want, drafts, conf, n)`` (fill the blocks of n = ``block_n``
drafts [have_b, want_b) of each sequence), a round drafts the first block only, runs the rule with
LSV_SEL_DRAFTED, drafts the blocks it asks for, and runs it again -- at most
ceil(G / block_n) times, all on the device -- so the drafter produces exactly the blocks the
rule's budget requests (``blocks`` after the round).  Other policies draft all G tokens.

Sampling (Sec. 3.1's sampling setting): ``accept="sample"`` with a temperature and a seed
uses lsv_accept's speculative rejection sampling; the drafter is then called as
``drafter(seq_len, drafts, conf, probs)`` and also writes its proposal distributions
probs [B, G, vocab] (draft k of sequence b drawn from probs[b, k]).  The Philox round index
is the round count, a host argument, so sampling rounds run eagerly (no capture)."""
import torch

from . import lsv, runtime

POLICIES = ("marginal", "exhaustive", "alg1", "joint", "g4", "static")


class DecodeLoop:
    def __init__(self, cfg, dm, kv, capacity, batch, G, policy, drafter, cost=None, alpha=2.2, block_n=8,
                 d_min=1, gamma0=None, max_ctx=None, device="cuda", accept="greedy", temperature=1.0, seed=0):
        if policy not in POLICIES:
            raise ValueError(f"policy must be one of {POLICIES}")
        if accept not in ("greedy", "sample"):
            raise ValueError("accept must be 'greedy' or 'sample'")
        if accept == "sample" and not temperature > 0.0:
            raise ValueError("sampling needs a temperature > 0")
        if policy in ("marginal", "exhaustive", "joint") and cost is None:
            raise ValueError("the marginal, exhaustive and joint rules need a cost table")
        if cost is not None and policy in ("marginal", "exhaustive", "joint"):
            need = batch * G + 1 if policy == "joint" else G + 1
            if len(cost) < need:
                raise ValueError(f"the {policy} rule reads {need} cost entries (cost[0..{need - 1}]); got {len(cost)}")
        B = batch
        self.cfg, self.dm, self.kv, self.cap, self.B, self.G = cfg, dm, kv, capacity, B, G
        self.policy, self.drafter, self.alpha, self.block_n, self.d_min = policy, drafter, alpha, block_n, d_min
        self.max_ctx = max_ctx or capacity
        self.max_rows = B * (G + 1)
        self.width = G + 1
        i32 = dict(dtype=torch.int32, device=device)
        self.seq_len = torch.zeros(B, **i32)
        self.roots = torch.zeros(B, **i32)
        self.drafts = torch.zeros((B, max(G, 1)), **i32)
        self.conf = torch.zeros((B, max(G, 1)), dtype=torch.float32, device=device)
        self.gamma = torch.zeros(B, **i32)
        self.aux = torch.zeros(B, **i32)
        self.row_off = torch.zeros(B + 1, **i32)
        self.status = torch.zeros(B, **i32)
        self.tokens = torch.zeros(self.max_rows, **i32)
        self.acc = torch.zeros(B, **i32)
        self.out = torch.zeros((B, self.width), **i32)
        self.logits = torch.zeros((self.max_rows, cfg.vocab), dtype=torch.float32, device=device)
        self.cost = torch.tensor(cost, dtype=torch.float64, device=device) if cost is not None else None
        # blocks on demand: blocks drafted this round per sequence
        self.on_demand = policy == "alg1" and G > 0 and hasattr(drafter, "fill_blocks")
        self.blocks = torch.zeros(B, **i32)
        self.no_blocks = torch.zeros(B, **i32)
        self.accept, self.temperature, self.seed, self.rounds = accept, float(temperature), int(seed), 0
        if accept == "sample":
            # proposal distributions in the drafter's layout, and in lsv_accept's (row
            # row_offsets[b] - b + v - 1 holds q_v of sequence b; one spare row takes the
            # positions past each sequence's gamma)
            self.probs = torch.zeros((B, max(G, 1), cfg.vocab), dtype=torch.float32, device=device)
            self.draft_probs = torch.zeros((B * max(G, 1) + 1, cfg.vocab), dtype=torch.float32, device=device)
            self.kk = torch.arange(max(G, 1), dtype=torch.int64, device=device)
            self.bb = torch.arange(B, dtype=torch.int64, device=device)
        self.ws = runtime.Workspace(lsv.lsv_verify_workspace_bytes(cfg, B, self.max_rows, capacity))
        self.aws = runtime.Workspace(lsv.lsv_accept_workspace_bytes(B, self.max_rows, cfg.vocab))
        g0 = G if gamma0 is None else gamma0
        self.gamma0 = g0
        self.graph = None
        if policy == "static":
            self.gamma.fill_(g0)
            self.row_off.copy_(torch.arange(0, B + 1, **i32) * (g0 + 1))

    def reset(self, seq_len, roots):
        """Start (or restart) from cached lengths seq_len[b] with pending tokens roots[b]."""
        self.seq_len.copy_(torch.as_tensor(seq_len, dtype=torch.int32))
        self.roots.copy_(torch.as_tensor(roots, dtype=torch.int32))
        if self.policy == "g4":  # a made-up previous round from which the rule gives gamma0
            g0 = self.gamma0
            prev, acc = (g0 - 2, g0 - 2) if g0 >= 2 else (g0 + 1, 0)
            self.gamma.fill_(prev)
            self.acc.fill_(acc)
            self.status.zero_()

    def _draft_on_demand(self):
        """Algorithm 1 with blocks on demand: the first block, then what the rule asks for."""
        B, G, n = self.B, self.G, self.block_n
        self.blocks.fill_(1)
        self.drafter.fill_blocks(self.seq_len, self.no_blocks, self.blocks, self.drafts, self.conf, n)
        for _ in range(-(-G // n)):
            self.aux.copy_(self.blocks)
            lsv.lsv_select_length(lsv.LSV_SEL_ALG1, B, G, self.conf, None, 1, G, self.alpha, n, lsv.LSV_SEL_DRAFTED,
                                  self.gamma, self.aux, self.row_off, self.status)
            self.drafter.fill_blocks(self.seq_len, self.blocks, self.aux, self.drafts, self.conf, n)
            torch.maximum(self.blocks, self.aux, out=self.blocks)
        # the rule over the drafted blocks ends here (it never asks for more than it reaches)
        self.aux.copy_(self.blocks)
        lsv.lsv_select_length(lsv.LSV_SEL_ALG1, B, G, self.conf, None, 1, G, self.alpha, n, lsv.LSV_SEL_DRAFTED,
                              self.gamma, self.aux, self.row_off, self.status)

    def round(self):
        B, G = self.B, self.G
        if self.on_demand:
            self._draft_on_demand()
        elif G > 0 and self.drafter is not None:  # no drafter: the drafts buffer keeps its contents
            if self.accept == "sample":
                self.drafter(self.seq_len, self.drafts, self.conf, self.probs)
            else:
                self.drafter(self.seq_len, self.drafts, self.conf)
            self.blocks.fill_(-(-G // self.block_n))
        if self.on_demand:
            pass  # the length came with the drafting
        elif self.policy in ("marginal", "exhaustive", "alg1"):
            mode = {"marginal": lsv.LSV_SEL_MARGINAL, "exhaustive": lsv.LSV_SEL_EXHAUSTIVE,
                    "alg1": lsv.LSV_SEL_ALG1}[self.policy]
            lsv.lsv_select_length(mode, B, G, self.conf, self.cost, 1, G, self.alpha, self.block_n, 0, self.gamma,
                                  self.aux, self.row_off, self.status)
        elif self.policy == "joint":
            lsv.lsv_select_joint(B, G, self.conf, self.cost, G, 0, self.gamma, None, self.row_off, self.status)
        elif self.policy == "g4":
            lsv.lsv_next_length_g4(B, self.gamma, self.acc, self.status, self.d_min, G, self.gamma, self.row_off,
                                   None)
        lsv.lsv_pack_block(B, G, self.row_off, self.max_rows, self.roots, self.drafts, self.tokens, None)
        if isinstance(self.kv, runtime.PagedKVCache):
            lsv.lsv_verify_paged(self.cfg, self.dm.buf, self.kv.buf, self.kv.n_pages, self.kv.table, self.kv.max_pages,
                                 B, self.seq_len, self.tokens, self.row_off, None, self.max_rows, self.max_ctx,
                                 self.logits, self.status, self.ws.buf, self.ws.nbytes)
        else:
            lsv.lsv_verify_block(self.cfg, self.dm.buf, self.kv.buf, self.cap, B, self.seq_len, self.tokens,
                                 self.row_off, self.max_rows, self.max_ctx, self.logits, self.status, self.ws.buf,
                                 self.ws.nbytes)
        if self.accept == "sample":
            # q_v of sequence b to row row_offsets[b] - b + v - 1 (v <= gamma_b), the rest to the spare row
            start = self.row_off[:-1].to(torch.int64) - self.bb
            dst = start[:, None] + self.kk[None, :]
            dst = torch.where(self.kk[None, :] < self.gamma.to(torch.int64)[:, None], dst, B * max(G, 1))
            self.draft_probs.index_copy_(0, dst.reshape(-1), self.probs.reshape(-1, self.cfg.vocab))
            lsv.lsv_accept(lsv.LSV_ACC_SAMPLE, B, self.cfg.vocab, self.logits, self.row_off, self.max_rows,
                           self.width, self.tokens, self.draft_probs, self.temperature, self.seed, self.rounds,
                           self.acc, self.out, self.seq_len, self.status, self.aws.buf, self.aws.nbytes)
        else:
            lsv.lsv_accept(lsv.LSV_ACC_GREEDY, B, self.cfg.vocab, self.logits, self.row_off, self.max_rows,
                           self.width, self.tokens, None, 0.0, 0, 0, self.acc, self.out, self.seq_len, self.status,
                           self.aws.buf, self.aws.nbytes)
        lsv.lsv_next_roots(B, self.acc, self.out, self.width, self.status, self.roots)
        self.rounds += 1

    def capture(self):
        """Record one round in a graph (run one round eagerly first to warm the launches)."""
        if self.accept == "sample":
            raise RuntimeError("sampling rounds take the round index from the host: run them eagerly")
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            self.round()

    def replay(self):
        self.graph.replay()

    def emitted(self):
        """This round's emitted tokens per sequence (host lists; synchronises)."""
        acc = self.acc.cpu().tolist()
        out = self.out.cpu().tolist()
        return [out[b][:acc[b] + 1] for b in range(self.B)]
