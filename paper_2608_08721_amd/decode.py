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
library's kernels."""
import torch

from . import lsv, runtime

POLICIES = ("marginal", "exhaustive", "alg1", "joint", "g4", "static")


class DecodeLoop:
    def __init__(self, cfg, dm, kv, capacity, batch, G, policy, drafter, cost=None, alpha=2.2, block_n=8,
                 d_min=1, gamma0=None, max_ctx=None, device="cuda"):
        if policy not in POLICIES:
            raise ValueError(f"policy must be one of {POLICIES}")
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

    def round(self):
        B, G = self.B, self.G
        if G > 0 and self.drafter is not None:  # no drafter: the drafts buffer keeps its contents
            self.drafter(self.seq_len, self.drafts, self.conf)
        if self.policy in ("marginal", "exhaustive", "alg1"):
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
        lsv.lsv_accept(lsv.LSV_ACC_GREEDY, B, self.cfg.vocab, self.logits, self.row_off, self.max_rows, self.width,
                       self.tokens, None, 0.0, 0, 0, self.acc, self.out, self.seq_len, self.status, self.aws.buf,
                       self.aws.nbytes)
        lsv.lsv_next_roots(B, self.acc, self.out, self.width, self.status, self.roots)

    def capture(self):
        """Record one round in a graph (run one round eagerly first to warm the launches)."""
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
