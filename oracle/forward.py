"""Target-model forward pass over a drafted block (oracle).  Test infrastructure only.

Paper, Sec. 3.1: the target evaluates all drafted positions in parallel in a
single forward pass, yielding p_v for every position.  The paper does not fix the
target architecture; the workloads use Llama-style pre-norm decoders (RMSNorm,
rotary position embedding, SwiGLU feed-forward, grouped-query attention), which
this module writes out directly in fp64:

  h = E[tok]
  per layer:
    a = R(N(h, g_attn))                    N(x, g) = x / sqrt(mean(x^2) + eps) * g
    q, k, v = a Wq^T, a Wk^T, a Wv^T
    q, k = rope(q, pos), rope(k, pos)      rotate-half pairs (i, i + hd/2),
                                           angle = pos * base^(-2i/hd)
    q, k, v = R(q), R(k), R(v);  cache[pos] <- k, v
    o = R(softmax(q K^T / sqrt(hd)) V)     keys 0..pos of the same sequence;
                                           query head h reads kv head h // (n_q / n_kv)
    h = h + o Wo^T
    a = R(N(h, g_ffn));  u = R(silu(a Wg^T) * (a Wu^T));  h = h + u Wd^T
  logits = R(N(h, g_final)) Wlm^T

R() is the identity for fp32 models.  For bf16 models it rounds to bf16
(fp64 -> fp32 -> bf16, nearest-even both times) at the points where a bf16 model
stores a matrix operand: the normalised activations, q, k, v, the attention output
and the SwiGLU output.  Everything else -- the residual stream h, every product and
the logits -- stays in fp64.  Weights arrive in their storage type (bf16 values are
exact in fp64).  This is the plain definition of the model; how a kernel schedules
the norm (for example folding the gain into the weights) is not mirrored here.

Row layout: ``tokens`` holds, per sequence b, rows row_offsets[b]..row_offsets[b+1]-1
at positions seq_len[b] + (row - row_offsets[b]); the block's K/V overwrite those
cache positions before attention reads them (causal within the block).
A prefill is the same call with the prompt as the block and seq_len = 0.
"""
import numpy as np

LSV_OK, LSV_ERR_INVALID_ARG, LSV_ERR_CAPACITY = 0, -1, -4


def round_bf16(x):
    """fp64 -> fp32 (nearest-even) -> bf16 (nearest-even) -> fp64."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def stored_to_f64(arr, dtype):
    a = np.asarray(arr)
    if dtype == "bf16":
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def rmsnorm(x, g, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(z):
    return z / (1.0 + np.exp(-z))


def rope(x, pos, base):
    """Rotate-half rotary embedding.  x: [rows, heads, hd]; pos: [rows] ints."""
    hd = x.shape[-1]
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = base ** (-2.0 * i / hd)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


class Model:
    """fp64 view of a model.  ``weights`` = synth.gen.model_weights(...) layout:
    row-major [out, in] matrices in the storage dtype."""

    def __init__(self, shape, weights, layers=None):
        self.m = shape
        self.dtype = shape.dtype
        self.w = weights
        self.n_layers = shape.n_layers if layers is None else layers
        self._cache = {}

    def f64(self, key, layer=None):
        """fp64 copy of a weight (cached per layer for small models)."""
        ck = (key, layer)
        if ck in self._cache:
            return self._cache[ck]
        src = self.w["layers"][layer][key] if layer is not None else self.w[key]
        out = stored_to_f64(src, self.dtype)
        if out.size <= (1 << 24):
            self._cache[ck] = out
        return out

    def R(self, x):
        return round_bf16(x) if self.dtype == "bf16" else x

    def linear(self, x, key, layer=None):
        """x @ W^T.  Large matrices are converted to fp64 in slices of output rows; every
        output element is still one full dot product."""
        src = self.w["layers"][layer][key] if layer is not None else self.w[key]
        if src.size <= (1 << 24):
            return x @ self.f64(key, layer).T
        out = np.empty((x.shape[0], src.shape[0]))
        step = max(1, (1 << 23) // src.shape[1])
        for s in range(0, src.shape[0], step):
            out[:, s:s + step] = x @ stored_to_f64(src[s:s + step], self.dtype).T
        return out

    def normed(self, h, gain):
        """R(N(h, gain)): the normalised activation a projection consumes."""
        return self.R(rmsnorm(h, gain, self.m.rms_eps))


class KVCache:
    """Per layer K and V, [B, n_kv, capacity, hd] in fp64 (bf16 values for bf16 models)."""

    def __init__(self, shape, batch, capacity, n_layers=None):
        L = shape.n_layers if n_layers is None else n_layers
        dims = (batch, shape.n_kv_heads, capacity, shape.head_dim)
        self.k = [np.zeros(dims) for _ in range(L)]
        self.v = [np.zeros(dims) for _ in range(L)]
        self.capacity = capacity


def tree_depths(parents):
    """Depth of every node of one tree (node 0 the root, parent[0] = -1, parent[r] < r);
    None when the parents do not form such a tree."""
    par = [int(p) for p in parents]
    if not par or par[0] != -1:
        return None
    depth = [0]
    for r in range(1, len(par)):
        if not 0 <= par[r] < r:
            return None
        depth.append(depth[par[r]] + 1)
    return depth


def ancestors(parents, r):
    """Node r and its ancestors, in increasing order (the root first)."""
    out = [r]
    while parents[out[-1]] >= 0:
        out.append(int(parents[out[-1]]))
    return out[::-1]


def verify_block(model, cache, seq_len, tokens, row_offsets, parents=None, collect_hidden=False):
    """One forward pass over the block; returns (logits fp64 [M, V], status [B]).

    parents (optional, [M]): the block of each sequence is a tree of drafts -- parents[r] is the
    parent of row r as a row index within its sequence's block (-1 for the sequence's first row,
    the root; a parent precedes its children).  Row r then sits at position seq_len + depth(r),
    is stored at cache slot seq_len + (r - row_offsets[b]), and attends to the cached context and
    to the slots of its ancestors and itself.  Without parents the block is a chain: row r's
    parent is r - 1, which is the plain causal block."""
    m = model.m
    off = [int(x) for x in row_offsets]
    B = len(off) - 1
    M = off[-1]
    tokens = np.asarray(tokens, dtype=np.int64)
    hd, nq, nkv = m.head_dim, m.n_q_heads, m.n_kv_heads
    group = nq // nkv
    status = np.zeros(B, np.int32)
    seq_of_row = np.zeros(M, np.int64)
    pos = np.zeros(M, np.int64)     # rotary position
    slot = np.zeros(M, np.int64)    # cache slot
    keys = [None] * M               # block slots a row attends to, besides the cached context
    for b in range(B):
        n = off[b + 1] - off[b]
        C = int(seq_len[b])
        par = list(range(-1, n - 1)) if parents is None else [int(p) for p in parents[off[b]:off[b + 1]]]
        depth = tree_depths(par) if n else []
        seq_of_row[off[b]:off[b + 1]] = b
        slot[off[b]:off[b + 1]] = C + np.arange(n)
        if depth is None:
            status[b] = LSV_ERR_INVALID_ARG
            continue
        pos[off[b]:off[b + 1]] = C + np.asarray(depth, dtype=np.int64)
        for i in range(n):
            keys[off[b] + i] = [C + j for j in ancestors(par, i)]
        if C + n > cache.capacity:
            status[b] = LSV_ERR_CAPACITY
        if np.any((tokens[off[b]:off[b + 1]] < 0) | (tokens[off[b]:off[b + 1]] >= m.vocab)):
            status[b] = LSV_ERR_INVALID_ARG

    emb = model.w["embed"]
    h = np.zeros((M, m.d_model))
    for r in range(M):
        if 0 <= tokens[r] < m.vocab:
            h[r] = stored_to_f64(emb[tokens[r]], model.dtype)
    hidden = []
    for l in range(model.n_layers):
        a = model.normed(h, model.f64("attn_norm", l))
        q = model.linear(a, "wq", l).reshape(M, nq, hd)
        k = model.linear(a, "wk", l).reshape(M, nkv, hd)
        v = model.linear(a, "wv", l).reshape(M, nkv, hd)
        q = model.R(rope(q, pos, m.rope_base))
        k = model.R(rope(k, pos, m.rope_base))
        v = model.R(v)
        for r in range(M):
            b = seq_of_row[r]
            if status[b] == LSV_OK:
                cache.k[l][b, :, slot[r], :] = k[r]
                cache.v[l][b, :, slot[r], :] = v[r]
        o = np.zeros((M, nq, hd))
        for r in range(M):
            b = seq_of_row[r]
            if status[b] != LSV_OK:
                continue
            C = int(seq_len[b])
            if keys[r] == list(range(C, C + len(keys[r]))):  # a chain prefix: the causal keys
                ks = slice(0, C + len(keys[r]))
            else:
                ks = np.concatenate([np.arange(C), np.asarray(keys[r], dtype=np.int64)])
            for hq in range(nq):
                kv = hq // group
                K = cache.k[l][b, kv, ks, :]
                Vv = cache.v[l][b, kv, ks, :]
                s = (K @ q[r, hq]) / np.sqrt(hd)
                s = s - s.max()
                p = np.exp(s)
                p = p / p.sum()
                o[r, hq] = p @ Vv
        o = model.R(o)
        h = h + model.linear(o.reshape(M, nq * hd), "wo", l)
        a = model.normed(h, model.f64("ffn_norm", l))
        u = model.R(silu(model.linear(a, "wg", l)) * model.linear(a, "wu", l))
        h = h + model.linear(u, "wd", l)
        if collect_hidden:
            hidden.append(h.copy())
    logits = model.linear(model.normed(h, stored_to_f64(model.w["final_norm"], model.dtype)), "lm_head")
    if collect_hidden:
        return logits, status, hidden
    return logits, status


def prefill(model, cache, prompts):
    """Fill the cache with each sequence's prompt; returns (last-row logits [B, V], seq_len)."""
    B = len(prompts)
    toks = np.concatenate([np.asarray(p, dtype=np.int64) for p in prompts])
    off = np.concatenate([[0], np.cumsum([len(p) for p in prompts])])
    logits, status = verify_block(model, cache, np.zeros(B, np.int64), toks, off)
    assert np.all(status == LSV_OK)
    last = logits[off[1:] - 1]
    return last, np.array([len(p) for p in prompts], dtype=np.int32)


def greedy_continuation(model, cache, seq_len, root, n):
    """n single-token greedy decode steps for one sequence (B = 1) starting from the
    pending token ``root``; returns the n tokens after root and leaves the cache
    holding root and the first n-1 of them.  Used to plant drafts the target accepts."""
    toks, cur, s = [], int(root), int(seq_len)
    for _ in range(n):
        logits, status = verify_block(model, cache, [s], [cur], [0, 1])
        assert status[0] == LSV_OK
        cur = int(np.argmax(logits[0]))
        toks.append(cur)
        s += 1
    return toks
