"""Acceptance of a verified draft block (oracle).  Test infrastructure only.

Paper, Sec. 3.1: after the target scores every drafted position in one forward
pass (giving p_v), the verification step compares q_v with p_v and accepts or
corrects each drafted token, leaving the target's output distribution unchanged.
The paper cites the standard speculative-sampling rule and does not restate it;
the algorithm below is our reading of that rule, fully specified so that GPU and
oracle agree bit for bit.

Row convention (per sequence b): the verify block holds g_b + 1 rows
[root, x_1, ..., x_g]; row v (0-based) is the target's prediction for the token
after position v, so row v-1 scores draft x_v and row g_b yields the bonus token.
Draft-distribution rows for sequence b start at row_offsets[b] - b.

Greedy (temperature 0):
  argmax = smallest index of the row maximum;
  a_b = largest a <= g_b with argmax(row v-1) == x_v for every v <= a;
  emitted tokens: x_1..x_a, then argmax(row a) (a correction if a < g_b, else the bonus).
Sampling (temperature T > 0):
  p_v = softmax(logits_v / T);
  draft v is accepted iff  u_v * q_v(x_v) < p_{v-1}(x_v), u_v ~ U(0,1) from Philox;
  at the first rejection (a = v - 1 accepted) the emitted token is drawn from
  max(0, p_a - q_{a+1}) renormalised (from p_a if that residual is identically 0);
  if all g drafts pass, the bonus is drawn from p_g.
  Categorical draws use the exponential race: y = argmin_x E_x / w_x over w_x > 0,
  E_x = -ln U_x, ties to the smallest x; P(y = x) = w_x / sum(w).
Status: a sequence whose logits rows (or the draft probabilities that the rule reads)
hold a non-finite value gets LSV_ERR_NONFINITE, a_b = 0, no emitted token, no commit;
a sequence with no rows gets LSV_ERR_INVALID_ARG (in sampling mode every sequence of the
batch does, since the draft-row indexing needs every sequence to own a row).
"""
import numpy as np

from . import philox

LSV_OK, LSV_ERR_INVALID_ARG, LSV_ERR_NONFINITE = 0, -1, -5


def argmax_first(row):
    """Smallest index attaining the maximum (numpy returns the first occurrence)."""
    return int(np.argmax(row))


def _empty(B, width):
    return np.zeros(B, np.int32), np.full((B, width), -1, np.int32), np.zeros(B, np.int32)


def accept_greedy(logits, row_offsets, tokens, out_width=None):
    logits = np.asarray(logits)
    off = [int(x) for x in row_offsets]
    B = len(off) - 1
    width = out_width or max(off[b + 1] - off[b] for b in range(B))
    acc, out, status = _empty(B, width)
    for b in range(B):
        r0, r1 = off[b], off[b + 1]
        g = r1 - r0 - 1
        rows = logits[r0:r1]
        if g < 0:
            status[b] = LSV_ERR_INVALID_ARG
            continue
        if not np.all(np.isfinite(rows)):
            status[b] = LSV_ERR_NONFINITE
            continue
        a = 0
        while a < g and argmax_first(rows[a]) == int(tokens[r0 + a + 1]):
            a += 1
        emitted = [int(t) for t in tokens[r0 + 1:r0 + 1 + a]] + [argmax_first(rows[a])]
        acc[b] = a
        out[b, :len(emitted)] = emitted
    return {"accept_len": acc, "out_tokens": out, "status": status}


def softmax_t(row, temperature):
    z = np.asarray(row, dtype=np.float64) / float(temperature)
    z = z - z.max()
    e = np.exp(z)
    return e / e.sum()


def race(weights, uniforms):
    """Exponential race: argmin over w>0 of (-ln U_x) / w_x; returns (winner, keys)."""
    w = np.asarray(weights, dtype=np.float64)
    e = -np.log(uniforms)
    keys = np.full(w.shape, np.inf)
    pos = w > 0
    keys[pos] = e[pos] / w[pos]
    return int(np.argmin(keys)), keys


def accept_sample(logits, row_offsets, tokens, draft_probs, temperature, seed, rnd, out_width=None):
    logits = np.asarray(logits)
    q_all = np.asarray(draft_probs)
    off = [int(x) for x in row_offsets]
    B = len(off) - 1
    V = logits.shape[1]
    width = out_width or max(off[b + 1] - off[b] for b in range(B))
    acc, out, status = _empty(B, width)
    diag = []
    if any(off[b + 1] - off[b] < 1 for b in range(B)):
        # draft rows are indexed row_offsets[b] - b + v - 1: undefined unless every sequence has a row
        status[:] = LSV_ERR_INVALID_ARG
        return {"accept_len": acc, "out_tokens": out, "status": status, "diag": [{} for _ in range(B)]}
    for b in range(B):
        r0, r1 = off[b], off[b + 1]
        g = r1 - r0 - 1
        qbase = r0 - b
        rows = logits[r0:r1]
        d = {"tests": [], "row": None, "residual": None, "keys": None, "weights": None}
        diag.append(d)
        if g < 0:
            status[b] = LSV_ERR_INVALID_ARG
            continue
        if not np.all(np.isfinite(rows)):
            status[b] = LSV_ERR_NONFINITE
            continue
        p = [softmax_t(rows[v], temperature) for v in range(g + 1)]
        a, rejected, bad = 0, False, False
        for v in range(1, g + 1):
            x = int(tokens[r0 + v])
            qx = float(q_all[qbase + v - 1, x])
            if not np.isfinite(qx):
                bad = True
                break
            px = float(p[v - 1][x])
            u = philox.accept_uniform(seed, rnd, b, v)
            d["tests"].append((u, qx, px))
            if u * qx < px:
                a += 1
            else:
                rejected = True
                break
        if bad:
            status[b] = LSV_ERR_NONFINITE
            continue
        if rejected:
            q_next = np.asarray(q_all[qbase + a], dtype=np.float64)
            if not np.all(np.isfinite(q_next)):
                status[b] = LSV_ERR_NONFINITE
                continue
            w = np.maximum(p[a] - q_next, 0.0)
            d["residual"] = True
            if not np.any(w > 0):
                w = p[a]
                d["residual"] = False
        else:
            w = p[a]
            d["residual"] = False
        y, keys = race(w, philox.sample_uniforms(seed, rnd, b, a, V))
        d.update(row=a, keys=keys, weights=w, p=p[a])
        emitted = [int(t) for t in tokens[r0 + 1:r0 + 1 + a]] + [y]
        acc[b] = a
        out[b, :len(emitted)] = emitted
    return {"accept_len": acc, "out_tokens": out, "status": status, "diag": diag}


def commit(seq_len, result):
    """seq_len[b] += a_b + 1 for sequences with status OK (root + accepted drafts)."""
    s = np.array(seq_len, dtype=np.int64).copy()
    ok = result["status"] == LSV_OK
    s[ok] += result["accept_len"][ok] + 1
    return s.astype(np.int32)
