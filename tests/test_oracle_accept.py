"""Pins for the acceptance oracle: brute-force greedy prefix matching, the lossless
property of speculative sampling (chi-square against the target distribution), the
closed-form acceptance rate, and special cases that reduce to greedy decoding."""
import numpy as np
import pytest
from scipy import stats

from oracle import accept as A


def brute_argmax(row):
    best = 0
    for j in range(1, len(row)):
        if row[j] > row[best]:
            best = j
    return best


def brute_greedy(logits, off, tokens):
    acc, outs = [], []
    for b in range(len(off) - 1):
        r0, r1 = off[b], off[b + 1]
        a = 0
        for v in range(1, r1 - r0):
            if brute_argmax(logits[r0 + v - 1]) != tokens[r0 + v]:
                break
            a += 1
        acc.append(a)
        outs.append(list(tokens[r0 + 1:r0 + 1 + a]) + [brute_argmax(logits[r0 + a])])
    return acc, outs


def test_greedy_matches_brute_force_with_ties():
    rng = np.random.default_rng(0)
    for trial in range(50):
        B = int(rng.integers(1, 5))
        V = int(rng.integers(2, 12))
        g = rng.integers(0, 6, size=B)
        off = np.concatenate([[0], np.cumsum(g + 1)])
        M = off[-1]
        logits = rng.integers(-3, 3, size=(M, V)).astype(np.float32)  # many exact ties
        tokens = rng.integers(0, V, size=M)
        for b in range(B):  # plant a matching prefix of random length
            k = int(rng.integers(0, g[b] + 1))
            for v in range(1, k + 1):
                tokens[off[b] + v] = brute_argmax(logits[off[b] + v - 1])
        res = A.accept_greedy(logits, off, tokens)
        acc, outs = brute_greedy(logits, off, tokens)
        assert list(res["accept_len"]) == acc
        for b in range(B):
            assert list(res["out_tokens"][b][:acc[b] + 1]) == outs[b]
            assert all(x == -1 for x in res["out_tokens"][b][acc[b] + 1:])


def test_greedy_planted_full_acceptance_and_commit():
    rng = np.random.default_rng(1)
    logits = rng.normal(size=(6, 50)).astype(np.float32)
    am = [int(np.argmax(r)) for r in logits]
    tokens = [7] + am[:5]
    res = A.accept_greedy(logits, [0, 6], tokens)
    assert res["accept_len"][0] == 5
    assert list(res["out_tokens"][0]) == am
    assert list(A.commit([100], res)) == [106]


def test_greedy_nonfinite_status():
    logits = np.zeros((4, 5), np.float32)
    logits[2, 3] = np.nan
    res = A.accept_greedy(logits, [0, 2, 4], [0, 3, 0, 0])
    assert list(res["status"]) == [0, A.LSV_ERR_NONFINITE]
    assert res["accept_len"][1] == 0 and all(res["out_tokens"][1] == -1)
    assert list(A.commit([10, 10], res)) == [11, 10]


def _dirichlet_rows(rng, n, V, conc=1.0):
    return rng.dirichlet([conc] * V, size=n)


def _trials(p_rows, q_rows, n_trials, temperature=1.0, seed=11, draft_seed=5):
    """Run the sampling rule on fixed target rows p_0..p_g (given as logits) with drafts drawn
    from q_1..q_g; returns the emitted-token sequences and accept lengths."""
    g = len(q_rows)
    logits = np.log(p_rows) * temperature
    rng = np.random.default_rng(draft_seed)
    emitted, acc = [], []
    cdf = np.cumsum(q_rows, axis=1)
    for t in range(n_trials):
        drafts = [int(np.searchsorted(cdf[v], rng.random() * cdf[v, -1], side="right")) for v in range(g)]
        tokens = [0] + drafts
        res = A.accept_sample(logits, [0, g + 1], tokens, q_rows.astype(np.float32), temperature, seed, t)
        a = int(res["accept_len"][0])
        acc.append(a)
        emitted.append(list(res["out_tokens"][0][:a + 1]))
    return emitted, np.array(acc)


def test_sampling_is_lossless_chi_square():
    """First emitted token ~ p_0; given draft 1 accepted, second emitted ~ p_1; given all g
    accepted, the bonus ~ p_g (fixed target rows, so p_v does not depend on the prefix)."""
    rng = np.random.default_rng(2)
    V, g, n = 8, 3, 20000
    p = _dirichlet_rows(rng, g + 1, V)
    q = _dirichlet_rows(rng, g, V)
    emitted, acc = _trials(p, q, n)
    first = np.bincount([e[0] for e in emitted], minlength=V)
    assert stats.chisquare(first, p[0] * n).pvalue > 1e-4
    sec = [e[1] for e in emitted if len(e) >= 2]
    c2 = np.bincount(sec, minlength=V)
    assert stats.chisquare(c2, p[1] * len(sec)).pvalue > 1e-4
    bonus = [e[g] for e in emitted if len(e) == g + 1]
    if len(bonus) > 500:
        cb = np.bincount(bonus, minlength=V)
        assert stats.chisquare(cb, p[g] * len(bonus)).pvalue > 1e-4


def test_sampling_detects_a_biased_rule():
    """The chi-square check has power: a rule that draws corrections from p instead of the
    residual max(0, p - q) shifts the first-token distribution and fails the same test."""
    rng = np.random.default_rng(2)
    V, g, n = 8, 1, 20000
    p = _dirichlet_rows(rng, g + 1, V)
    q = _dirichlet_rows(rng, g, V)
    draws = np.random.default_rng(9)
    first = np.zeros(V)
    cdf = np.cumsum(q[0])
    for t in range(n):
        x = int(np.searchsorted(cdf, draws.random() * cdf[-1], side="right"))
        if draws.random() * q[0][x] < p[0][x]:
            first[x] += 1
        else:
            first[int(np.searchsorted(np.cumsum(p[0]), draws.random(), side="right"))] += 1
    assert stats.chisquare(first, p[0] * n).pvalue < 1e-4


def test_acceptance_rate_closed_form():
    """P(draft 1 accepted) = sum_x min(p_0(x), q_1(x))."""
    rng = np.random.default_rng(3)
    V, n = 6, 20000
    p = _dirichlet_rows(rng, 2, V)
    q = _dirichlet_rows(rng, 1, V)
    _, acc = _trials(p, q, n)
    rate = np.minimum(p[0], q[0]).sum()
    se = np.sqrt(rate * (1 - rate) / n)
    assert abs((acc >= 1).mean() - rate) < 5 * se


def test_q_equals_p_accepts_everything():
    rng = np.random.default_rng(4)
    V, g = 16, 5
    p = _dirichlet_rows(rng, g + 1, V)
    emitted, acc = _trials(p, p[:g].copy(), 200)
    # u * q < p with q == p holds for every u < 1 (up to float32 rounding of q)
    assert (acc == g).mean() > 0.97


def test_one_hot_target_reduces_to_greedy():
    rng = np.random.default_rng(5)
    V, g = 20, 4
    logits = rng.normal(size=(g + 1, V))
    am = logits.argmax(axis=1)
    logits = np.where(np.arange(V)[None, :] == am[:, None], 1000.0, 0.0).astype(np.float32)
    q = _dirichlet_rows(rng, g, V).astype(np.float32)
    for t in range(30):
        drafts = [int(am[0]), int(am[1]), int(rng.integers(V)), int(rng.integers(V))]
        tokens = [0] + drafts
        res = A.accept_sample(logits, [0, g + 1], tokens, q, 1.0, 3, t)
        gr = A.accept_greedy(logits, [0, g + 1], tokens)
        assert res["accept_len"][0] == gr["accept_len"][0]
        assert list(res["out_tokens"][0]) == list(gr["out_tokens"][0])


def test_race_is_categorical():
    from oracle import philox
    w = np.array([0.1, 0.0, 0.3, 0.6])
    wins = np.bincount([A.race(w, philox.sample_uniforms(1, r, 0, 0, 4))[0] for r in range(20000)], minlength=4)
    assert wins[1] == 0
    assert stats.chisquare(wins[[0, 2, 3]], w[[0, 2, 3]] * 20000).pvalue > 1e-4
