"""Pins for the length-selector oracle (LibraSpec Sec. 3.2-3.4, Algorithm 1).

Each check comes from outside the oracle's own formula: brute-force enumeration of
the prefix-acceptance model, closed forms, Theorems 3.2/3.5/3.6 as invariants, and
hand-derived special cases (tests/golden)."""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import selector as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "selector_special_cases.json")


def brute_expected_accepted(q, d, start=1):
    """E[# consecutively accepted drafts among start..d] by enumerating every accept/reject
    pattern of independent drafts with acceptance probabilities q (proof of Thm. 3.3)."""
    idx = list(range(start, d + 1))
    total = 0.0
    for pattern in itertools.product((0, 1), repeat=len(idx)):
        prob = 1.0
        for k, acc in zip(idx, pattern):
            prob *= q[k - 1] if acc else (1.0 - q[k - 1])
        run = 0
        for acc in pattern:
            if not acc:
                break
            run += 1
        total += prob * run
    return total


def affine(G, a, c):
    return [0.0] + [a + c * d for d in range(1, G + 1)]


def rand_q(rng, G):
    kind = rng.integers(3)
    if kind == 0:
        return list(rng.random(G))
    if kind == 1:
        return list(rng.beta(8, 2, G) * 0.92 ** np.arange(1, G + 1))
    return list(np.round(rng.random(G), 1))  # coarse values: many exact ties


def test_constant_confidence_closed_form():
    for r in (0.3, 0.9, 0.97):
        N = S.expected_accepted([r] * 24)
        for d in range(1, 25):
            assert N[d - 1] == pytest.approx(r * (1 - r ** d) / (1 - r), rel=1e-13)
        Nb = S.expected_accepted([r] * 24, bonus=True)
        assert Nb[-1] == pytest.approx(1 + N[-1], rel=1e-15)


def test_expected_accepted_brute_force():
    rng = np.random.default_rng(0)
    for _ in range(40):
        G = int(rng.integers(1, 9))
        q = list(rng.random(G))
        N = S.expected_accepted(q)
        for d in range(1, G + 1):
            assert N[d - 1] == pytest.approx(brute_expected_accepted(q, d), rel=1e-12, abs=1e-15)


def test_exhaustive_brute_force():
    """Exhaustive optimum vs an argmax computed from the enumerated expectation."""
    rng = np.random.default_rng(1)
    for _ in range(60):
        G = int(rng.integers(1, 8))
        q = list(rng.random(G))
        cost = [0.0] + list(np.cumsum(rng.random(G) + 0.01) + rng.random())
        d_max = int(rng.integers(1, G + 1))
        f = [brute_expected_accepted(q, d) / cost[d] for d in range(1, d_max + 1)]
        best = max(f)
        cands = [d + 1 for d, v in enumerate(f) if v >= best * (1 - 1e-12)]
        got = S.select_exhaustive(q, cost, d_max)
        assert got in cands
        if len(cands) == 1:
            assert got == cands[0]


def test_thm32_mediant_equivalence():
    """Thm. 3.2: extending d -> d' improves f iff the appended segment's gain/cost exceeds
    the current average; truncating improves f iff the removed suffix's ratio is lower."""
    rng = np.random.default_rng(2)
    for _ in range(200):
        G = 16
        q = rand_q(rng, G)
        cost = [0.0] + list(np.cumsum(rng.random(G) + 0.01) + rng.random())
        N = S.expected_accepted(q)
        f = S.objective(q, cost)
        for d in range(1, G + 1):
            for d2 in range(1, G + 1):
                if d2 == d:
                    continue
                lo, hi = min(d, d2), max(d, d2)
                seg = (N[hi - 1] - N[lo - 1]) / (cost[hi] - cost[lo])
                avg = N[d - 1] / cost[d]
                if abs(seg - avg) <= 1e-9 * max(abs(avg), 1e-300) or abs(f[d2 - 1] - f[d - 1]) <= 1e-12 * f[d - 1]:
                    continue
                improves = f[d2 - 1] > f[d - 1]
                assert improves == (seg > avg if d2 > d else seg < avg)


def test_thm35_unimodality_criterion():
    """Thm. 3.5 with a constant marginal cost c: f(d+1) > f(d)  <=>  P_{d+1} > c f(d)."""
    rng = np.random.default_rng(3)
    for _ in range(300):
        G = 24
        q = rand_q(rng, G)
        a, c = float(rng.random() * 3 + 0.01), float(rng.random() + 0.01)
        cost = affine(G, a, c)
        P = S.prefix_products(q)
        f = S.objective(q, cost)
        for d in range(1, G):
            lhs = f[d] - f[d - 1]
            rhs = P[d] - c * f[d - 1]
            if abs(lhs) < 1e-12 * max(f[d - 1], 1e-300) or abs(rhs) < 1e-12 * max(P[d], 1e-300):
                continue
            assert (lhs > 0) == (rhs > 0)


@pytest.mark.parametrize("bonus", [False, True])
def test_thm36_marginal_converges_to_optimum(bonus):
    """Thm. 3.6: with q in [0,1] and a convex cost table, iterated beneficial adjustments from
    any start reach the exhaustive optimum, f increasing along the way, in |d0 - d*| steps."""
    rng = np.random.default_rng(4)
    for t in range(400):
        G = int(rng.integers(1, 33))
        q = rand_q(rng, G)
        if t % 2:
            cost = affine(G, float(rng.random() * 2 + 0.01), float(rng.random() * 0.2 + 1e-3))
        else:  # convex: non-decreasing increments
            inc = np.sort(rng.random(G) + 1e-3)
            cost = [0.0] + list(np.cumsum(inc) + rng.random() * 2 + 0.01)
        d_max = int(rng.integers(1, G + 1))
        best = S.select_exhaustive(q, cost, d_max, bonus)
        f = S.objective(q, cost, bonus)
        for d0 in range(1, d_max + 1):
            d, steps = S.select_marginal(q, cost, d0, d_max, bonus)
            assert d == best, (q, cost, d0)
            assert steps == abs(d0 - best)
        # trajectory values never decrease (strictly increase on extensions)
        d = 1
        while d < best:
            assert f[d] > f[d - 1]
            d += 1


def test_marginal_nonconvex_can_stop_early():
    """A step in the cost table (as at a tile boundary) breaks the hypothesis of Thm. 3.5:
    the one-step walk can stop at a local maximum below the exhaustive optimum."""
    G = 16
    q = [0.97] * G
    cost = [0.0] + [1 + 0.02 * d + (0.5 if d > 2 else 0.0) for d in range(1, G + 1)]
    assert S.select_exhaustive(q, cost, G) == 16
    assert S.select_marginal(q, cost, 1, G)[0] == 2


def test_alg1_eps_is_floor_of_positionwise_bound():
    """eps* = min_i floor(alpha * S_i + i) with S_i the expected number of further accepted
    drafts from position i on (brute-force enumeration), as in Algorithm 1."""
    rng = np.random.default_rng(5)
    for _ in range(60):
        d = int(rng.integers(1, 8))
        q = list(rng.random(d))
        alpha = float(rng.choice([1.8, 2.0, 2.2, 0.7, 3.1]))
        want = min(math.floor(alpha * brute_expected_accepted(q, d, start=i) + i) for i in range(1, d + 1))
        assert S.eps_star(q, d, alpha) == want


def test_alg1_invariants():
    rng = np.random.default_rng(6)
    for _ in range(500):
        G = int(rng.integers(2, 33))
        q = rand_q(rng, G)
        d_max = int(rng.integers(1, G + 1))
        n = int(rng.integers(1, G + 1))
        alpha = float(rng.choice([1.8, 2.0, 2.2, 0.5, 5.0]))
        trace = []
        d, blocks = S.select_alg1(q, d_max, alpha, n, trace)
        assert 1 <= d <= d_max
        d_peak = max([min(n, d_max)] + [min(e, d_max) for (d0, e, _b) in trace if e > d0])
        assert blocks == max(1, math.ceil(d_peak / n))
        if trace and trace[-1][1] <= trace[-1][0]:       # ended on the single rollback
            assert d == trace[-1][1]
        # every extension step satisfied eps* > d and moved to min(eps*, d_max)
        for (d0, e, _), nxt in zip(trace, trace[1:]):
            assert e > d0 and nxt[0] == min(e, d_max)


def test_golden_special_cases():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        q, G = c["q"], len(c["q"])
        cost = affine(G, c["cost"]["a"], c["cost"]["c"])
        exp = c["expect"]
        if "exhaustive" in exp:
            assert S.select_exhaustive(q, cost, c["d_max"]) == exp["exhaustive"], c["name"]
        if "marginal_any_start" in exp:
            for d0 in range(1, c["d_max"] + 1):
                assert S.select_marginal(q, cost, d0, c["d_max"])[0] == exp["marginal_any_start"], c["name"]
        trace = []
        d, blocks = S.select_alg1(q, c["d_max"], c["alpha"], c["n"], trace)
        assert [d, blocks] == exp["alg1"], c["name"]
        if "alg1_trace" in exp:
            assert [list(t) for t in trace] == exp["alg1_trace"], c["name"]


def test_select_dispatch_and_batch():
    q = [[0.9, 0.8, 0.5, 0.1], [0.0, 0.0, 0.0, 0.0]]
    cost = affine(4, 1.0, 0.05)
    g, a = S.select_batch(S.SEL_EXHAUSTIVE, q, cost, 1, 4, 2.0, 2)
    assert g[1] == 1 and a == [0, 0]
    g2, _ = S.select_batch(S.SEL_MARGINAL, q, cost, 4, 4, 2.0, 2)
    assert g2 == g


def test_alg1_blocks_on_demand_ends_where_the_full_rule_ends():
    """Algorithm 1 drafts a new block only when the budget of drafted but unused tokens goes
    negative.  Run with the first block only, then again with the blocks each call asks for,
    the rule never reads a confidence that was not drafted (q is cut to the drafted blocks)
    and ends with the length and block count of the rule over all G confidences, after at
    most ceil(d_max / n) calls."""
    rng = np.random.default_rng(16)
    for _ in range(600):
        G = int(rng.integers(1, 41))
        q = rand_q(rng, G)
        d_max = int(rng.integers(1, G + 1))
        n = int(rng.integers(1, G + 1))
        alpha = float(rng.choice([1.8, 2.0, 2.2, 0.5, 5.0]))
        want = S.select_alg1(q, d_max, alpha, n)
        k, calls = 1, 0
        while True:
            calls += 1
            g, blocks = S.select_alg1(q[:k * n], d_max, alpha, n, drafted=k)
            if g:
                break
            assert blocks > k          # a request is always for more than is drafted
            k = blocks
        assert (g, blocks) == want
        assert calls <= -(-d_max // n)


def test_alg1_blocks_on_demand_golden_traces():
    """With one block drafted, the rule stops at the first length of the golden trace that
    runs past the block and asks for ceil(d / n) blocks; if the trace never leaves the first
    block the answer is the golden one."""
    for c in json.load(open(GOLDEN))["cases"]:
        exp = c["expect"]
        if "alg1_trace" not in exp:
            continue
        n, d_max = c["n"], c["d_max"]
        lengths = [t[0] for t in exp["alg1_trace"]]
        last = exp["alg1_trace"][-1]
        if last[1] > last[0]:          # ended by reaching d_max: that length is reached too
            lengths.append(min(last[1], d_max))
        past = [d for d in lengths if d > n]
        g, blocks = S.select_alg1(c["q"][:n], d_max, c["alpha"], n, drafted=1)
        if past:
            assert (g, blocks) == (0, -(-past[0] // n)), c["name"]
        else:
            assert [g, blocks] == exp["alg1"], c["name"]
