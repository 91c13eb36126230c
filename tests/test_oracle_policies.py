"""Pins of the baseline length policy oracle (Sec. 4.1; Appendix B, baseline details):
closed forms of the rule's trajectories, its step set, its clamps, and the tie between
"every draft accepted" and the acceptance oracle's accepted-draft count."""
import numpy as np
import pytest

from oracle import accept as OA
from oracle import policies as OP


@pytest.mark.parametrize("g0,d_min,d_max", [(10, 1, 60), (3, 1, 20), (1, 1, 16), (7, 4, 9)])
def test_all_accepted_rounds_climb_by_two_to_the_cap(g0, d_min, d_max):
    g = g0
    for t in range(1, 40):
        g, e = OP.g4_next(g, g, d_min, d_max)  # a == gamma: no rejection
        assert e == OP.OK and g == min(g0 + 2 * t, d_max)


@pytest.mark.parametrize("g0,d_min,d_max", [(10, 1, 60), (20, 3, 20), (5, 5, 9)])
def test_rejected_rounds_fall_by_one_to_the_floor(g0, d_min, d_max):
    g = g0
    for t in range(1, 40):
        g, e = OP.g4_next(g, 0, d_min, d_max)  # the first draft rejected (a = 0 < gamma)
        assert e == OP.OK and g == max(g0 - t, d_min)


def test_steps_are_plus_two_or_minus_one_inside_the_bounds():
    rng = np.random.default_rng(5)
    for _ in range(2000):
        g = int(rng.integers(0, 64))
        a = int(rng.integers(0, g + 1))
        nxt, e = OP.g4_next(g, a, 1, 63)
        assert e == OP.OK and 1 <= nxt <= 63
        if 1 < g < 61:
            assert nxt - g == (2 if a == g else -1)


def test_failed_rounds_and_bad_records():
    assert OP.g4_next(9, 3, 1, 16, ok=False) == (9, OP.OK)  # no outcome: kept
    assert OP.g4_next(30, 3, 1, 16, ok=False) == (16, OP.OK)  # kept, then clamped
    assert OP.g4_next(9, 10, 2, 16) == (2, OP.INVALID_ARG)  # more accepted than drafted
    assert OP.g4_next(-1, 0, 2, 16) == (2, OP.INVALID_ARG)
    assert OP.g4_next(64, 64, 2, 16) == (2, OP.INVALID_ARG)  # past the one-wave block limit
    assert OP.g4_next(0, 0, 1, 16) == (2, OP.OK)  # no drafts, no rejection


def test_batch_row_offsets():
    nxt, err, off = OP.g4_next_batch([4, 4, 0, 12], [4, 1, 0, 12], 1, 13, status=[0, 0, 0, -5])
    assert nxt == [6, 3, 2, 12] and err == [0] * 4
    assert off == [0, 7, 11, 14, 27]


def _greedy_block(rng, V, g, a):
    """One sequence's verify logits and tokens with exactly a leading drafts matching the
    row argmax (draft a+1, when it exists, does not)."""
    logits = rng.normal(size=(g + 1, V))
    toks = rng.integers(0, V, size=g + 1)
    for v in range(1, g + 1):
        best = int(np.argmax(logits[v - 1]))
        toks[v] = best if v <= a else (best + 1) % V
    return logits, toks


def test_all_accepted_means_the_acceptance_count_equals_gamma():
    rng = np.random.default_rng(11)
    V = 50
    for g, a in [(5, 5), (5, 4), (5, 0), (1, 1), (0, 0), (12, 11)]:
        logits, toks = _greedy_block(rng, V, g, a)
        res = OA.accept_greedy(logits, [0, g + 1], toks, out_width=g + 1)
        assert res["accept_len"][0] == a
        nxt, _ = OP.g4_next(g, int(res["accept_len"][0]), 1, 60)
        assert nxt == (g + 2 if a == g else max(g - 1, 1))
