"""Pins of the joint batched selector oracle (the batch form of Eq. 2's objective):
brute force over every allocation on small batches, its batch-1 reduction to the exhaustive
rule, and the prefix structure of the greedy allocation."""
import itertools

import numpy as np
import pytest

from oracle import selector as S


def _case(rng, B, G, kind):
    if kind == 0:
        conf = rng.random((B, G))
    elif kind == 1:
        conf = np.round(rng.random((B, G)), 1)  # exact ties between increments
    else:
        conf = rng.beta(8, 2, (B, G)) * 0.92 ** np.arange(1, G + 1)
    conf = conf.astype(np.float32)
    base = rng.uniform(0.5, 2.0)
    slope = rng.uniform(0.0, 0.2)
    cost = np.array([base + slope * r + (0.3 if r > B * G // 2 else 0.0) for r in range(B * G + 1)])
    return conf, cost


@pytest.mark.parametrize("B,G", [(1, 6), (2, 5), (3, 4), (4, 3)])
def test_joint_matches_brute_force(B, G):
    rng = np.random.default_rng(B * 10 + G)
    for trial in range(30):
        conf, cost = _case(rng, B, G, trial % 3)
        bonus = trial % 2 == 1
        g, R = S.select_joint(conf, cost, G, bonus)
        assert sum(g) == R and all(1 <= x <= G for x in g)
        best = max(S.joint_objective(conf, cost, list(v), bonus)
                   for v in itertools.product(range(1, G + 1), repeat=B))
        got = S.joint_objective(conf, cost, g, bonus)
        assert got >= best * (1 - 1e-12), (conf, cost, g)


def test_batch_of_one_is_the_exhaustive_rule():
    rng = np.random.default_rng(4)
    for trial in range(200):
        G = int(rng.integers(1, 20))
        conf, cost = _case(rng, 1, G, trial % 3)
        bonus = trial % 2 == 0
        g, R = S.select_joint(conf, cost, G, bonus)
        assert g == [S.select_exhaustive([float(v) for v in conf[0]], cost, G, bonus)]


def test_allocation_takes_the_largest_increments():
    # q = 1 everywhere in sequence 0 (every increment is 1) and 0.5 in sequence 1
    conf = np.array([[1.0] * 4, [0.5] * 4], np.float32)
    cost = np.array([1.0] * 9)  # flat cost: more drafts never hurt, all of them are taken
    g, R = S.select_joint(conf, cost, 4)
    assert g == [4, 4] and R == 8
    cost = np.array([1.0] * 5 + [1e9] * 4)  # at most 4 drafts in total
    g, R = S.select_joint(conf, cost, 4)
    assert g == [3, 1] and R == 4  # sequence 0's increments (1.0) beat sequence 1's second (0.25)
