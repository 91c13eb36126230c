"""GPU length selector vs the oracle, bit for bit (binary64, no fused multiply-add)."""
import numpy as np
import pytest
import torch

from oracle import selector as S
from paper_2608_08721_amd import lsv
from tests.lsv_testing import note

pytestmark = pytest.mark.gpu


def gpu_select(mode, conf, cost, d_init, d_max, alpha, n, flags):
    B, G = conf.shape
    c = torch.tensor(conf, dtype=torch.float32, device="cuda")
    co = torch.tensor(cost, dtype=torch.float64, device="cuda") if cost is not None else None
    g = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    aux = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    st = torch.full((B,), 99, dtype=torch.int32, device="cuda")
    ro = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda") if B <= 64 else None
    lsv.lsv_select_length(mode, B, G, c, co, d_init, d_max, alpha, n, flags, g, aux, ro, st)
    torch.cuda.synchronize()
    g_np = g.cpu().numpy()
    if ro is not None:  # the verify row layout: root plus gamma drafts per sequence
        assert ro.cpu().numpy().tolist() == [0] + list(np.cumsum(g_np + 1))
    return g_np, aux.cpu().numpy(), st.cpu().numpy()


def random_conf(rng, B, G):
    kind = rng.integers(5)
    if kind == 0:
        x = rng.random((B, G))
    elif kind == 1:
        x = rng.beta(8, 2, (B, G)) * 0.92 ** np.arange(1, G + 1)
    elif kind == 2:
        x = np.round(rng.random((B, G)), 1)          # exact ties
    elif kind == 3:
        x = rng.choice([0.0, 1.0, 0.5, 0.9], size=(B, G))
    else:
        x = 1.0 - rng.random((B, G)) ** 6
    return x.astype(np.float32)


def random_cost(rng, G):
    kind = rng.integers(4)
    d = np.arange(G + 1, dtype=np.float64)
    if kind == 0:
        c = rng.random() * 2 + 0.01 + (rng.random() * 0.2) * d
    elif kind == 1:
        c = np.concatenate([[0.0], np.cumsum(np.sort(rng.random(G)) + 1e-3)]) + rng.random()
    elif kind == 2:   # tile-step table
        c = 1.0 + 0.02 * d + 0.5 * (d > rng.integers(1, G + 1))
    else:
        c = rng.random(G + 1) + 0.05
    c[0] = 0.0
    return c


def test_selector_parity_random():
    rng = np.random.default_rng(123)
    n_cases = 0
    for trial in range(90):
        G = int(rng.choice([1, 2, 3, 7, 16, 32, 64]))
        B = 64 if trial % 4 else 97   # beyond one wave: no row offsets
        conf = random_conf(rng, B, G)
        cost = random_cost(rng, G)
        for mode in (S.SEL_MARGINAL, S.SEL_EXHAUSTIVE, S.SEL_ALG1):
            flags = int(rng.integers(2)) if mode != S.SEL_ALG1 else 0
            d_max = int(rng.integers(1, G + 1))
            d_init = int(rng.integers(1, G + 1))
            alpha = float(rng.choice([1.8, 2.0, 2.2, 0.5, 3.7]))
            n = int(rng.integers(1, G + 1))
            g, aux, st = gpu_select(mode, conf, cost if mode != S.SEL_ALG1 else None, d_init, d_max, alpha, n, flags)
            want_g, want_a = S.select_batch(mode, conf, list(cost), d_init, d_max, alpha, n, flags)
            assert np.all(st == 0)
            assert list(g) == want_g, (trial, mode)
            assert list(aux) == want_a, (trial, mode)
            n_cases += B
    note(f"selector parity: {n_cases} sequences bit-exact")


def test_selector_rejects_bad_confidence_and_cost():
    conf = np.full((3, 8), 0.5, np.float32)
    conf[1, 3] = np.nan
    conf[2, 0] = 1.5
    cost = np.linspace(0, 1.4, 9)
    g, aux, st = gpu_select(S.SEL_EXHAUSTIVE, conf, cost, 1, 8, 2.0, 4, 0)
    assert list(st) == [0, lsv.LSV_ERR_INVALID_ARG, lsv.LSV_ERR_INVALID_ARG]
    assert g[1] == 0 and g[2] == 0 and g[0] == S.select_exhaustive([0.5] * 8, list(cost), 8)
    bad = cost.copy()
    bad[5] = -1.0
    g, aux, st = gpu_select(S.SEL_MARGINAL, conf[:1], bad, 1, 8, 2.0, 4, 0)
    assert st[0] == lsv.LSV_ERR_INVALID_ARG
    g, aux, st = gpu_select(S.SEL_MARGINAL, conf[:1], bad, 1, 4, 2.0, 4, 0)  # cost[5] beyond d_max: unused
    assert st[0] == 0


def test_selector_paper_hyperparameters():
    """The paper's settings: alpha 2.0 with d_max 60 and initial length 10, alpha 2.2 with d_max 24 and block 16
    (Sec. 4, implementation details)."""
    rng = np.random.default_rng(7)
    for alpha, d_max, n in ((2.0, 60, 10), (2.2, 24, 16)):
        G = 64 if d_max > 32 else 32
        conf = (rng.beta(8, 2, (64, G)) * 0.97 ** np.arange(1, G + 1)).astype(np.float32)
        g, aux, st = gpu_select(S.SEL_ALG1, conf, None, 1, d_max, alpha, n, 0)
        want = S.select_batch(S.SEL_ALG1, conf, None, 1, d_max, alpha, n)
        assert list(g) == want[0] and list(aux) == want[1]


def gpu_joint(conf, cost, d_max, flags):
    B, G = conf.shape
    c = torch.tensor(conf, dtype=torch.float32, device="cuda")
    co = torch.tensor(cost, dtype=torch.float64, device="cuda")
    g = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    tot = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    ro = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda")
    st = torch.full((B,), 99, dtype=torch.int32, device="cuda")
    lsv.lsv_select_joint(B, G, c, co, d_max, flags, g, tot, ro, st)
    torch.cuda.synchronize()
    return g.cpu().numpy(), int(tot.cpu()[0]), ro.cpu().numpy(), st.cpu().numpy()


@pytest.mark.parametrize("B,G", [(1, 16), (3, 5), (8, 16), (17, 33), (64, 64)])
def test_joint_selector_parity(B, G):
    """Joint batched selection vs the oracle, bit for bit: gamma, the total and the row layout."""
    rng = np.random.default_rng(B * 100 + G)
    for trial in range(4):
        conf = random_conf(rng, B, G)
        d_max = G if trial % 2 == 0 else int(rng.integers(1, G + 1))
        R = np.arange(B * d_max + 1)
        base, slope = rng.uniform(0.5, 2.0), rng.uniform(0.0, 0.05)
        cost = base + slope * R + np.where(R > B * d_max * rng.uniform(0.3, 0.9), rng.uniform(0, 1), 0.0)
        if trial == 3:
            cost = base + slope * np.sqrt(R)  # concave: many drafts in total
        flags = S.FLAG_BONUS if trial % 2 else 0
        g, tot, ro, st = gpu_joint(conf, cost, d_max, flags)
        want_g, want_R = S.select_joint(conf, cost, d_max, bool(flags))
        assert g.tolist() == want_g and tot == want_R and np.all(st == 0)
        assert ro.tolist() == [0] + list(np.cumsum(np.array(want_g) + 1))
    note(f"  joint B={B} G={G}: 4 cases bit-exact (last total {tot})")


def test_joint_selector_rejects_bad_input():
    conf = np.full((3, 4), 0.5, np.float32)
    conf[1, 2] = np.nan
    cost = np.ones(3 * 4 + 1)
    g, tot, ro, st = gpu_joint(conf, cost, 4, 0)
    assert g.tolist() == [0, 0, 0] and tot == 0 and np.all(st == lsv.LSV_ERR_INVALID_ARG)
    assert ro.tolist() == [0, 1, 2, 3]
    conf[1, 2] = 0.5
    cost[7] = 0.0  # a needed entry (R in [3, 12])
    g, tot, ro, st = gpu_joint(conf, cost, 4, 0)
    assert np.all(st == lsv.LSV_ERR_INVALID_ARG)
    cost[7] = 1.0
    cost[1] = np.nan  # below the smallest total: never read
    g, tot, ro, st = gpu_joint(conf, cost, 4, 0)
    assert np.all(st == 0) and tot == 12


def test_alg1_blocks_on_demand_parity():
    """LSV_SEL_DRAFTED: d_aux brings the blocks drafted so far; gamma (0 = more blocks
    needed) and the blocks out match the oracle bit for bit, and iterating the requests on
    the device ends on the all-confidences answer."""
    rng = np.random.default_rng(77)
    for trial in range(40):
        B = int(rng.integers(1, 97))
        G = int(rng.integers(1, 65))
        conf = random_conf(rng, B, G)
        d_max = int(rng.integers(1, G + 1))
        n = int(rng.integers(1, min(G, 16) + 1))
        alpha = float(rng.choice([1.8, 2.0, 2.2, 0.5, 4.0]))
        drafted = rng.integers(1, -(-G // n) + 2, size=B).astype(np.int32)
        poisoned = conf.copy()   # confidences not drafted yet: never read
        for b in range(B):
            poisoned[b, min(int(drafted[b]) * n, G):] = np.nan
        c = torch.tensor(poisoned, device="cuda")
        g = torch.full((B,), -7, dtype=torch.int32, device="cuda")
        aux = torch.tensor(drafted, device="cuda")
        st = torch.full((B,), 99, dtype=torch.int32, device="cuda")
        lsv.lsv_select_length(S.SEL_ALG1, B, G, c, None, 1, d_max, alpha, n, lsv.LSV_SEL_DRAFTED, g, aux, None, st)
        torch.cuda.synchronize()
        assert (st.cpu().numpy() == 0).all()
        for b in range(B):
            want = S.select_alg1([float(v) for v in conf[b]], d_max, alpha, n, drafted=int(drafted[b]))
            assert (int(g[b]), int(aux[b])) == want, (trial, b)
        # the request loop on the device: first block only, then what each call asks for
        have = torch.ones(B, dtype=torch.int32, device="cuda")
        c = torch.tensor(conf, device="cuda")
        aux.fill_(1)
        have.fill_(1)
        for _ in range(-(-d_max // n)):
            lsv.lsv_select_length(S.SEL_ALG1, B, G, c, None, 1, d_max, alpha, n, lsv.LSV_SEL_DRAFTED, g, aux, None, st)
            torch.maximum(have, aux, out=have)
            aux.copy_(have)
        g_eager, a_eager, _ = gpu_select(S.SEL_ALG1, conf, None, 1, d_max, alpha, n, 0)
        lsv.lsv_select_length(S.SEL_ALG1, B, G, c, None, 1, d_max, alpha, n, lsv.LSV_SEL_DRAFTED, g, aux, None, st)
        torch.cuda.synchronize()
        assert np.array_equal(g.cpu().numpy(), g_eager) and np.array_equal(aux.cpu().numpy(), a_eager)
    note("  ALG1 with blocks on demand: 40 batches bit-exact, request loops end on the full-G answer")


def test_alg1_blocks_on_demand_rejects_bad_input():
    c = torch.full((2, 8), 0.9, device="cuda")
    g = torch.zeros(2, dtype=torch.int32, device="cuda")
    st = torch.zeros(2, dtype=torch.int32, device="cuda")
    with pytest.raises(lsv.LsvError):   # needs d_aux
        lsv.lsv_select_length(S.SEL_ALG1, 2, 8, c, None, 1, 8, 2.0, 4, lsv.LSV_SEL_DRAFTED, g, None, None, st)
    aux = torch.tensor([0, 2], dtype=torch.int32, device="cuda")
    lsv.lsv_select_length(S.SEL_ALG1, 2, 8, c, None, 1, 8, 2.0, 4, lsv.LSV_SEL_DRAFTED, g, aux, None, st)
    torch.cuda.synchronize()
    assert st.cpu().tolist() == [lsv.LSV_ERR_INVALID_ARG, 0] and int(g[0]) == 0
