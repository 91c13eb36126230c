"""Speculative-length selection (oracle).  Test infrastructure only.

Paper: LibraSpec, Sec. 3.2-3.4, Appendix A.
All arithmetic is IEEE binary64 with one rounding per operation, in the order
written (Python floats never fuse a multiply into an add), so the GPU selector --
compiled with FMA contraction disabled -- must agree bit for bit.

Notation (paper): q_k drafter confidence of draft k (k = 1..G), standing in for
the target acceptance probability p_k (Assumption 3.7); d = speculative length;
T(d) = verification cost of length d (``cost[d]``, cost[0] unused).

* P_j = prod_{k<=j} q_k is the probability that drafts 1..j are all accepted
  (prefix acceptance, proof of Thm. 3.3 with i = 1);
* N(d) = E[tau_d] = sum_{j<=d} P_j (linearity of expectation, same proof);
* f(d) = N(d) / T(d) is the simplified speedup objective of Eq. 2 up to the
  constant per-token target latency.

Readings where the paper is silent (each listed in the design notes):
* the bonus token is excluded from E[tau_d] as in the paper's formula; flag
  ``BONUS`` adds the +1 of the always-emitted correction/bonus token;
* EXHAUSTIVE returns the smallest maximiser of f over 1..d_max;
* MARGINAL moves one position at a time: extend while f(d+1) > f(d) strictly
  (Def. 3.1 requires a strict gain), else contract while f(d-1) >= f(d);
* ALG1 follows Algorithm 1: eps_i = floor(alpha * S_i + i) with S_i summed up to
  the *current* d, eps* = min_i eps_i; the length climbs to min(eps*, d_max) while
  eps* > d and settles on eps* at the first d where eps* <= d (the single rollback);
  the blocks counted are those the drafter needs to cover the highest length reached.
"""
import math

SEL_MARGINAL, SEL_EXHAUSTIVE, SEL_ALG1 = 0, 1, 2
FLAG_BONUS = 1


def prefix_products(q):
    """[P_1, ..., P_G] with P_j = P_{j-1} * q_j, P_0 = 1 (left-to-right products)."""
    out, p = [], 1.0
    for x in q:
        p = p * float(x)
        out.append(p)
    return out


def expected_accepted(q, bonus=False):
    """[N(1), ..., N(G)], N(d) = [bonus] + sum_{j<=d} P_j, accumulated left to right."""
    out, n = [], (1.0 if bonus else 0.0)
    for pj in prefix_products(q):
        n = n + pj
        out.append(n)
    return out


def objective(q, cost, bonus=False):
    """[f(1), ..., f(G)], f(d) = N(d) / cost[d]."""
    N = expected_accepted(q, bonus)
    return [N[d - 1] / float(cost[d]) for d in range(1, len(q) + 1)]


def select_exhaustive(q, cost, d_max, bonus=False):
    """Smallest d in [1, d_max] maximising f(d) (the exhaustive-search optimum)."""
    f = objective(q, cost, bonus)
    best = 1
    for d in range(2, d_max + 1):
        if f[d - 1] > f[best - 1]:
            best = d
    return best


def select_marginal(q, cost, d_init, d_max, bonus=False):
    """Iterated single beneficial adjustments of size one (Def. 3.1, Thm. 3.5/3.6).

    Returns (d, steps)."""
    f = objective(q, cost, bonus)
    d = min(max(d_init, 1), d_max)
    steps = 0
    while True:
        if d < d_max and f[d] > f[d - 1]:        # f(d+1) > f(d): extension is beneficial
            d += 1
        elif d > 1 and f[d - 2] >= f[d - 1]:     # f(d-1) >= f(d): truncation does not lose
            d -= 1
        else:
            break
        steps += 1
    return d, steps


def suffix_gain(q, i, d):
    """S_i = sum_{j=i}^{d} prod_{k=i}^{j} q_k (expected extra accepted drafts from
    position i on, given drafts before i were accepted; proof of Thm. 3.3)."""
    s, p = 0.0, 1.0
    for j in range(i, d + 1):
        p = p * float(q[j - 1])
        s = s + p
    return s


def eps_star(q, d, alpha):
    """min_{i=1..d} floor(alpha * S_i + i)  (Algorithm 1, position-wise bounds)."""
    best = None
    for i in range(1, d + 1):
        e = math.floor(alpha * suffix_gain(q, i, d) + i)
        best = e if best is None or e < best else best
    return best


def select_alg1(q, d_max, alpha, n, trace=None, drafted=None):
    """Algorithm 1 (LibraSpec), restated.  q holds the confidences of all G drafted tokens;
    d_max <= G.

    eps*(d) = min_i eps_i over the positions of the current length d is the longest length
    that every position-wise bound (Thm. 3.3) admits.  The length starts at the drafter's
    block size n and climbs along d -> min(eps*(d), d_max) while that raises it; at the first
    d where it does not, the length settles on eps*(d) itself -- the same length or a single
    step back, after which the rule stops.  Reaching d_max also stops it.

    The budget of Algorithm 1 counts drafted tokens not yet used: new blocks of n are drafted
    only when an extension runs past what is drafted, so the drafter has produced
    ceil(d_peak / n) blocks (at least one) when the highest length reached is d_peak, and the
    budget at length d is (-d) mod n.

    Returns (d, blocks).  ``trace`` (a list) receives (d, eps*(d), budget) for every
    evaluation of eps*.

    drafted (blocks on demand): only the first drafted * n confidences exist (q may be
    shorter).  When the length reaches past them -- the budget of drafted but unused tokens
    goes negative -- the rule cannot go on: it returns (0, blocks), blocks = ceil(d / n) being
    what the drafter must have produced before the rule is run again.  Run again with more
    blocks it takes the same steps, so it ends where the rule over all G confidences ends."""
    avail = len(q) if drafted is None else min(drafted * n, len(q))
    d = min(n, d_max)
    settled = None
    while settled is None and d < d_max and d <= avail:
        e = eps_star(q, d, alpha)
        if trace is not None:
            trace.append((d, e, (-d) % n))
        if e > d:
            d = min(e, d_max)      # climb
        else:
            settled = e            # stay, or one step back
    blocks = max(1, -(-d // n))    # d is the highest length reached here
    if settled is None and d > avail:
        return 0, blocks           # more blocks first
    return (d if settled is None else settled), blocks


def select(mode, q, cost, d_init, d_max, alpha, n, flags=0):
    """Dispatch one sequence; returns (gamma, aux) with aux = steps (MARGINAL),
    0 (EXHAUSTIVE) or blocks (ALG1)."""
    bonus = bool(flags & FLAG_BONUS)
    if mode == SEL_MARGINAL:
        return select_marginal(q, cost, d_init, d_max, bonus)
    if mode == SEL_EXHAUSTIVE:
        return select_exhaustive(q, cost, d_max, bonus), 0
    if mode == SEL_ALG1:
        return select_alg1(q, d_max, alpha, n)
    raise ValueError(mode)


def select_batch(mode, conf, cost, d_init, d_max, alpha, n, flags=0):
    """conf: [B][G] float32 confidences; returns (gamma[B], aux[B])."""
    g, a = [], []
    for row in conf:
        x, y = select(mode, [float(v) for v in row], cost, d_init, d_max, alpha, n, flags)
        g.append(x)
        a.append(y)
    return g, a


def select_joint(conf, cost, d_max, bonus=False):
    """Joint batched selection: gamma_b in [1, d_max] maximising
        F(gamma) = sum_b N_b(gamma_b) / cost[sum_b gamma_b]
    (Eq. 2's expected-tokens-per-verify-time objective over a batch whose verify cost is
    shared; the paper states only the per-sequence rule, so this extension and its readings
    are the library's).  cost[R] is the verify cost of a batch with R drafts in total
    (R in [B, B * d_max]; lower entries unused).

    For a fixed total R the best allocation gives every sequence its first draft and then
    the R - B largest increments P_{b,j} (2 <= j <= d_max): each N_b has non-increasing
    increments (P_{b,j+1} = P_{b,j} q_{b,j+1} <= P_{b,j}), so an exchange argument makes the
    greedy choice optimal.  Ties between increments go to the smaller b, then the smaller j
    (which keeps every sequence's choice a prefix).  F is then evaluated for every R with
    N_b from ``expected_accepted`` summed over b in order, and the smallest maximising R
    wins.  Returns (gamma[B], R)."""
    B = len(conf)
    P = [prefix_products([float(v) for v in row]) for row in conf]
    N = [expected_accepted([float(v) for v in row], bonus) for row in conf]
    inc = sorted(((-P[b][j - 1], b, j) for b in range(B) for j in range(2, d_max + 1)))
    gamma = [1] * B
    best_f, best_R, best_g = None, None, None
    for R in range(B, B * d_max + 1):
        if R > B:
            _, b, j = inc[R - B - 1]
            gamma[b] = j
        s = 0.0
        for b in range(B):
            s = s + N[b][gamma[b] - 1]
        f = s / float(cost[R])
        if best_f is None or f > best_f:
            best_f, best_R, best_g = f, R, list(gamma)
    return best_g, best_R


def joint_objective(conf, cost, gamma, bonus=False):
    """F(gamma) for a given allocation (used by the brute-force pins)."""
    s = 0.0
    for row, g in zip(conf, gamma):
        s = s + expected_accepted([float(v) for v in row], bonus)[g - 1]
    return s / float(cost[sum(gamma)])
