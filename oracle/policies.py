"""Baseline speculative-length policies (oracle).  Test infrastructure only.

Paper: LibraSpec, Sec. 4.1 (baselines) and Appendix B (baseline details).  The
comparison experiments run, besides LibraSpec, a static length (one gamma for every
round, swept over a range: nothing to compute) and the dynamic rule of Gemma 4's multi-token
prediction adapted to the diffusion drafter ("G4-style"): after a round in which
every drafted token was accepted the next round drafts two more, after a round
with at least one rejection one fewer.

The paper prints no trajectory of the rule, so it is parity unpinned by a printed example;
the tests pin it by the closed forms of the stated rule's trajectories and by its link to the
acceptance oracle's count of accepted drafts.

Readings where the paper is silent (each listed in the design notes):
* "every drafted token accepted" means a == gamma, where a counts the accepted
  drafts (the bonus token is not a draft); a round of gamma = 0 has no rejection;
* the rule states no bounds: the result is clamped to [d_min, d_max];
* a round that failed (status not OK) carries no outcome: the length is kept;
* a record outside 0 <= gamma < max_seq_rows, or with a outside [0, gamma] on an OK
  round, is unusable: the length restarts at d_min and the record is flagged.
"""

OK, INVALID_ARG = 0, -1


def g4_next(gamma, a, d_min, d_max, ok=True, max_seq_rows=64):
    """(next length, flag) for one sequence."""
    valid = 0 <= gamma < max_seq_rows and (not ok or 0 <= a <= gamma)
    if not valid:
        raw = d_min
    elif not ok:
        raw = gamma
    elif a == gamma:  # no draft rejected
        raw = gamma + 2
    else:  # at least one rejection
        raw = gamma - 1
    return min(max(raw, d_min), d_max), (OK if valid else INVALID_ARG)


def g4_next_batch(gamma, accept_len, d_min, d_max, status=None):
    """Per-sequence next lengths, flags and the next verify block's row offsets
    (root plus gamma_next drafts per sequence)."""
    nxt, err, off = [], [], [0]
    for b in range(len(gamma)):
        ok = status is None or int(status[b]) == OK
        g, e = g4_next(int(gamma[b]), int(accept_len[b]), d_min, d_max, ok)
        nxt.append(g)
        err.append(e)
        off.append(off[-1] + g + 1)
    return nxt, err, off

