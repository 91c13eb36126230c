"""Token plumbing between decoding rounds (oracle).  Test infrastructure only.

Paper: LibraSpec, Sec. 3.1.  A round verifies the token emitted last (the root) followed
by the round's drafts; it emits the accepted drafts and one more token (the correction
or bonus token), which is the next round's root.  With greedy acceptance the emitted
stream is the target's own greedy continuation whatever the drafts and lengths were
(the lossless property), so plain greedy decoding (``forward.greedy_continuation``) is
the reference for a whole multi-round loop.
"""

OK, INVALID_ARG = 0, -1


def pack_block(row_offsets, roots, drafts, G, max_rows, tokens):
    """Fill ``tokens`` (list, length >= max_rows) in place: row r0_b = root_b, then the
    first rows_b - 1 drafts of sequence b.  Returns the per-sequence status; a sequence
    whose rows are empty, run past max_rows or exceed G + 1 writes nothing."""
    status = []
    for b in range(len(roots)):
        r0, r1 = int(row_offsets[b]), int(row_offsets[b + 1])
        ok = r0 >= 0 and r1 > r0 and r1 <= max_rows and r1 - r0 - 1 <= G
        status.append(OK if ok else INVALID_ARG)
        if ok:
            tokens[r0] = int(roots[b])
            for k in range(1, r1 - r0):
                tokens[r0 + k] = int(drafts[b][k - 1])
    return status


def next_roots(accept_len, out_tokens, width, status, roots):
    """roots[b] = out_tokens[b][accept_len[b]] for sequences whose round succeeded."""
    out = list(roots)
    for b in range(len(out)):
        a = int(accept_len[b])
        if (status is None or int(status[b]) == OK) and 0 <= a < width:
            out[b] = int(out_tokens[b][a])
    return out
