"""Pins for the oracle's Philox4x64-10: numpy's Philox bit generator (the same published
algorithm, an independent implementation) is the known-answer source."""
import numpy as np

from oracle import philox as P


def numpy_blocks(key, start_counter, n_blocks):
    """numpy.random.Philox increments the 256-bit counter before each block, so its k-th
    block (k = 0, 1, ...) is Philox(counter = start + k + 1, key)."""
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(start_counter, dtype=np.uint64))
    raw = bg.random_raw(4 * n_blocks)
    return [tuple(int(x) for x in raw[4 * k:4 * k + 4]) for k in range(n_blocks)]


def test_scalar_matches_numpy_philox():
    for key in [(0, 0), (7, 0), (2**64 - 1, 12345), (0xDEADBEEF, 2**63)]:
        for start in [(0, 0, 0, 0), (5, 9, 2**40, 3)]:
            blocks = numpy_blocks(key, start, 3)
            for k, blk in enumerate(blocks):
                ctr = list(start)
                ctr[0] += k + 1
                assert P.philox4x64(ctr, key) == blk


def test_vectorised_matches_scalar():
    rng = np.random.default_rng(0)
    c = rng.integers(0, 2**63, size=(4, 50), dtype=np.uint64) * np.uint64(2) + np.uint64(1)
    k = rng.integers(0, 2**63, size=(2, 50), dtype=np.uint64)
    out = P.philox4x64_np(c[0], c[1], c[2], c[3], k[0], k[1])
    for i in range(50):
        want = P.philox4x64([int(c[j, i]) for j in range(4)], (int(k[0, i]), int(k[1, i])))
        assert tuple(int(out[j][i]) for j in range(4)) == want


def test_unit_interval_and_layout():
    assert P.to_unit(0) == 2.0 ** -53
    assert P.to_unit(2**64 - 1) == 1.0 - 2.0 ** -53 < 1.0
    u = P.sample_uniforms(3, 7, 2, 5, 11)
    for x in range(11):
        w = P.philox4x64((x >> 2, 5 | (2 << 32), 7, 0), (3, P.STREAM_SAMPLE))[x & 3]
        assert u[x] == P.to_unit(w)
    assert P.accept_uniform(3, 7, 2, 4) == P.to_unit(P.philox4x64((0, 4 | (2 << 32), 7, 0), (3, P.STREAM_ACCEPT))[0])
    big = P.sample_uniforms(1, 0, 0, 0, 200000)
    assert abs(big.mean() - 0.5) < 0.005 and 0 < big.min() and big.max() < 1
