"""Philox4x64-10 counter-based RNG (oracle).  Test infrastructure only.

Written from the published definition (J. K. Salmon, M. A. Moraes, R. O. Dror,
D. E. Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC'11): a 4-word
counter and a 2-word key; each of the 10 rounds multiplies counter words 0 and 2
by the round multipliers, mixes the high halves with the other counter words
and the key, and the key is bumped by the Weyl constants between rounds.

The sampling acceptance reads one uniform per decision:
    U = ((w >> 12) + 0.5) * 2^-52   (a 52-bit fraction; every value is exact in
    binary64 and lies strictly inside (0, 1) -- with 53 bits the top word would round to 1).
Counter layout (a reading of ours; the paper only says acceptance is lossless):
    accept test, draft v of sequence b :  key (seed, STREAM_ACCEPT),
                                          counter (0, v | b << 32, round, 0), word 0
    categorical draw over token x, row r : key (seed, STREAM_SAMPLE),
                                          counter (x >> 2, r | b << 32, round, 0), word x & 3
"""
import numpy as np

MASK64 = (1 << 64) - 1
PHILOX_M0 = 0xD2E7470EE14C6C93
PHILOX_M1 = 0xCA5A826395121157
PHILOX_W0 = 0x9E3779B97F4A7C15
PHILOX_W1 = 0xBB67AE8584CAA73B
STREAM_ACCEPT = 1
STREAM_SAMPLE = 2


def philox4x64(counter, key, rounds=10):
    """Scalar reference on Python ints: counter = (c0, c1, c2, c3), key = (k0, k1)."""
    c0, c1, c2, c3 = (int(x) & MASK64 for x in counter)
    k0, k1 = (int(x) & MASK64 for x in key)
    for _ in range(rounds):
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        hi0, lo0 = p0 >> 64, p0 & MASK64
        hi1, lo1 = p1 >> 64, p1 & MASK64
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
        k0 = (k0 + PHILOX_W0) & MASK64
        k1 = (k1 + PHILOX_W1) & MASK64
    return c0, c1, c2, c3


def _mulhilo(a, b):
    """64x64 -> (hi, lo) on uint64 numpy arrays via 32-bit limbs."""
    m32 = np.uint64(0xFFFFFFFF)
    s32 = np.uint64(32)
    a_lo, a_hi = a & m32, a >> s32
    b_lo, b_hi = b & m32, b >> s32
    ll = a_lo * b_lo
    lh = a_lo * b_hi
    hl = a_hi * b_lo
    hh = a_hi * b_hi
    mid = (ll >> s32) + (lh & m32) + (hl & m32)
    lo = (ll & m32) | ((mid & m32) << s32)
    hi = hh + (lh >> s32) + (hl >> s32) + (mid >> s32)
    return hi, lo


def philox4x64_np(c0, c1, c2, c3, k0, k1, rounds=10):
    """Vectorised Philox4x64 over uint64 arrays (broadcasting); returns 4 arrays."""
    with np.errstate(over="ignore"):
        c0, c1, c2, c3 = (np.asarray(x, dtype=np.uint64) for x in (c0, c1, c2, c3))
        k0 = np.asarray(k0, dtype=np.uint64)
        k1 = np.asarray(k1, dtype=np.uint64)
        c0, c1, c2, c3, k0, k1 = np.broadcast_arrays(c0, c1, c2, c3, k0, k1)
        c0, c1, c2, c3, k0, k1 = (x.copy() for x in (c0, c1, c2, c3, k0, k1))
        m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
        w0, w1 = np.uint64(PHILOX_W0), np.uint64(PHILOX_W1)
        for _ in range(rounds):
            hi0, lo0 = _mulhilo(c0, m0)
            hi1, lo1 = _mulhilo(c2, m1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
            k0 = k0 + w0
            k1 = k1 + w1
    return c0, c1, c2, c3


def to_unit(w):
    """Uniform in (0, 1) from the top 52 bits of a 64-bit word (scalar int or uint64 array)."""
    if isinstance(w, np.ndarray):
        return ((w >> np.uint64(12)).astype(np.float64) + 0.5) * 2.0 ** -52
    return ((int(w) >> 12) + 0.5) * 2.0 ** -52


def accept_uniform(seed, rnd, b, v):
    """Uniform for the ratio test of draft v (1-based) of sequence b in round rnd."""
    w = philox4x64((0, (v & 0xFFFFFFFF) | (b << 32), rnd, 0), (seed, STREAM_ACCEPT))[0]
    return to_unit(w)


def sample_uniforms(seed, rnd, b, r, vocab):
    """Uniforms U_x, x = 0..vocab-1, for a categorical draw from row r of sequence b."""
    x = np.arange(vocab, dtype=np.uint64)
    n_ctr = (vocab + 3) // 4
    c0 = np.arange(n_ctr, dtype=np.uint64)
    c1 = np.uint64((r & 0xFFFFFFFF) | (b << 32))
    out = philox4x64_np(c0, c1, np.uint64(rnd), np.uint64(0), np.uint64(seed), np.uint64(STREAM_SAMPLE))
    words = np.stack(out, axis=1).reshape(-1)[:vocab]
    assert words.shape == x.shape
    return to_unit(words)
