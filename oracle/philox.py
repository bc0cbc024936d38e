"""Philox4x32-10 and the noise transforms of the GSQ step.  Test infrastructure only.

The paper draws g ~ Gumbel(0, 1) for every logit at every forward pass and
resamples it on each pass (Alg. 1; §3.3 "Gradient accumulation").  It does not
name a generator.  Both the oracle and the HIP path implement one
counter-based generator, Philox4x32-10, from its published definition
(J. Salmon, M. Moraes, R. Dror, D. Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11), so that the noise of coordinate e, level k at step t is a
pure function of (seed, e, k, t) and both sides draw the same numbers.

Counter layout (a reading of ours, stated once here):
    key     = (seed mod 2^32, seed >> 32)
    counter = (e mod 2^32, e >> 32, t, stream * 256 + j)
    e       = global coordinate index ((b * O) + o) * I + i
    j       = block of four levels: word r of block j feeds level k = 4 j + r
    stream  = 0 for step noise, 1 for the initial logit noise of Eq. 4

Pinned by: rocRAND's host Philox4x32-10 (tests/test_oracle_rng.py), chi-square
uniformity, Gumbel moments (mean = Euler-Mascheroni constant, variance pi^2/6),
and the Gumbel-max property (argmax(l + g) ~ softmax(l)).
"""
import numpy as np

_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = 0x9E3779B9
_W1 = 0xBB67AE85
_MASK32 = 0xFFFFFFFF

STREAM_STEP = 0
STREAM_INIT = 1


def philox4x32_10(c0, c1, c2, c3, key):
    """Ten Philox rounds on counters (c0..c3) with a 64-bit key.

    Each round multiplies words 0 and 2 by the two round multipliers, keeps
    the 64-bit products' halves, and mixes them with the other two words and
    the round key; the round key is bumped by the two Weyl constants between
    rounds (SC'11, Philox-4x32).
    """
    c = [np.asarray(x, dtype=np.uint32).copy() for x in (c0, c1, c2, c3)]
    c = np.broadcast_arrays(*c)
    c = [np.array(x, dtype=np.uint32) for x in c]
    k0 = int(key) & _MASK32
    k1 = (int(key) >> 32) & _MASK32
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _W0) & _MASK32
            k1 = (k1 + _W1) & _MASK32
        prod0 = _M0 * c[0].astype(np.uint64)
        prod1 = _M1 * c[2].astype(np.uint64)
        hi0 = (prod0 >> np.uint64(32)).astype(np.uint32)
        lo0 = (prod0 & np.uint64(_MASK32)).astype(np.uint32)
        hi1 = (prod1 >> np.uint64(32)).astype(np.uint32)
        lo1 = (prod1 & np.uint64(_MASK32)).astype(np.uint32)
        c = [hi1 ^ c[1] ^ np.uint32(k0), lo1, hi0 ^ c[3] ^ np.uint32(k1), lo0]
    return c


def raw_words(seed, e, t, stream, n_levels):
    """uint32 words for coordinates ``e`` (int64 array), shape (len(e), n_levels)."""
    e = np.asarray(e, dtype=np.uint64)
    lo = (e & np.uint64(_MASK32)).astype(np.uint32)
    hi = (e >> np.uint64(32)).astype(np.uint32)
    out = np.empty((e.size, 4 * ((n_levels + 3) // 4)), dtype=np.uint32)
    for j in range((n_levels + 3) // 4):
        words = philox4x32_10(lo, hi, np.uint32(t & _MASK32),
                              np.uint32(stream * 256 + j), seed)
        for r in range(4):
            out[:, 4 * j + r] = words[r]
    return out[:, :n_levels]


def uniform(words):
    """Map 32-bit words to u in (0, 1): the top 23 bits plus one half, times 2^-23.

    Every value is exactly representable in float32 and lies in
    [2^-24, 1 - 2^-24], so both logarithms of the Gumbel transform are finite.
    """
    return ((np.asarray(words, dtype=np.uint32) >> np.uint32(9)).astype(np.float64) + 0.5) * 2.0 ** -23


def gumbel(seed, e, t, n_levels):
    """Gumbel(0,1) noise g = -ln(-ln u), evaluated in float64, stored as float32.

    Returns float64 values that are exactly float32-representable, shape
    (len(e), n_levels).  Alg. 1 draws these once per logit per forward pass.
    """
    u = uniform(raw_words(seed, e, t, STREAM_STEP, n_levels))
    return np.float32(-np.log(-np.log(u))).astype(np.float64)


def init_normals(seed, e, n_levels):
    """Standard normals for the initial logit noise of Eq. 4 (Box-Muller).

    Words (x0, x1) of each Philox block give z = sqrt(-2 ln u0) cos(2 pi u1)
    for level 4j and the matching sine for level 4j+1; words (x2, x3) give
    levels 4j+2 and 4j+3.  Evaluated in float64, stored as float32.
    """
    u = uniform(raw_words(seed, e, 0, STREAM_INIT, 4 * ((n_levels + 3) // 4)))
    z = np.empty_like(u)
    for a in range(0, u.shape[1], 2):
        rad = np.sqrt(-2.0 * np.log(u[:, a]))
        ang = 2.0 * np.pi * u[:, a + 1]
        z[:, a] = rad * np.cos(ang)
        z[:, a + 1] = rad * np.sin(ang)
    return np.float32(z[:, :n_levels]).astype(np.float64)
