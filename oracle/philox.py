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
    e       = global coordinate index ((b * O) + o) * I + i
    chunk   = the four coordinates e0 .. e0 + 3, e0 = e - e mod 4
    stream  = 0 for step noise, 1 for the initial logit noise of Eq. 4
    sample  = index m of an independent draw within one step (0 for a single draw)
    The chunk's 4 K values (coordinate e0 + q, level k, at flat position f = q K + k) are
    the words of K Philox calls: call j = f div 4 has counter
    (e0 mod 2^32, e0 >> 32, t, (sample * 256 + stream) * 256 + j), and position f takes
    its word f mod 4.  No word is drawn and left unused, whatever K is.

Pinned by: rocRAND's host Philox4x32-10 (tests/test_oracle_rng.py), chi-square
uniformity, Gumbel moments (mean = Euler-Mascheroni constant, variance pi^2/6),
the Gumbel-max property (argmax(l + g) ~ softmax(l)), and for the logistic
values of the binary relaxations: moments (0, pi^2/3), the logistic CDF, and
the law of a difference of two of the generator's Gumbel values.
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


def raw_words(seed, e, t, stream, n_levels, sample=0):
    """uint32 words for coordinates ``e`` (int64 array), shape (len(e), n_levels).

    Follows the chunk layout above: coordinate e, level k sits at flat position
    f = (e mod 4) K + k of its chunk's stream, i.e. word f mod 4 of call f div 4.
    """
    e = np.asarray(e, dtype=np.uint64).reshape(-1)
    e0 = e - (e % np.uint64(4))
    lo = (e0 & np.uint64(_MASK32)).astype(np.uint32)
    hi = (e0 >> np.uint64(32)).astype(np.uint32)
    q = (e % np.uint64(4)).astype(np.int64)
    out = np.empty((e.size, n_levels), dtype=np.uint32)
    calls = {}
    for k in range(n_levels):
        f = q * n_levels + k
        j, w = f // 4, f % 4
        for jj in np.unique(j):
            if jj not in calls:
                calls[jj] = philox4x32_10(lo, hi, np.uint32(t & _MASK32),
                                          np.uint32((sample * 256 + stream) * 256 + int(jj)), seed)
            sel = j == jj
            for ww in range(4):
                m = sel & (w == ww)
                out[m, k] = calls[jj][ww][m]
    return out


def uniform(words):
    """Map 32-bit words to u in (0, 1): the top 23 bits plus one half, times 2^-23.

    Every value is exactly representable in float32 and lies in
    [2^-24, 1 - 2^-24], so both logarithms of the Gumbel transform are finite.
    """
    return ((np.asarray(words, dtype=np.uint32) >> np.uint32(9)).astype(np.float64) + 0.5) * 2.0 ** -23


def gumbel(seed, e, t, n_levels, sample=0):
    """Gumbel(0,1) noise g = -ln(-ln u), evaluated in float64, stored as float32.

    Returns float64 values that are exactly float32-representable, shape
    (len(e), n_levels).  Alg. 1 draws these once per logit per forward pass;
    ``sample`` selects one of several independent draws of the same step.
    """
    u = uniform(raw_words(seed, e, t, STREAM_STEP, n_levels, sample))
    return np.float32(-np.log(-np.log(u))).astype(np.float64)


def logistic(seed, e, t, n_values, sample=0):
    """Logistic(0,1) noise d = ln u - ln(1 - u), evaluated in float64, stored as float32.

    A two-element Gumbel-Softmax with logits {-l, l} (§3) sees its two Gumbel draws only
    through their difference g1 - g0, and the difference of two independent Gumbel(0,1)
    variables is Logistic(0,1); so the binary relaxations draw that difference directly, one
    value per pair (reading), from the same word stream and chunk layout as ``gumbel``.
    1 - u is exact for every u of ``uniform``.  Returns float64 values that are exactly
    float32-representable, shape (len(e), n_values).
    """
    u = uniform(raw_words(seed, e, t, STREAM_STEP, n_values, sample))
    return np.float32(np.log(u) - np.log(1.0 - u)).astype(np.float64)


def init_normals(seed, e, n_levels):
    """Standard normals for the initial logit noise of Eq. 4 (Box-Muller).

    In each chunk's word stream (stream 1, t = 0) the words at flat positions
    (2m, 2m + 1) form one Box-Muller pair: position 2m takes
    z = sqrt(-2 ln u_2m) cos(2 pi u_2m+1) and position 2m + 1 the matching sine.
    A pair never straddles two Philox calls.  Evaluated in float64, stored as float32.
    """
    e = np.asarray(e, dtype=np.uint64).reshape(-1)
    q = (e % np.uint64(4)).astype(np.int64)
    e0 = e - (e % np.uint64(4))
    z = np.empty((e.size, n_levels))
    for k in range(n_levels):
        f = q * n_levels + k
        fk = [uniform(_word_at(seed, e0, STREAM_INIT, ff)) for ff in (f - (f & 1), f | 1)]
        rad = np.sqrt(-2.0 * np.log(fk[0]))
        ang = 2.0 * np.pi * fk[1]
        z[:, k] = np.where(f & 1, rad * np.sin(ang), rad * np.cos(ang))
    return np.float32(z).astype(np.float64)


def _word_at(seed, e0, stream, f):
    """Word at flat position ``f`` (array) of the stream of chunks starting at ``e0``."""
    lo = (e0 & np.uint64(_MASK32)).astype(np.uint32)
    hi = (e0 >> np.uint64(32)).astype(np.uint32)
    out = np.empty(e0.size, dtype=np.uint32)
    j, w = f // 4, f % 4
    for jj in np.unique(j):
        sel = j == jj
        words = philox4x32_10(lo[sel], hi[sel], np.uint32(0), np.uint32(stream * 256 + int(jj)), seed)
        for ww in range(4):
            m = w[sel] == ww
            out[np.flatnonzero(sel)[m]] = words[ww][m]
    return out
