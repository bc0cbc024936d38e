"""Pins of the oracle's generator: Philox4x32-10, the uniform map, Gumbel and normal noise."""
import subprocess

import numpy as np
import pytest
from scipy import stats

from oracle import philox

EULER_GAMMA = 0.5772156649015329


def test_philox_matches_rocrand_host_implementation(rocrand_philox):
    """Philox4x32-10 equals rocRAND's independent implementation on random keys/counters."""
    rng = np.random.default_rng(5)
    words = rng.integers(0, 2**32, size=(3000, 6), dtype=np.uint64)
    words[:4] = [[0] * 6, [0xFFFFFFFF] * 6, [1, 0, 0, 0, 0, 0], [0, 0, 0, 0, 0, 1]]
    text = "\n".join(" ".join(f"{int(x):x}" for x in row) for row in words) + "\n"
    out = subprocess.run([rocrand_philox], input=text, capture_output=True, text=True, check=True)
    ref = np.array([[int(x, 16) for x in line.split()] for line in out.stdout.strip().splitlines()],
                   dtype=np.uint64)
    key = (words[:, 0] | (words[:, 1] << np.uint64(32)))
    got = np.empty_like(ref)
    for n in range(len(words)):
        r = philox.philox4x32_10(words[n, 2], words[n, 3], words[n, 4], words[n, 5], int(key[n]))
        got[n] = [int(x) for x in r]
    np.testing.assert_array_equal(got, ref)


def test_counter_layout_fields_all_reach_the_output():
    """Changing any of (e low, e high, t, stream, level block, seed) changes every output word."""
    base = philox.raw_words(7, np.array([5], np.int64), 3, 0, 8)
    for other in (philox.raw_words(7, np.array([6], np.int64), 3, 0, 8),
                  philox.raw_words(7, np.array([5 + 2**32], np.int64), 3, 0, 8),
                  philox.raw_words(7, np.array([5], np.int64), 4, 0, 8),
                  philox.raw_words(7, np.array([5], np.int64), 3, 1, 8),
                  philox.raw_words(8, np.array([5], np.int64), 3, 0, 8),
                  philox.raw_words(7 + 2**32, np.array([5], np.int64), 3, 0, 8)):
        assert np.all(other != base)
    # the levels of one coordinate come from different words, not from a shifted copy
    assert np.all(base[0, 4:] != base[0, :4])


@pytest.mark.parametrize("K", [2, 3, 5, 8])
def test_chunk_stream_layout(K):
    """The 4 K values of an aligned chunk of four coordinates are the words of K calls, in
    order: coordinate e0 + q, level k is word (qK + k) mod 4 of call (qK + k) div 4."""
    seed, t, e0 = 99, 5, 4 * 1234567
    got = philox.raw_words(seed, np.arange(e0, e0 + 4), t, 0, K).reshape(-1)
    calls = [philox.philox4x32_10(e0, 0, t, j, seed) for j in range(K)]
    want = np.array([int(c[r]) for c in calls for r in range(4)], dtype=np.uint32)
    np.testing.assert_array_equal(got, want)
    # every coordinate of the chunk agrees with a lookup of its own
    for q in range(4):
        np.testing.assert_array_equal(philox.raw_words(seed, [e0 + q], t, 0, K)[0], want[q * K:(q + 1) * K])


def test_uniform_map_is_exact_and_uniform():
    w = np.array([0, 1, 511, 512, 2**32 - 1], dtype=np.uint32)
    u = philox.uniform(w)
    assert u[0] == 2.0**-24 and u[-1] == 1 - 2.0**-24
    assert u[1] == u[0] and u[3] == 3 * 2.0**-24
    assert np.all(u.astype(np.float32).astype(np.float64) == u)
    words = philox.raw_words(1, np.arange(250_000, dtype=np.int64), 0, 0, 4).reshape(-1)
    counts = np.bincount(words >> np.uint32(24), minlength=256)
    assert stats.chisquare(counts).pvalue > 1e-4


def test_gumbel_moments():
    """Gumbel(0,1): mean = Euler-Mascheroni constant, variance = pi^2 / 6."""
    g = philox.gumbel(3, np.arange(500_000, dtype=np.int64), 11, 4).reshape(-1)
    n = g.size
    var = np.pi**2 / 6
    assert abs(g.mean() - EULER_GAMMA) < 5 * np.sqrt(var / n)
    # variance of the sample variance for Gumbel: (mu4 - sigma^4)/n with excess kurtosis 12/5
    mu4 = (3 + 12 / 5) * var**2
    assert abs(g.var() - var) < 5 * np.sqrt((mu4 - var**2) / n)
    assert stats.kstest(g[:200_000], stats.gumbel_r.cdf).pvalue > 1e-4


def test_gumbel_max_samples_the_softmax():
    """argmax_k (l_k + g_k) ~ Categorical(softmax(l)) (the Gumbel-max identity behind Alg. 1)."""
    l = np.array([0.3, -1.2, 1.0, 0.1, -0.4])
    n = 300_000
    g = philox.gumbel(9, np.arange(n, dtype=np.int64), 0, 5)
    k = np.argmax(l + g, axis=1)
    p = np.exp(l) / np.exp(l).sum()
    assert stats.chisquare(np.bincount(k, minlength=5), n * p).pvalue > 1e-4


def test_logistic_moments_and_cdf():
    """Logistic(0,1): mean 0, variance pi^2 / 3, CDF 1 / (1 + e^-x), symmetric."""
    d = philox.logistic(4, np.arange(400_000, dtype=np.int64), 13, 2).reshape(-1)
    n = d.size
    var = np.pi**2 / 3
    assert abs(d.mean()) < 5 * np.sqrt(var / n)
    mu4 = (3 + 6 / 5) * var**2                  # excess kurtosis of the logistic: 6/5
    assert abs(d.var() - var) < 5 * np.sqrt((mu4 - var**2) / n)
    assert stats.kstest(d[:200_000], stats.logistic.cdf).pvalue > 1e-4
    # the word -> value map is monotone and antisymmetric under u -> 1 - u (x -> ~x)
    w = np.array([0, 1 << 9, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFF], dtype=np.uint32)
    u = philox.uniform(w)
    val = np.log(u) - np.log(1.0 - u)
    assert np.all(np.diff(val) >= 0)
    np.testing.assert_allclose(val + (np.log(1 - u) - np.log(u)), 0.0, atol=0)


def test_logistic_has_the_law_of_a_difference_of_two_gumbels():
    """The binary relaxation's noise replaces g1 - g0 of two independent Gumbel(0,1) values: the
    generator's logistic values and differences of its Gumbel values have one law (two-sample
    KS), and the logistic values are the transform ln(u / (1 - u)) of the same words."""
    g = philox.gumbel(6, np.arange(150_000, dtype=np.int64), 3, 2)
    d = philox.logistic(6, np.arange(150_000, 300_000, dtype=np.int64), 3, 2).reshape(-1)
    assert stats.ks_2samp(g[:, 1] - g[:, 0], d).pvalue > 1e-4
    e = np.arange(1000, dtype=np.int64)
    u = philox.uniform(philox.raw_words(6, e, 3, philox.STREAM_STEP, 2))
    want = np.float32(np.log(u / (1 - u))).astype(np.float64)
    got = philox.logistic(6, e, 3, 2)
    assert np.abs(got - want).max() <= 2 * np.abs(want).max() * 2.0**-24


def test_init_normals_are_standard_normal():
    z = philox.init_normals(2, np.arange(200_000, dtype=np.int64), 8).reshape(-1)
    assert abs(z.mean()) < 5 / np.sqrt(z.size)
    assert abs(z.var() - 1) < 5 * np.sqrt(2 / z.size)
    assert stats.kstest(z[:200_000], "norm").pvalue > 1e-4
    # the sine and cosine halves of one Box-Muller pair are uncorrelated
    zz = philox.init_normals(2, np.arange(100_000, dtype=np.int64), 2)
    assert abs(np.corrcoef(zz[:, 0], zz[:, 1])[0, 1]) < 5 / np.sqrt(zz.shape[0])
