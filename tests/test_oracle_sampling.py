"""Pins of the sampler oracle (CPU only).

* Philox4x64-10 known answers from numpy.random.Philox, an independent
  implementation of the same published generator (numpy increments its
  counter before each block, so its state counter c yields block c + 1);
* uniforms exactly of the form (m + 0.5) * 2^-23, m the top 23 bits of a word;
* Gumbel-max draws follow softmax(logits / T) (chi-square test);
* temperature 0 is argmax with the lowest index on ties.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import sampling as osm


def _numpy_block(counter, key):
    c = np.array(counter, dtype=object)
    # numpy pre-increments the 256-bit counter: start from counter - 1 (with borrow)
    val = int(c[0]) + (int(c[1]) << 64) + (int(c[2]) << 128) + (int(c[3]) << 192) - 1
    val %= 1 << 256
    start = np.array([(val >> (64 * i)) & ((1 << 64) - 1) for i in range(4)], dtype=np.uint64)
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=start)
    return bg.random_raw(4)


@pytest.mark.parametrize("counter,key", [
    ((1, 0, 0, 0), (0, 0)),
    ((7, 3, 0, 0), (5, 7)),
    ((0, 0, 0, 0), (12345, 678)),                       # borrow across all words
    ((2**64 - 1, 2**63 + 5, 9, 1), (2**64 - 1, 2**64 - 2)),
    ((17407, 19007, 0, 0), (203, 575)),
])
def test_philox_matches_numpy(counter, key):
    ours = osm.philox4x64_10(np.array(counter, dtype=np.uint64), key)
    assert np.array_equal(ours, _numpy_block(counter, key))


def test_philox_vectorised_equals_scalar():
    ctr = np.array([[5, g, 0, 0] for g in range(10)], dtype=np.uint64)
    many = osm.philox4x64_10(ctr, (1, 2))
    for g in range(10):
        assert np.array_equal(many[g], _numpy_block((5, g, 0, 0), (1, 2)))


def test_uniform_word_layout_and_exactness():
    u = osm.uniforms(11, 22, 33, 21)
    big = osm.uniforms(1, 2, 3, 4096)
    mb = big.astype(np.float64) * 2**23 - 0.5
    assert np.all(mb == np.round(mb)) and mb.max() >= 2**22
    blk = _numpy_block((33, 0, 0, 0), (11, 22))
    w0 = int(blk[0]) & 0xFFFFFFFF
    w1 = int(blk[0]) >> 32
    assert u[0] == np.float32(((w0 >> 9) + 0.5) / 2**23)
    assert u[1] == np.float32(((w1 >> 9) + 0.5) / 2**23)
    blk2 = _numpy_block((33, 2, 0, 0), (11, 22))
    assert u[20] == np.float32((((int(blk2[2]) & 0xFFFFFFFF) >> 9) + 0.5) / 2**23)
    m = u.astype(np.float64) * 2**23 - 0.5
    assert np.all(m == np.round(m)) and np.all((u > 0) & (u < 1))


def test_gumbel_max_follows_softmax():
    rng = np.random.default_rng(0)
    V, T, n = 16, 0.7, 20000
    logits = rng.standard_normal(V) * 1.5
    counts = np.zeros(V)
    for pos in range(n):
        counts[osm.sample(logits, T, 42, 7, pos)] += 1
    p = np.exp(logits / T - np.max(logits / T))
    p /= p.sum()
    chi = stats.chisquare(counts, p * n)
    assert chi.pvalue > 1e-3, chi


def test_greedy_and_ties():
    l = np.array([0.5, 2.0, -1.0, 2.0, 1.9])
    assert osm.sample(l, 0.0, 1, 1, 1) == 1
    assert osm.top2_gap(osm.scores(l, 0.0, 1, 1, 1)) == 0.0
    # a very low temperature concentrates on the argmax
    l2 = np.array([0.0, 5.0, 1.0])
    assert all(osm.sample(l2, 0.01, 3, 4, p) == 1 for p in range(50))


def test_logprob_closed_forms():
    V = 151936
    assert osm.logprob(np.zeros(V), 1.0, 17) == pytest.approx(-np.log(V), abs=1e-12)   # uniform
    a, b = 2.5, -1.0                                                                     # two tokens: log sigmoid
    assert osm.logprob(np.array([a, b]), 1.0, 0) == pytest.approx(-np.log1p(np.exp(b - a)), abs=1e-14)
    assert osm.logprob(np.array([a, b]), 0.5, 1) == pytest.approx(-np.log1p(np.exp((a - b) / 0.5)), abs=1e-12)
    big = np.full(1000, -1e4)
    big[3] = 1e4                                                                         # no overflow, p -> 1
    assert osm.logprob(big, 1.0, 3) == pytest.approx(0.0, abs=1e-12)
    assert osm.logprob(big, 1.0, 4) == pytest.approx(-2e4, rel=1e-12)


def test_logprob_invariants():
    rng = np.random.default_rng(4)
    l = rng.standard_normal(300) * 3
    for T in (0.0, 0.7, 1.0, 1.6):
        lp = np.array([osm.logprob(l, T, v) for v in range(300)])
        assert np.exp(lp).sum() == pytest.approx(1.0, abs=1e-12)                       # a distribution
        assert osm.logprob(l + 123.0, T, 7) == pytest.approx(lp[7], abs=1e-12)         # shift invariance
        t = 1.0 if T == 0 else T
        assert osm.logprob(l / t, 1.0, 11) == pytest.approx(lp[11], abs=1e-12)          # temperature = rescaled logits
        assert np.argmax(lp) == np.argmax(l)                                            # monotone in the logit


def test_stop_at_eos():
    assert osm.stop_at([5, 9, 3, 9, 1], 9) == [5, 9]
    assert osm.stop_at([5, 9, 3], 4) == [5, 9, 3]
    assert osm.stop_at([4], 4) == [4]
