"""Pins of the stochastic-verification oracle (no GPU).

* Philox4x32-10 against the published known-answer vectors of its authors'
  Random123 distribution (counter, key -> output).
* The sampler's fp32 log against numpy's.
* Gumbel-max sampling: empirical frequencies over many independent rows match
  softmax(x / T); at a very low temperature the sample is the argmax.
* Stochastic acceptance: a request's drafts are all accepted with probability
  prod_j p_j(d_j), the rows being independent draws.
* Determinism in (seed, offset, row) and separation across them.
"""
from __future__ import annotations

import math
import os

import numpy as np
import pytest

import oracle

def _load_kat():
    """(counter, key, output) word tuples from tests/golden/philox4x32_10_kat.txt."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "philox4x32_10_kat.txt")
    out = []
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if not line:
                continue
            w = [int(x, 16) for x in line]
            assert len(w) == 10, line
            out.append((tuple(w[0:4]), tuple(w[4:6]), tuple(w[6:10])))
    return out


KAT = _load_kat()


@pytest.mark.parametrize("ctr,key,want", KAT)
def test_philox_known_answers(ctr, key, want):
    assert oracle.philox4x32_10(ctr, key).tolist() == list(want)


def test_sample_log_accuracy():
    x = np.concatenate([np.logspace(-8, 1.3, 50000), [1.0, 2.0, 0.5, 3e-8, 17.3]]).astype(np.float32)
    got = oracle.sample_log(x).astype(np.float64)
    ref = np.log(x.astype(np.float64))
    assert np.all(np.abs(got - ref) <= 3e-7 * np.maximum(np.abs(ref), 1.0))
    assert oracle.sample_log(np.float32([1.0]))[0] == 0.0


def _rows(logits, n):
    return np.tile(np.asarray(logits, dtype=np.float32), (n, 1))


@pytest.mark.parametrize("T", [0.6, 1.0, 1.7])
def test_gumbel_max_frequencies_match_softmax(T):
    x = np.array([1.0, 0.2, -0.5, 2.1, 2.0, -3.0], dtype=np.float32)
    n = 40000
    got = oracle.sample(_rows(x, n), oracle.F32, T, seed=1234, offset=7)
    freq = np.bincount(got, minlength=x.size) / n
    z = x.astype(np.float64) * float(oracle.inv_temperature(T))
    p = np.exp(z - z.max())
    p /= p.sum()
    sigma = np.sqrt(p * (1 - p) / n)
    assert np.all(np.abs(freq - p) <= 5 * sigma + 1e-12), (freq, p)


def test_low_temperature_is_the_argmax():
    rng = np.random.default_rng(3)
    x = rng.permutation(np.arange(64, dtype=np.float32) * 0.1).reshape(1, 64)
    x = np.tile(x, (50, 1))
    for r in range(50):
        x[r] = rng.permutation(x[r])
    got = oracle.sample(x, oracle.F32, 1e-3, seed=9)
    want, _ = oracle.argmax(x, oracle.F32, with_gap=False)
    assert np.array_equal(got, want)


def test_stochastic_acceptance_rate():
    # one request, k = 3 drafts, every row with the same distribution: all
    # three drafts accepted with probability p(d1) p(d2) p(d3)
    x = np.array([0.0, 1.0, 0.5, -1.0], dtype=np.float32)
    T = 0.8
    z = x.astype(np.float64) * float(oracle.inv_temperature(T))
    p = np.exp(z - z.max())
    p /= p.sum()
    drafts = [1, 2, 1]
    R = 20000
    n = 4
    logits = _rows(x, R * n)
    samp = oracle.sample(logits, oracle.F32, T, seed=77)
    q_start = np.arange(0, R * n + 1, n, dtype=np.int32)
    tokens = np.tile(np.array([3] + drafts, dtype=np.int32), R)
    acc, ne, em = oracle.accept(q_start, tokens, samp)
    full = float(np.mean(acc == 3))
    want = p[1] * p[2] * p[1]
    assert abs(full - want) <= 5 * math.sqrt(want * (1 - want) / R)
    first_reject = float(np.mean(acc == 0))
    assert abs(first_reject - (1 - p[1])) <= 5 * math.sqrt(p[1] * (1 - p[1]) / R)
    # the token emitted at a first-position rejection follows p without d1
    rej = acc == 0
    bonus = em[q_start[:-1][rej]]
    assert not np.any(bonus == 1)
    resid = np.delete(p, 1) / (1 - p[1])
    freq = np.bincount(bonus, minlength=4)[[0, 2, 3]] / rej.sum()
    assert np.all(np.abs(freq - resid) <= 5 * np.sqrt(resid * (1 - resid) / rej.sum()))


def test_determinism_and_counter_separation():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((64, 1000)).astype(np.float32)
    a = oracle.sample(x, oracle.F32, 1.0, seed=5, offset=0)
    assert np.array_equal(a, oracle.sample(x, oracle.F32, 1.0, seed=5, offset=0))
    for other in (oracle.sample(x, oracle.F32, 1.0, seed=6, offset=0),
                  oracle.sample(x, oracle.F32, 1.0, seed=5, offset=1),
                  oracle.sample(x, oracle.F32, 1.0, seed=5 + (1 << 32), offset=0)):
        assert np.mean(a != other) > 0.5
    # identical rows draw different samples (the row is part of the counter)
    same = np.tile(x[:1], (64, 1))
    s = oracle.sample(same, oracle.F32, 1.0, seed=5)
    assert len(set(s.tolist())) > 20


def test_special_rows():
    x = np.zeros((3, 8), dtype=np.float32)
    x[0, 5] = np.nan
    x[0, 6] = np.nan
    x[1, :] = -np.inf
    x[2, :] = -np.inf
    x[2, 3] = 0.0
    s = oracle.sample(x, oracle.F32, 0.7, seed=1)
    assert s.tolist() == [5, 0, 3]


def test_noise_term_is_bounded_and_monotone():
    # the uniform is an odd multiple of 2^-24 strictly inside (0, 1) for every
    # word, so the noise is finite, increasing in the word, and at its extremes
    # -log(-log(u)) of the extreme uniforms
    top = np.arange(0, 1 << 23, 997, dtype=np.uint64)
    w = np.concatenate([(top << 9), (top << 9) | 0x1FF,
                        [0, 1, 0x1FF, 0xFFFFFE00, 0xFFFFFFFF, 0x80000000, 0x7FFFFFFF]]).astype(np.uint32)
    u, g = oracle.gumbel_of_word(w)
    k = (w >> 9).astype(np.float64)
    np.testing.assert_array_equal(u.astype(np.float64), (2 * k + 1) * 2.0 ** -24)
    assert np.all((u > 0) & (u < 1)) and np.all(np.isfinite(g))
    order = np.argsort(w, kind="stable")
    assert np.all(np.diff(g[order].astype(np.float64)) >= 0)
    lo, hi = oracle.gumbel_of_word(np.uint32([0, 0xFFFFFFFF]))[1].astype(np.float64)
    assert abs(lo - (-math.log(-math.log(2.0 ** -24)))) < 1e-5
    assert abs(hi - (-math.log(-math.log1p(-2.0 ** -24)))) < 1e-4 * 16.6


def test_dominant_logit_wins_every_row_of_a_large_vocabulary():
    # one token 30 nats above 131071 others: every other token together has
    # probability 131071 e^-30 ~ 1e-8 per row, so 400 rows all draw the
    # dominant token; an unbounded noise term (u rounding to 1) would not
    V, R = 1 << 17, 400
    x = np.zeros((R, V), dtype=np.float32)
    x[:, 777] = 30.0
    s = oracle.sample(x, oracle.F32, 1.0, seed=2024, offset=0)
    assert np.all(s == 777), int((s != 777).sum())
