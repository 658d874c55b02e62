"""Pins of the oracle's request-bound sampler (Sec. IV, "Shape-Aligned
Sampling": y_t = S(l_t, R(s, t))) against facts that do not come from its
own code: the published Philox4x32-10 known-answer vectors, the uniform's
exact bounds, the Gumbel-max rule's sampling distribution (it must draw
from softmax(l / T)), closed forms of the log-probability, and the rule's
invariances."""
import math

import numpy as np
import pytest

import oracle


@pytest.mark.parametrize("ctr,key,expect", [
    # known-answer vectors of Philox4x32-10 published with the generator
    # (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011)
    ([0, 0, 0, 0], [0, 0], [0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8]),
    ([0xffffffff] * 4, [0xffffffff] * 2, [0x408f276d, 0x41c83b0e, 0xa20bc7c6, 0x6d5451fd]),
    ([0x243f6a88, 0x85a308d3, 0x13198a2e, 0x03707344], [0xa4093822, 0x299f31d0],
     [0xd16cfe09, 0x94fdcceb, 0x5001e420, 0x24126ea1]),
])
def test_philox_known_answers(ctr, key, expect):
    assert [int(x) for x in oracle.philox4x32_10(ctr, key)] == expect


def test_uniform_is_strictly_inside_the_unit_interval():
    lo = oracle.uniform(0, 0)
    hi = oracle.uniform(0xffffffff, 0xffffffff)
    assert lo == 2.0 ** -53                 # (0 + 1/2) 2^-52
    assert hi == 1.0 - 2.0 ** -53           # (2^52 - 1/2) 2^-52, exactly representable
    assert 0.0 < lo < hi < 1.0


def test_gumbel_max_draws_from_softmax():
    """Empirical frequencies over 40000 steps (counters) match
    softmax(l / T) within five binomial standard deviations per class."""
    l = np.array([1.0, 0.5, -0.3, 2.0, 0.0, -1.5], np.float32)
    T = 0.7
    N = 40000
    counts = np.zeros(l.size)
    for t in range(N):
        tok, _ = oracle.sample(l, 42, t, T)
        counts[tok] += 1
    z = np.exp(l.astype(np.float64) / T)
    p = z / z.sum()
    sd = np.sqrt(p * (1 - p) / N)
    assert np.all(np.abs(counts / N - p) < 5 * sd), (counts / N, p)


def test_greedy_is_the_first_argmax():
    l = np.array([0.5, 3.0, -1.0, 3.0, 2.0], np.float32)
    for T in (0.0, -1.0):
        tok, _ = oracle.sample(l, 7, 3, T)
        assert tok == int(np.argmax(l)) == 1          # numpy: first occurrence


def test_logprob_closed_forms():
    V = 1000
    tok, lp = oracle.sample(np.full(V, 0.25, np.float32), 1, 1, 0.6)
    assert abs(lp - (-math.log(V))) < 1e-12           # equal logits: every token has 1/V
    l = np.zeros(V, np.float32)
    l[17] = 100.0
    tok, lp = oracle.sample(l, 2, 5, 1.0)
    assert tok == 17 and abs(lp) <= V * math.exp(-100.0)   # one dominant logit: probability 1 - O(V e^-100)


def test_temperature_is_a_logit_scale():
    """T = 0.5 on l draws the same token as T = 1 on 2 l (exact scaling), with the same log-probability."""
    rng = np.random.default_rng(3)
    for t in range(50):
        l = rng.normal(0, 2, 300).astype(np.float32)
        a = oracle.sample(l, 9, t, 0.5)
        b = oracle.sample((2 * l).astype(np.float32), 9, t, 1.0)
        assert a[0] == b[0] and abs(a[1] - b[1]) < 1e-12


def test_variate_is_bound_to_seed_and_step():
    """Same (seed, step, logits) -> same token; the stream of one seed does
    not depend on which other seeds are drawn in between (there is no
    state), and different seeds give different streams."""
    rng = np.random.default_rng(4)
    l = rng.normal(0, 1, 64).astype(np.float32)
    first = [oracle.sample(l, 42, t, 1.0)[0] for t in range(200)]
    interleaved = []
    for t in range(200):
        oracle.sample(l, 1234 + t, t, 1.0)            # another request's draw
        interleaved.append(oracle.sample(l, 42, t, 1.0)[0])
    assert first == interleaved
    other = [oracle.sample(l, 43, t, 1.0)[0] for t in range(200)]
    assert sum(a != b for a, b in zip(first, other)) > 100


def test_logprob_of_two_tokens_and_shift_invariance():
    """Logits (0, ln 3) give probabilities (1/4, 3/4); adding a constant to
    every logit changes neither the draw nor its log-probability."""
    l = np.array([0.0, math.log(3.0)], np.float32)     # softmax -> (1/4, 3/4)
    for t in range(20):
        tok, lp = oracle.sample(l, 11, t, 1.0)
        expect = math.log(0.25) if tok == 0 else math.log(0.75)
        assert abs(lp - expect) < 1e-7                 # log(3) rounded to fp32
    rng = np.random.default_rng(5)
    x = rng.normal(0, 1, 100).astype(np.float32)
    a = oracle.sample(x, 3, 8, 1.0)
    b = oracle.sample((x + np.float32(4.0)).astype(np.float32), 3, 8, 1.0)
    assert a[0] == b[0] and abs(a[1] - b[1]) < 1e-6
