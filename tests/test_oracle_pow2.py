"""Pins of the oracle's power-of-two attention weights (Sec. II-E, eq. logsm:
A~_j = 2^-k_j, k_j = round(M - x_j) >= 0; both products by powers of two with
the INT8 values of eq. av).

Readings: k_j = M - ceil(x_j - 1/2), i.e. M - x_j rounded half up (k - M then
depends on x alone, so the weights of an online pass whose running maximum
rises are exact rescales of the final ones); O = sum A~ v / sum A~ over all
keys (eq. av leaves the normalisation out; no k_max cut). Pinned by:
* the rounding rule itself, against exact rationals, ties included;
* integer scores, where 2^-k is the softmax weight 2^(x - M) exactly;
* exact rational attention on small inputs;
* online tiles and splits, key order, and a common integer shift of all
  scores, none of which may change O.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle


def _rows(rng, T):
    return (rng.integers(-127, 128, size=(T, 64)).astype(np.int8),
            rng.integers(-3, 9, size=T).astype(np.int8))


def _exact(x, v8, g):
    """O in exact rationals: M = ceil(max x), k = floor(M - x + 1/2)."""
    x = [Fraction(float(a)) for a in np.asarray(x, np.float32)]
    M = max(math.ceil(a) for a in x)
    ks = [math.floor(M - a + Fraction(1, 2)) for a in x]       # M - x rounded half up
    wts = [Fraction(1, 2 ** kk) for kk in ks]
    den = sum(wts)
    out = []
    for d in range(64):
        num = sum(wt * int(v8[t, d]) * Fraction(2) ** (-int(g[t])) for t, wt in enumerate(wts))
        out.append(num / den)
    return np.array([float(o) for o in out]), M, ks


def test_rounding_rule_against_exact_rationals():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(300) * 6).astype(np.float32)
    x[:8] = [2.5, -1.5, 0.5, 3.0, -2.0, 7.5,        # ties and integers
             -0.49999997, 0.49999997]               # one fp32 ulp off a tie
    v8, g = _rows(rng, 300)
    out, M = oracle.attend_x(x, v8, g, pow2=True)
    ref, Mr, ks = _exact(x, v8, g)
    assert M == Mr
    assert min(ks) >= 0                               # eq. logsm: k >= 0
    assert np.abs(out - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())
    # the rule: |k - (M - x)| <= 1/2, with M - x = n + 1/2 going to n + 1
    for a, kk in zip(x.tolist(), ks):
        d = Fraction(M) - Fraction(a)
        assert abs(kk - d) <= Fraction(1, 2)
        if d.denominator == 2:
            assert kk == d + Fraction(1, 2)


def test_rounding_rule_near_ties():
    """x = n + 1/2 and its fp32 neighbours on both sides, for scores of both
    signs and magnitudes up to 2^22: every weight follows M - x rounded half up
    exactly. (A rule that forms x - 1/2 in fp32 rounds -0.5 + 2^-25 to -1 and
    halves that key's weight.)"""
    base = []
    for n in (-40, -7, -3, -2, -1, 0, 1, 2, 5, 300, 2 ** 21):
        t = np.float32(n + 0.5)
        base += [t, np.nextafter(t, np.float32(np.inf)), np.nextafter(t, np.float32(-np.inf))]
    base += [np.float32(-0.49999997), np.float32(0.49999997), np.float32(-2.0 ** -25),
             np.float32(2.0 ** 22 - 0.5)]
    g = np.zeros(2, np.int8)
    for a in base:
        # two keys: the probed score and the maximum's key at ceil(a); one-hot
        # values read the probed key's share, 1 / (1 + 2^k)
        top = np.float32(np.ceil(np.float64(a)))
        x = np.array([a, top], np.float32)
        v = np.zeros((2, 64), np.int8)
        v[0, 0] = 1
        out, M = oracle.attend_x(x, v, g, pow2=True)
        k = math.floor(Fraction(M) - Fraction(float(a)) + Fraction(1, 2))
        assert M == int(top)
        assert out[0] == 1.0 / (1.0 + 2.0 ** k), (float(a), k, out[0])


def test_rounding_rule_printed_counterexample():
    # x = -0.5 + 2^-25 and -0.1 under M = 0: both round to k = 0, so a one-hot
    # value on the first key carries exactly half of the mass
    x = np.array([-0.49999997, -0.1], np.float32)
    assert float(x[0]) == -0.5 + 2.0 ** -25
    v = np.zeros((2, 64), np.int8)
    v[0, 0] = 1
    out, M = oracle.attend_x(x, v, np.zeros(2, np.int8), pow2=True)
    assert M == 0 and out[0] == 0.5


def test_integer_scores_give_the_softmax():
    rng = np.random.default_rng(2)
    x = rng.integers(-20, 5, size=200).astype(np.float32)
    v8, g = _rows(rng, 200)
    a, _ = oracle.attend_x(x, v8, g, pow2=True)
    b, _ = oracle.attend_x(x, v8, g, pow2=False)
    assert np.array_equal(a, b)


@pytest.mark.parametrize("tile,split", [(1, 7), (7, 64), (64, 100), (128, 513)])
def test_online_and_splits_equal_two_pass(tile, split):
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(513) * 4).astype(np.float32)
    v8, g = _rows(rng, 513)
    a, Ma = oracle.attend_x(x, v8, g, pow2=True)
    b, Mb = oracle.attend_x(x, v8, g, pow2=True, split_len=split, tile=tile)
    assert Ma == Mb and np.abs(a - b).max() <= 1e-12 * np.abs(a).max()


def test_key_order_and_integer_shift_do_not_matter():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal(400) * 5).astype(np.float32)
    v8, g = _rows(rng, 400)
    a, M = oracle.attend_x(x, v8, g, pow2=True)
    p = rng.permutation(400)
    b, _ = oracle.attend_x(x[p], v8[p], g[p], pow2=True)
    c, Mc = oracle.attend_x(x + np.float32(13.0), v8, g, pow2=True)
    assert np.abs(a - b).max() <= 1e-12 * np.abs(a).max()
    assert Mc == M + 13 and np.abs(a - c).max() <= 1e-12 * np.abs(a).max()


def test_weights_within_half_a_binade_of_the_softmax():
    # each power-of-two weight is within a factor 2^(1/2) of 2^(x - M), so the
    # two normalisers are too
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(256) * 3).astype(np.float32)
    v8 = np.zeros((256, 64), np.int8)
    v8[:, 0] = 1
    g = np.zeros(256, np.int8)
    # with v = e_0 for every key, O_0 = 1 for both rules; use a one-hot value
    # to read one weight share at a time
    for t in (0, 17, 200):
        v = np.zeros((256, 64), np.int8)
        v[t, 0] = 1
        a, _ = oracle.attend_x(x, v, g, pow2=True)
        b, _ = oracle.attend_x(x, v, g, pow2=False)
        assert 0.5 <= a[0] / b[0] <= 2.0
    a, _ = oracle.attend_x(x, v8, g, pow2=True)
    assert abs(a[0] - 1.0) < 1e-15
