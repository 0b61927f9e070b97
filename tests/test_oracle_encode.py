"""Pins for the oracle's key encoder (Sec. II-A eq. pot, Sec. II-D eq. mant).

The oracle decides each code by brute force over the grid in fp64 log2
distance. These tests check it against things fixed independently of that:
  * an exact classifier built here from rational arithmetic: for adjacent grid
    values g_a < g_b the fp32 threshold theta = RD_fp32(sqrt(g_a g_b)) is
    derived and verified with exact integers (theta^2 < g_a g_b <
    nextup(theta)^2), so for fp32 u "above the log-midpoint" is exactly
    u > theta; run over all 65536 fp16 bit patterns at several scales;
  * the error range and RMS printed in Sec. II-D;
  * structural facts: the absmax element decodes to s, sign symmetry, zero rows,
    the Hadamard matrix and exact rational rotations.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.integrate
import scipy.linalg

import oracle

E = 6
GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                   "paper_constants.json")))


def grid(k):
    """Sorted [(value, e, j)] of (1 + j/2^k) 2^-e, e in 0..E, j < 2^k."""
    g = [(Fraction(2**k + j, 2**(k + e)), e, j)
         for e in range(E + 1) for j in range(2**k)]
    return sorted(g)


def rd_sqrt_f32(tau2: Fraction) -> np.float32:
    """Largest fp32 theta with theta^2 < tau2 (tau2 not an fp32 square)."""
    th = np.float32(math.sqrt(float(tau2)))
    while Fraction(float(th)) ** 2 >= tau2:
        th = np.nextafter(th, np.float32(0))
    while Fraction(float(np.nextafter(th, np.float32(np.inf)))) ** 2 < tau2:
        th = np.nextafter(th, np.float32(np.inf))
    nx = np.nextafter(th, np.float32(np.inf))
    assert Fraction(float(th)) ** 2 < tau2 < Fraction(float(nx)) ** 2
    return th


def exact_classifier(k):
    g = grid(k)
    thetas = np.array([rd_sqrt_f32(a[0] * b[0]) for a, b in zip(g[:-1], g[1:])],
                      np.float32)
    theta_zero = rd_sqrt_f32(Fraction(1, 2**(2 * E + 1)))  # 2^-(E+1/2)
    return g, thetas, theta_zero


def classify(u, k):
    """(zero, e, j) per fp32 ratio u (NaN -> zero)."""
    g, thetas, theta_zero = exact_classifier(k)
    u = np.asarray(u, np.float32)
    zero = ~(u > theta_zero)  # also true for NaN
    idx = np.searchsorted(thetas, u, side="left")  # number of thetas < u
    idx = np.minimum(idx, len(g) - 1)
    es = np.array([x[1] for x in g])[idx]
    js = np.array([x[2] for x in g])[idx]
    return zero, es, js


def unpack(se, cm, k):
    """(neg, e, j) [rows, 64] from the cache layout."""
    rows = se.shape[0]
    m = np.arange(64)
    nib = (se[:, m // 2] >> (4 * (m % 2))) & 15
    neg, e = (nib >> 3) & 1, nib & 7
    j = np.zeros((rows, 64), np.int64)
    for b in range(k):
        j |= ((cm[:, 8 * b + m // 8] >> (m % 8)) & 1).astype(np.int64) << b
    return neg, e, j


def all_fp16_rows():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    return bits.reshape(1024, 64)


def decoded_ratio(e, j, k):
    return (1.0 + j / 2.0**k) * np.exp2(-e.astype(np.float64))


def test_golden_field_width():
    # 4-bit field = 1 sign + 3 exponent bits; values 0..7, 7 = zero
    assert 2**3 - 2 == GOLD["exp_max_for_4bit_field"]["value"] == E


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("s", [1.0, 0.001, 3.7, 65504.0, 2.0**-20])
def test_exhaustive_fp16_vs_exact_thresholds(k, s):
    kb = all_fp16_rows()
    se, cm, sc = oracle.encode_keys(kb, mant_bits=k,
                                    key_scale=np.full(1024, s, np.float32))
    neg, e, j = unpack(se, cm if k else np.zeros((1024, 0), np.uint8), k)
    x = kb.view(np.float16).astype(np.float32)
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        u = np.abs(x) / np.float32(s)
    zero, ee, jj = classify(u, k)
    assert np.array_equal(e == 7, zero)
    nz = ~zero
    assert np.array_equal(e[nz], ee[nz])
    assert np.array_equal(j[nz], jj[nz])
    assert np.array_equal(neg[nz], np.signbit(x)[nz].astype(neg.dtype))
    # canonical zero: neg = 0, j = 0
    assert not neg[zero].any() and not j[zero].any()


@pytest.mark.parametrize("k", [0, 1, 4])
def test_absmax_mode_matches_exact_classifier(k):
    rng = np.random.default_rng(11)
    x = (rng.standard_normal((512, 64)) *
         rng.uniform(0.5, 4, 64)).astype(np.float16)
    se, cm, sc = oracle.encode_keys(x.view(np.uint16), mant_bits=k)
    xf = x.astype(np.float32)
    assert np.array_equal(sc, np.abs(xf).max(axis=1))
    neg, e, j = unpack(se, cm if k else np.zeros((512, 0), np.uint8), k)
    zero, ee, jj = classify(np.abs(xf) / sc[:, None], k)
    assert np.array_equal(e == 7, zero)
    assert np.array_equal(e[~zero], ee[~zero]) and np.array_equal(j[~zero], jj[~zero])
    # the absmax element decodes to exactly s: u = 1 -> e = 0, j = 0
    am = np.abs(xf).argmax(axis=1)
    r = np.arange(512)
    assert (e[r, am] == 0).all() and (j[r, am] == 0).all()
    assert (neg[r, am] == (xf[r, am] < 0)).all()


def test_pot4_relative_error_range():
    lo, hi = GOLD["pot4_rel_err_range"]["printed"]
    assert abs((2**-0.5 - 1) - lo) < 1e-3 and abs((2**0.5 - 1) - hi) < 1e-3
    rng = np.random.default_rng(3)
    t = rng.uniform(0.0, 6.0, 64 * 2000)  # u = 2^-t inside the exponent range
    u = np.exp2(-t).astype(np.float32).reshape(-1, 64)
    se, _, _ = oracle.encode_keys(u.astype(np.float16).view(np.uint16),
                                  key_scale=np.ones(u.shape[0], np.float32))
    uf = u.astype(np.float16).astype(np.float64)
    _, e, _ = unpack(se, None, 0)
    ok = e != 7
    rel = np.exp2(-e[ok].astype(np.float64)) / uf[ok] - 1.0
    assert rel.min() >= 2**-0.5 - 1 - 1e-6
    assert rel.max() <= 2**0.5 - 1 + 1e-6
    # both ends of the range are approached
    assert rel.min() < 2**-0.5 - 1 + 0.01 and rel.max() > 2**0.5 - 1 - 0.01


def test_pot4_rms_matches_integral():
    g = GOLD["pot4_rel_err_rms"]
    val, _ = scipy.integrate.quad(lambda x: (2.0**x - 1.0) ** 2, -0.5, 0.5)
    rms = math.sqrt(val)
    assert abs(rms - g["integral_value"]) < 5e-5
    assert abs(rms - g["printed"]) < 2e-3  # the paper's rounded print
    rng = np.random.default_rng(5)
    t = rng.uniform(0.5, 5.5, 64 * 4000)
    u = np.exp2(-t).astype(np.float32).reshape(-1, 64)
    se, _, _ = oracle.encode_keys(
        u.astype(np.float16).view(np.uint16),
        key_scale=np.ones(u.shape[0], np.float32))
    _, e, _ = unpack(se, None, 0)
    uf = u.astype(np.float16).astype(np.float64)
    rel = np.exp2(-e.astype(np.float64)) / uf - 1.0
    assert abs(math.sqrt(np.mean(rel**2)) - rms) < 2e-3


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_mantissa_mean_set_bits(k):
    # Sec. II-D: mean cost 1 + k/2 shifts, i.e. about k/2 set mantissa bits
    rng = np.random.default_rng(7)
    t = rng.uniform(0.5, 5.5, 64 * 2000)
    u = np.exp2(-t).astype(np.float32).reshape(-1, 64)
    se, cm, _ = oracle.encode_keys(u.astype(np.float16).view(np.uint16),
                                   mant_bits=k,
                                   key_scale=np.ones(u.shape[0], np.float32))
    _, e, j = unpack(se, cm, k)
    bits = np.array([bin(v).count("1") for v in j[e != 7].ravel()])
    assert abs(bits.mean() - k / 2) < 0.1 * k + 0.05


@pytest.mark.parametrize("k", [0, 2, 4])
def test_sign_symmetry_and_zero_rows(k):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((64, 64)).astype(np.float16)
    x[5] = 0  # an all-zero row
    a = oracle.encode_keys(x.view(np.uint16), mant_bits=k)
    b = oracle.encode_keys((-x).view(np.uint16), mant_bits=k)
    na, ea, ja = unpack(a[0], a[1], k)
    nb, eb, jb = unpack(b[0], b[1], k)
    assert np.array_equal(ea, eb) and np.array_equal(ja, jb)
    nz = ea != 7
    assert np.array_equal(na[nz], 1 - nb[nz])
    assert a[2][5] == 0 and (ea[5] == 7).all() and not ja[5].any()


def test_mantissa_decodes_closer_than_pot4():
    rng = np.random.default_rng(13)
    x = rng.standard_normal((256, 64)).astype(np.float16)
    xf = x.astype(np.float64)
    errs = []
    for k in [0, 1, 2, 4]:
        se, cm, sc = oracle.encode_keys(x.view(np.uint16), mant_bits=k)
        neg, e, j = unpack(se, cm if k else np.zeros((256, 0), np.uint8), k)
        val = np.where(e == 7, 0.0, (1 - 2 * neg) * decoded_ratio(e, j, k)) \
            * sc[:, None]
        errs.append(np.sqrt(np.mean((val - xf) ** 2)))
    assert errs[0] > errs[1] > errs[2] > errs[3]


def test_hadamard_matrix_and_key_rotation_exact():
    H = scipy.linalg.hadamard(64)
    assert np.array_equal(H @ H.T, 64 * np.eye(64, dtype=H.dtype))
    rng = np.random.default_rng(17)
    x = (rng.standard_normal((8, 64)) * 3).astype(np.float16)
    rot = oracle.rotate_keys(x.view(np.uint16))
    for r in range(8):
        # fp16 values are integer multiples of 2^-24
        ints = [int(Fraction(float(v)) * 2**24) for v in x[r].astype(np.float64)]
        for i in range(64):
            exact = Fraction(sum(int(H[i, jj]) * ints[jj] for jj in range(64)),
                             8 * 2**24)
            assert rot[r, i] == np.float32(float(exact))


def test_hadamard_query_fwht():
    H = scipy.linalg.hadamard(64)
    rng = np.random.default_rng(19)
    for _ in range(20):
        q = rng.standard_normal(64).astype(np.float32)
        out = oracle.fwht_query(q)
        exact = [Fraction(sum(int(H[i, jj]) * Fraction(float(q[jj]))
                              for jj in range(64)), 8) for i in range(64)]
        ex32 = np.array([np.float32(float(v)) for v in exact], np.float32)
        # within one fp32 ulp of the exact rotation
        ulp = np.spacing(np.abs(ex32))
        assert (np.abs(out.astype(np.float64) - ex32) <= ulp).all()
    # limited exponent range: the fp64 butterfly is exact, one rounding only
    q = (rng.integers(-2**20, 2**20, 64) / 2.0**10).astype(np.float32)
    out = oracle.fwht_query(q)
    exact = (H.astype(np.int64) @ (q.astype(np.float64) * 2**10).astype(np.int64))
    assert np.array_equal(out, (exact / (8.0 * 2**10)).astype(np.float32))
