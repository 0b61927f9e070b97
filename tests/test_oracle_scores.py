"""Pins for the oracle's query quantiser and exact SAC scores.

Sec. II-A (INT8 query, per-vector step), Sec. II-B eq. (sac), Sec. II-C
eq. (exact), Sec. I-A (binary attention = PoT restricted to e = 0).

Checks are independent of how the oracle computes: the quantiser against its
error bound, scores against brute-force integer matrix products of the decoded
operands (numpy int64 matmul), the printed accumulator bound, the binary
special case, the left-shift invariant and the real-valued dot product.
"""
import json
import os

import numpy as np
import pytest

import oracle
from workloads import make_decode_inputs

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                   "paper_constants.json")))


def unpack(se, cm, k):
    rows = se.shape[0]
    m = np.arange(64)
    nib = (se[:, m // 2] >> (4 * (m % 2))) & 15
    neg, e = (nib >> 3) & 1, nib & 7
    j = np.zeros((rows, 64), np.int64)
    for b in range(k):
        j |= ((cm[:, 8 * b + m // 8] >> (m % 8)) & 1).astype(np.int64) << b
    return neg, e, j


def key_integers(se, cm, k, F):
    """Integer key values sigma (2^k + j) 2^(F - e) (0 for the zero code)."""
    neg, e, j = unpack(se, cm, k)
    mag = (2**k + j) * (2 ** np.maximum(F - e, 0))
    return np.where(e == 7, 0, np.where(neg == 1, -mag, mag)).astype(np.int64)


def test_query_quantiser_error_bound():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((200, 64)).astype(np.float32)
    q[3] *= 1e-30
    q[4] *= 1e20
    qh, dl, _ = oracle.quantize_query(q)
    amax = np.abs(q).max(axis=1)
    assert np.allclose(dl, amax / 127, rtol=2e-7, atol=0)
    assert np.abs(qh).max() <= 127
    r = np.arange(200)
    assert (np.abs(qh[r, np.abs(q).argmax(axis=1)]) == 127).all()
    # rounding error of a correctly rounded quantiser: |q - D q^| <= D/2 (+ulp)
    err = np.abs(q.astype(np.float64) - dl[:, None].astype(np.float64) * qh)
    assert (err <= dl[:, None] * (0.5 + 1e-5)).all()


def _rn_f32(fr):
    """The fp32 nearest to the rational fr, ties to even, decided exactly."""
    from fractions import Fraction
    c = np.float32(float(fr))
    cands = [c, np.nextafter(c, np.float32(np.inf)), np.nextafter(c, np.float32(-np.inf))]
    best = min(cands, key=lambda f: (abs(Fraction(float(f)) - fr),
                                     int(np.float32(f).view(np.uint32)) & 1))
    return np.float32(best)


def test_query_step_is_the_correctly_rounded_quotient():
    """Delta = amax / 127 rounded once to fp32 (Sec. II-A: one step per vector),
    bit for bit against the exact rational quotient. The amax values are chosen
    so that amax * fl32(1/127) rounds differently, and so that a double-rounded
    quotient would too, where such values exist among the samples."""
    from fractions import Fraction
    rng = np.random.default_rng(11)
    cand = rng.uniform(0.1, 1e4, 20000).astype(np.float32)
    recip = np.float32(1.0) / np.float32(127.0)
    differ = cand[(cand * recip) != (cand / np.float32(127.0))][:40]
    assert len(differ) >= 20
    amax = np.concatenate([differ, np.float32([127.0, 1.0, 3.0e-38, 3.0e38])])
    q = np.zeros((len(amax), 64), np.float32)
    q[:, 5] = amax
    q[:, 9] = -amax / np.float32(3.0)
    _, dl, _ = oracle.quantize_query(q)
    for a, d in zip(amax.tolist(), dl.tolist()):
        want = _rn_f32(Fraction(a) / 127)
        assert np.float32(d).view(np.uint32) == want.view(np.uint32), (a, d, want)


def test_query_quantiser_ties_round_to_even():
    """amax = 127 makes the scale 127/amax exactly 1, so q^ is q rounded to
    the nearest integer with ties to even (Sec. II-A, INT8 query): 2.5 -> 2,
    3.5 -> 4, -2.5 -> -2, 0.5 -> 0, 126.5 -> 126; the clamp keeps 127."""
    q = np.zeros((1, 64), np.float32)
    vals = {0: 127.0, 1: 2.5, 2: 3.5, 3: -2.5, 4: -3.5, 5: 0.5, 6: -0.5, 7: 1.5,
            8: 126.5, 9: -126.5, 10: 2.4999998, 11: 2.5000002, 12: -1.5, 13: 4.5}
    want = {0: 127, 1: 2, 2: 4, 3: -2, 4: -4, 5: 0, 6: 0, 7: 2, 8: 126, 9: -126,
            10: 2, 11: 3, 12: -2, 13: 4}
    for m, v in vals.items():
        q[0, m] = v
    qh, dl, _ = oracle.quantize_query(q)
    assert dl[0] == np.float32(1.0)
    for m, w in want.items():
        assert int(qh[0, m]) == w, (m, vals[m], int(qh[0, m]))


def test_query_quantiser_zero_vector():
    qh, dl, _ = oracle.quantize_query(np.zeros((2, 64), np.float32))
    assert not qh.any() and not dl.any()


@pytest.mark.parametrize("k,F", [(0, 7), (0, 6), (1, 7), (2, 7), (4, 7),
                                 (4, 12), (0, 12)])
def test_scores_equal_bruteforce_integer_dot(k, F):
    d = make_decode_inputs(21 + k, B=2, Hq=4, Hkv=2, T=37)
    rows = d["k_bits"].reshape(-1, 64)
    se, cm, sc = oracle.encode_keys(rows, mant_bits=k)
    r = oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], d["t_cap"],
                          d["kv_head_of_q"], 2, 4, 2, 37, mant_bits=k,
                          frac_bits=F)
    kint = key_integers(se, cm if k else np.zeros((len(se), 0), np.uint8), k,
                        F).reshape(2, 2, d["t_cap"], 64)[:, :, :37]
    for b in range(2):
        for i in range(4):
            h = d["kv_head_of_q"][i]
            ref = kint[b, h] @ r["qhat"][b, i].astype(np.int64)
            assert np.array_equal(ref, r["scores"][b, i])


def test_scores_track_the_real_dot_product():
    # S^ = Delta s 2^-(F+k) acc approximates q . K within the code error
    d = make_decode_inputs(5, B=1, Hq=8, Hkv=1, T=400)
    rows = d["k_bits"].reshape(-1, 64)
    kf = rows.view(np.float16).astype(np.float64)
    for k, tol in [(0, 0.25), (4, 0.03)]:
        se, cm, sc = oracle.encode_keys(rows, mant_bits=k)
        r = oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], d["t_cap"],
                              d["kv_head_of_q"], 1, 8, 1, 400, mant_bits=k)
        s_hat = (r["delta"][0][:, None].astype(np.float64) * sc[None, :]
                 * r["scores"][0] * 2.0 ** -(7 + k))
        s_true = d["q"][0].astype(np.float64) @ kf.T
        rel = np.linalg.norm(s_hat - s_true) / np.linalg.norm(s_true)
        assert rel < tol, (k, rel)


def test_binary_attention_special_case():
    # all |K_m| equal -> every code has e = 0 -> acc = 2^F sum sigma q^
    rng = np.random.default_rng(2)
    sign = rng.choice([-1.0, 1.0], size=(16, 64))
    kb = (sign * 0.75).astype(np.float16)
    se, cm, sc = oracle.encode_keys(kb.view(np.uint16))
    _, e, _ = unpack(se, None, 0)
    assert (e == 0).all()
    q = rng.standard_normal((1, 1, 64)).astype(np.float32)
    v = np.zeros((16, 64), np.float16).view(np.uint16)
    r = oracle.pot_decode(q, se, None, sc, v, 16, np.zeros(1, np.int32),
                          1, 1, 1, 16)
    expect = 2**7 * (sign.astype(np.int64) @ r["qhat"][0, 0].astype(np.int64))
    assert np.array_equal(r["scores"][0, 0], expect)


def test_accumulator_bound_is_the_printed_one():
    g = GOLD["acc_bound_d64_F7"]
    q = np.ones((1, 1, 64), np.float32)  # q^ = 127 everywhere
    kb = np.ones((1, 64), np.float16)    # every code e = 0, sigma = +1
    se, _, sc = oracle.encode_keys(kb.view(np.uint16))
    r = oracle.pot_decode(q, se, None, sc, np.zeros((1, 64), np.uint16), 1,
                          np.zeros(1, np.int32), 1, 1, 1, 1)
    assert r["scores"][0, 0, 0] == g["exact"] == 64 * 127 * 2**7
    assert abs(g["exact"] - g["printed"]) / g["printed"] < 0.005
    r = oracle.pot_decode(-q, se, None, sc, np.zeros((1, 64), np.uint16), 1,
                          np.zeros(1, np.int32), 1, 1, 1, 1)
    assert r["scores"][0, 0, 0] == -g["exact"]


def test_left_shift_invariant_refuses_F_below_E():
    # F = 5 < E = 6: a code with e = 6 would need a right shift (eq. exact)
    kb = np.full((1, 64), 2.0**-6, np.float16)
    kb[0, 0] = 1.0
    se, _, sc = oracle.encode_keys(kb.view(np.uint16))
    _, e, _ = unpack(se, None, 0)
    assert e.max() == 6
    args = (np.ones((1, 1, 64), np.float32), se, None, sc,
            np.zeros((1, 64), np.uint16), 1, np.zeros(1, np.int32), 1, 1, 1, 1)
    oracle.pot_decode(*args, frac_bits=6)
    with pytest.raises(ValueError):
        oracle.pot_decode(*args, frac_bits=5)


def test_head_room_F_only_rescales():
    d = make_decode_inputs(8, B=1, Hq=2, Hkv=1, T=50)
    rows = d["k_bits"].reshape(-1, 64)
    se, cm, sc = oracle.encode_keys(rows, mant_bits=2)
    res = [oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], d["t_cap"],
                             d["kv_head_of_q"], 1, 2, 1, 50, mant_bits=2,
                             frac_bits=F) for F in (6, 7, 9)]
    assert np.array_equal(res[0]["scores"] * 2, res[1]["scores"])
    assert np.array_equal(res[1]["scores"] * 4, res[2]["scores"])
    assert np.array_equal(res[0]["x"], res[1]["x"])
    assert np.array_equal(res[1]["x"], res[2]["x"])


def test_int8_oracle_scores_bruteforce():
    d = make_decode_inputs(31, B=1, Hq=4, Hkv=2, T=29)
    rows = d["k_bits"].reshape(-1, 64)
    codes, sc = oracle.int8_encode_keys(rows)
    xf = rows.view(np.float16).astype(np.float32)
    assert np.allclose(sc, np.abs(xf).max(axis=1) / 127, rtol=2e-7)
    err = np.abs(xf - sc[:, None] * codes.astype(np.float32))
    assert (err <= sc[:, None] * 0.5001).all()
    tc = d["t_cap"]
    r = oracle.int8_decode(d["q"], codes, sc, d["v_bits"], tc,
                           d["kv_head_of_q"], 1, 4, 2, 29)
    c = codes.reshape(2, tc, 64)[:, :29].astype(np.int64)
    for i in range(4):
        h = d["kv_head_of_q"][i]
        assert np.array_equal(c[h] @ r["qhat"][0, i].astype(np.int64),
                              r["scores"][0, i])


def test_log2_domain_score_follows_the_recorded_fp32_order():
    # the paper leaves the fp32 order open; the order fixed here is x = fl32(fl32(float(acc) * s) * c),
    # c = fl32(fl32(Delta * log2e_f32) * 2^-(F+k+3)); the GPU must match it
    d = make_decode_inputs(12, B=1, Hq=2, Hkv=1, T=500, t_cap=500)
    rows = d["k_bits"].reshape(-1, 64)
    for k in (0, 4):
        se, cm, sc = oracle.encode_keys(rows, mant_bits=k)
        r = oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], d["t_cap"],
                              d["kv_head_of_q"], 1, 2, 1, 500, mant_bits=k)
        log2e = np.float32(np.log2(np.e))
        assert log2e.view(np.uint32) == 0x3FB8AA3B
        for i in range(2):
            c = np.float32(r["delta"][0, i] * log2e) * np.float32(2.0 ** -(7 + k + 3))
            x = (r["scores"][0, i].astype(np.float32) * sc) * np.float32(c)
            assert np.array_equal(x, r["x"][0, i])
