"""Pins of the oracle's INT8 value quantiser and of its decode with INT8 values
(Sec. II-E: V as INT8 codes with a power-of-two per-token scale 2^-g).

The paper does not state how g and the codes are rounded; the reading is
g = the largest integer with max|v| 2^g <= 127 and v^ = round-half-even(v 2^g).
What pins it, independently of the oracle's own arithmetic:
* every finite fp16 value as a one-element row, against exact rationals;
* invariants: the row maximum lands in [64, 127], the error is at most half a
  step 2^-g-1, ties go to even, sign symmetry, doubling the row lowers g by 1;
* the decode with INT8 values equals the fp16-value decode exactly when every
  value is representable as v^ 2^-g, and differs from it by at most the
  largest quantisation error otherwise (O is a convex combination of rows).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workloads import make_decode_inputs


def _fp16_bits(x):
    return np.asarray(x, np.float16).view(np.uint16)


def test_every_fp16_value_as_a_one_element_row():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    finite = (bits & 0x7C00) != 0x7C00
    bits = bits[finite]
    rows = np.zeros((bits.size, 64), np.uint16)
    rows[:, 0] = bits
    rows[:, 5] = 0x8000  # a negative zero elsewhere in the row changes nothing
    vh, g = oracle.quantize_values(rows)
    assert np.all(vh[:, 1:] == 0)
    vals = bits.view(np.float16).astype(np.float64)
    for i in range(bits.size):
        x = Fraction(float(vals[i]))
        gi, ci = int(g[i]), int(vh[i, 0])
        if x == 0:
            assert (gi, ci) == (0, 0)
            continue
        a = abs(x)
        # g is the largest integer with |x| 2^g <= 127
        assert a * Fraction(2) ** gi <= 127 < a * Fraction(2) ** (gi + 1), (vals[i], gi)
        # the code is x 2^g rounded to the nearest integer, ties to even
        assert ci == round(x * Fraction(2) ** gi), (vals[i], gi, ci)


def test_row_invariants_on_seeded_rows():
    rng = np.random.default_rng(5)
    scales = 2.0 ** rng.integers(-20, 14, size=512)
    v = (rng.standard_normal((512, 64)) * scales[:, None]).astype(np.float16)
    v[7] = 0.0
    vh, g = oracle.quantize_values(_fp16_bits(v))
    vf = v.astype(np.float64)
    nz = np.abs(vf).max(axis=1) > 0
    amax_code = np.abs(vh.astype(np.int32)).max(axis=1)
    assert np.all((amax_code[nz] >= 64) & (amax_code[nz] <= 127))
    assert g[7] == 0 and np.all(vh[7] == 0)
    deq = vh.astype(np.float64) * np.exp2(-g.astype(np.float64))[:, None]
    assert np.all(np.abs(vf - deq) <= np.exp2(-g.astype(np.float64) - 1)[:, None])
    # sign symmetry
    vh_n, g_n = oracle.quantize_values(_fp16_bits(-v))
    assert np.array_equal(g_n, g) and np.array_equal(vh_n, -vh)
    # doubling the row (exact in fp16 where it stays finite) lowers g by one
    small = (np.abs(vf).max(axis=1) < 1e4) & nz
    vh_2, g_2 = oracle.quantize_values(_fp16_bits((v[small] * 2).astype(np.float16)))
    assert np.array_equal(g_2, g[small] - 1) and np.array_equal(vh_2, vh[small])


def test_ties_round_to_even():
    # max 127 -> g = 0, so the codes are the values rounded: 2.5 -> 2, 3.5 -> 4,
    # -2.5 -> -2, 0.5 -> 0, 1.5 -> 2, 126.5 -> 126
    row = np.zeros(64, np.float16)
    row[:7] = [127, 2.5, 3.5, -2.5, 0.5, 1.5, 126.5]
    vh, g = oracle.quantize_values(_fp16_bits(row[None]))
    assert g[0] == 0
    assert list(vh[0, :7]) == [127, 2, 4, -2, 0, 2, 126]
    # max 63.75: 63.75 * 2 = 127.5 > 127, so g stays 0 and 63.75 rounds to 64
    row = np.zeros(64, np.float16)
    row[0] = 63.75
    vh, g = oracle.quantize_values(_fp16_bits(row[None]))
    assert g[0] == 0 and vh[0, 0] == 64


def _exact_values(rng, B, Hkv, t_cap):
    """Values n 2^-g with n in [-127, 127], max |n| in [64, 127], g in 0..10:
    exact in fp16 and returned unchanged by the quantiser."""
    n = rng.integers(-127, 128, size=(B, Hkv, t_cap, 64))
    n[..., 0] = rng.integers(64, 128, size=(B, Hkv, t_cap)) * rng.choice([-1, 1], (B, Hkv, t_cap))
    gg = rng.integers(0, 11, size=(B, Hkv, t_cap))
    v = (n * np.exp2(-gg.astype(np.float64))[..., None]).astype(np.float16)
    assert np.array_equal(v.astype(np.float64), n * np.exp2(-gg.astype(np.float64))[..., None])
    return v, n.astype(np.int8), gg.astype(np.int8)


def _decode_both(d, v8, g, **kw):
    se, cm, sc = oracle.encode_keys(d["k_bits"].reshape(-1, 64), mant_bits=kw.get("mant_bits", 0))
    args = (d["q"], se, cm, sc)
    tail = (d["t_cap"], d["kv_head_of_q"], d["B"], d["Hq"], d["Hkv"], d["T"])
    r16 = oracle.pot_decode(*args, d["v_bits"], *tail, **kw)
    r8 = oracle.pot_decode_v8(*args, v8.reshape(-1, 64), g.reshape(-1), *tail, **kw)
    return r16, r8


def test_v8_decode_equals_fp16_decode_on_exact_values():
    rng = np.random.default_rng(9)
    d = make_decode_inputs(9, B=2, Hq=8, Hkv=2, T=300)
    v, n, gg = _exact_values(rng, 2, 2, d["t_cap"])
    d["v_bits"] = v.view(np.uint16)
    vh, g = oracle.quantize_values(d["v_bits"])
    assert np.array_equal(vh, n.reshape(-1, 64)) and np.array_equal(g, gg.reshape(-1))
    r16, r8 = _decode_both(d, vh, g)
    assert np.array_equal(r16["out"], r8["out"])
    assert np.array_equal(r16["scores"], r8["scores"])
    assert np.array_equal(r16["m_final"], r8["m_final"])


@pytest.mark.parametrize("tile", [1, 7, 128])
def test_v8_online_equals_two_pass(tile):
    d = make_decode_inputs(10, B=1, Hq=4, Hkv=1, T=513)
    vh, g = oracle.quantize_values(d["v_bits"])
    se, cm, sc = oracle.encode_keys(d["k_bits"].reshape(-1, 64))
    tail = (d["t_cap"], d["kv_head_of_q"], 1, 4, 1, 513)
    a = oracle.pot_decode_v8(d["q"], se, cm, sc, vh, g, *tail)
    b = oracle.pot_decode_v8(d["q"], se, cm, sc, vh, g, *tail, split_len=100, tile=tile)
    assert np.abs(a["out"] - b["out"]).max() < 1e-12


def test_v8_decode_within_the_quantisation_error():
    d = make_decode_inputs(11, B=2, Hq=8, Hkv=2, T=700)
    vh, g = oracle.quantize_values(d["v_bits"])
    r16, r8 = _decode_both(d, vh, g)
    # O is a convex combination of value rows in both, with the same weights
    v = d["v_bits"].view(np.float16).astype(np.float64).reshape(-1, 64)
    deq = vh.astype(np.float64) * np.exp2(-g.astype(np.float64))[:, None]
    live = np.zeros((2, 2, d["t_cap"]), bool)
    live[:, :, :700] = True
    bound = np.abs(v - deq)[live.reshape(-1)].max()
    err = np.abs(r16["out"] - r8["out"]).max()
    assert 0 < err <= bound + 1e-12, (err, bound)
