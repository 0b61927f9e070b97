"""Pins for the oracle's integer-log2 softmax and A.V (Sec. II-E eq. logsm).

* the online form (integer running maximum, exact 2^dM rescales, exact split
  merge) equals the two-pass form for any tiling and split count;
* M = ceil(max x) is an integer with max x - M in (-1, 0], independent of the
  split count, and the per-split maxima reduce to it;
* the output equals a textbook softmax (float max, natural exp) of the
  dequantised scores over the fp16 values;
* the Hadamard rotation preserves unquantised scores;
* the fp16 baseline oracle equals a numpy softmax(q16 K^T / 8) V.
"""
import numpy as np
import pytest
import scipy.linalg

import oracle
from workloads import make_decode_inputs


def _pot(d, k=0, F=7, had=False, **kw):
    rows = d["k_bits"].reshape(-1, 64)
    se, cm, sc = oracle.encode_keys(rows, mant_bits=k, hadamard=had)
    r = oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], d["t_cap"],
                          d["kv_head_of_q"], d["B"], d["Hq"], d["Hkv"], d["T"],
                          mant_bits=k, frac_bits=F, hadamard=had, **kw)
    return r, sc


@pytest.mark.parametrize("T", [1, 7, 300])
def test_online_equals_two_pass(T):
    d = make_decode_inputs(40 + T, B=1, Hq=4, Hkv=1, T=T)
    ref, _ = _pot(d)
    for tile in (1, 7, 128, T):
        for split in (1, 3, 64):
            split_len = max(1, -(-T // split))
            r, _ = _pot(d, tile=tile, split_len=split_len)
            assert np.abs(r["out"] - ref["out"]).max() < 1e-12


def test_integer_max_properties():
    d = make_decode_inputs(3, B=2, Hq=4, Hkv=2, T=257)
    for split_len in (1, 16, 100, 257):
        r, _ = _pot(d, split_len=split_len)
        xm = r["x"].max(axis=2)
        assert r["m_final"].dtype == np.int32
        diff = xm.astype(np.float64) - r["m_final"]
        assert (diff <= 0).all() and (diff > -1).all()
        assert np.array_equal(r["m_split"].max(axis=2), r["m_final"])
        if split_len == 1:
            assert np.array_equal(r["m_split"], np.ceil(r["x"]).astype(np.int32))


@pytest.mark.parametrize("k,had", [(0, False), (1, False), (4, True)])
def test_output_is_textbook_softmax_of_dequantised_scores(k, had):
    d = make_decode_inputs(55, B=1, Hq=8, Hkv=2, T=333, t_cap=333)
    r, sc = _pot(d, k=k, had=had)
    v = d["v_bits"].view(np.float16).astype(np.float64)
    for i in range(8):
        h = d["kv_head_of_q"][i]
        s_hat = (np.float64(r["delta"][0, i]) * sc.reshape(2, 333)[h]
                 * r["scores"][0, i] * 2.0 ** -(7 + k))
        z = s_hat / 8.0
        w = np.exp(z - z.max())
        o = (w[:, None] * v[0, h]).sum(0) / w.sum()
        # x is rounded to fp32 in a pinned order; weights agree to ~1e-7
        assert np.abs(o - r["out"][0, i]).max() < 1e-5


def test_padding_rows_beyond_T_are_not_read():
    d = make_decode_inputs(6, B=2, Hq=2, Hkv=1, T=40, t_cap=64)
    r, _ = _pot(d)
    assert np.abs(r["out"]).max() < 10  # poison values are 60000


def test_hadamard_preserves_unquantised_scores():
    H = scipy.linalg.hadamard(64).astype(np.float64) / 8.0
    rng = np.random.default_rng(4)
    q = rng.standard_normal(64)
    K = rng.standard_normal((100, 64)) * rng.uniform(0.5, 4, 64)
    assert np.allclose((H @ q) @ (K @ H.T).T, q @ K.T, rtol=1e-12, atol=1e-10)
    qr = oracle.fwht_query(q.astype(np.float32)).astype(np.float64)
    kb = K.astype(np.float16)
    kr = oracle.rotate_keys(kb.view(np.uint16)).astype(np.float64)
    assert np.allclose(qr @ kr.T, q.astype(np.float32).astype(np.float64)
                       @ kb.astype(np.float64).T, rtol=1e-5, atol=1e-4)


def test_fp16_oracle_matches_numpy_softmax():
    d = make_decode_inputs(77, B=2, Hq=4, Hkv=2, T=65, t_cap=65)
    out = oracle.fp16_decode(d["q"], d["k_bits"], d["v_bits"], d["t_cap"],
                             d["kv_head_of_q"], 2, 4, 2, 65)
    k = d["k_bits"].view(np.float16).astype(np.float64)
    v = d["v_bits"].view(np.float16).astype(np.float64)
    q16 = d["q"].astype(np.float16).astype(np.float64)
    for b in range(2):
        for i in range(4):
            h = d["kv_head_of_q"][i]
            z = k[b, h] @ q16[b, i] / 8.0
            w = np.exp(z - z.max())
            assert np.allclose(out[b, i], w @ v[b, h] / w.sum(), atol=1e-12)


def test_fp16_conversion_matches_ieee():
    rng = np.random.default_rng(8)
    xs = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-9, 6, 3000),
                         [65504, 65519.99, 65520, 6.1e-5, 5.96e-8, 2.98e-8, 0.0, -0.0]])
    xs = xs.astype(np.float32)
    for x in xs:
        assert oracle.float_to_half(float(x)) == int(np.float16(x).view(np.uint16))
    for bits in range(0, 65536, 7):
        h = np.uint16(bits).view(np.float16)
        if np.isnan(h):
            continue
        assert oracle.half_to_float(bits) == float(h)
