"""GPU parity of the decoded-weight score path (pot_dot_decode_attention).

PoT-Mk codes are decoded to 16-bit integer weights sigma (2^k + j) 2^(7-e)
and scored with v_dot2 (PoT-4 goes through the byte path of
pot_ds4a_decode_attention). The int32 scores are exactly those of eq. (sac)
with eq. (mant), so the bar is pot_decode_attention's: codes, q^, Delta,
scores and integer maxima bit-exact against the oracle, O within 2e-3, over
every mantissa width and head-group size, ragged tails, head-room, Hadamard,
forced splits and degenerate rows.
"""
import numpy as np
import pytest

from parity_util import assert_pot_parity, gpu_encode, gpu_pot_decode
from workloads import make_decode_inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (8, 4), (8, 2), (32, 4)])
def test_dot_every_mantissa_width_and_group(k, Hq, Hkv):
    d = make_decode_inputs(300 + 10 * k + Hq // Hkv, B=2, Hq=Hq, Hkv=Hkv, T=700)
    assert_pot_parity(d, mant_bits=k, engine="dot")


def test_dot_tinyllama_layer_t32768_potm1():
    d = make_decode_inputs(320, B=1, Hq=32, Hkv=4, T=32768)
    err, g = assert_pot_parity(d, mant_bits=1, engine="dot")
    print(f"dot PoT-M1 T=32768 splits={g['n_splits']} O err {err:.3e}")


def test_dot_batch8_hadamard_potm4_t2048():
    d = make_decode_inputs(321, B=8, Hq=32, Hkv=4, T=2048)
    err, g = assert_pot_parity(d, mant_bits=4, hadamard=True, engine="dot")
    print(f"dot Hadamard PoT-M4 B=8 T=2048 splits={g['n_splits']} O err {err:.3e}")


@pytest.mark.parametrize("T,t_cap", [(1, 8), (63, 64), (257, 320), (4099, 4104)])
@pytest.mark.parametrize("k", [1, 4])
def test_dot_ragged(T, t_cap, k):
    d = make_decode_inputs(330 + T + k, B=2, Hq=8, Hkv=2, T=T, t_cap=t_cap)
    assert_pot_parity(d, mant_bits=k, engine="dot")


@pytest.mark.parametrize("F", [6, 12])
def test_dot_head_room(F):
    d = make_decode_inputs(340 + F, B=1, Hq=8, Hkv=1, T=600)
    assert_pot_parity(d, mant_bits=2, frac_bits=F, engine="dot")


def test_dot_forced_splits_and_degenerate_rows():
    d = make_decode_inputs(350, B=2, Hq=8, Hkv=1, T=2000)
    k = d["k_bits"].reshape(2, 1, -1, 64)
    k[0, 0, 5] = 0          # all-zero key row (s = 0, all zero codes)
    k[1, 0, :50] = 0
    d["q"][1, 3] = 0.0      # zero query (q^ = 0, Delta = 0)
    assert_pot_parity(d, mant_bits=3, force_splits=7, engine="dot")


@pytest.mark.parametrize("k", [1, 4])
def test_dot_scores_equal_shift_path(k):
    d = make_decode_inputs(360 + k, B=2, Hq=32, Hkv=4, T=1500)
    rows = d["k_bits"].reshape(-1, 64)
    se, cm, sc = gpu_encode(rows, k)
    a = gpu_pot_decode(d, se, cm, sc, mant_bits=k, engine="sac")
    b = gpu_pot_decode(d, se, cm, sc, mant_bits=k, engine="dot")
    assert np.array_equal(a["scores"], b["scores"])
    assert np.array_equal(a["m_final"], b["m_final"])
    assert float(np.abs(a["out"] - b["out"]).max()) <= 1e-5
