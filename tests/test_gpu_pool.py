"""GPU parity of the CU-wide variant of the shift-accumulate decode kernels
(pot_debug.force_wg_waves): one workgroup of 16 waves (12 at k = 3, 4) per
(split, kv head, batch) whose waves claim the split's 64-key tiles from a
counter in LDS. Same bar as the four-wave kernels: q^, Delta, int32 scores,
the final and per-split integer maxima bit-exact against the oracle, O within
2e-3; with ragged lengths, fewer tiles than waves, several splits, every
mantissa width and group size, Hadamard, the fused append, and against the
four-wave kernel on the same inputs (agreement to fp32 rounding: the order of
the sums depends on which wave claimed which tile).
"""
import numpy as np
import pytest
import torch

import paper_2609_09208_amd as pa
from parity_util import DEV, assert_pot_parity, gpu_encode, gpu_pot_decode
from workloads import make_decode_inputs

pytestmark = pytest.mark.gpu


def pool_waves(k):
    return 16 if k <= 2 else 12


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_pool_every_mantissa_width_and_group(k, G):
    Hkv = 2
    d = make_decode_inputs(800 + 10 * k + G, B=2, Hq=G * Hkv, Hkv=Hkv, T=2900)
    err, g = assert_pot_parity(d, mant_bits=k, force_splits=1, wg_waves=pool_waves(k))
    print(f"pool k={k} G={G} waves={g['wg_waves']} O err {err:.2e}")


@pytest.mark.parametrize("T,t_cap", [(1, 8), (63, 64), (65, 72), (1000, 1032), (4100, 4104)])
def test_pool_ragged_and_few_tiles(T, t_cap):
    # T = 1 and 63: one tile for 16 waves; 65: two tiles, the second ragged
    d = make_decode_inputs(830 + T, B=2, Hq=16, Hkv=2, T=T, t_cap=t_cap)
    err, g = assert_pot_parity(d, force_splits=1, wg_waves=16)
    print(f"pool T={T} t_cap={t_cap} O err {err:.2e}")


@pytest.mark.parametrize("S", [2, 3, 7])
def test_pool_several_splits(S):
    d = make_decode_inputs(840 + S, B=2, Hq=32, Hkv=4, T=6000)
    err, g = assert_pot_parity(d, mant_bits=1, force_splits=S, wg_waves=16)
    tiles = -(-6000 // 256)  # splits are whole 256-key tiles
    assert g["n_splits"] == -(-tiles // -(-tiles // S))
    print(f"pool splits={g['n_splits']} O err {err:.2e}")


@pytest.mark.parametrize("k", [0, 4])
def test_pool_hadamard(k):
    d = make_decode_inputs(850 + k, B=2, Hq=16, Hkv=2, T=3000)
    err, _ = assert_pot_parity(d, mant_bits=k, hadamard=True, force_splits=2,
                               wg_waves=pool_waves(k))
    print(f"pool Hadamard k={k} O err {err:.2e}")


def test_pool_matches_four_wave_kernel():
    d = make_decode_inputs(860, B=3, Hq=32, Hkv=4, T=5000)
    se, cm, sc = gpu_encode(d["k_bits"].reshape(-1, 64), 2)
    a = gpu_pot_decode(d, se, cm, sc, mant_bits=2, force_splits=2, wg_waves=4)
    b = gpu_pot_decode(d, se, cm, sc, mant_bits=2, force_splits=2, wg_waves=16)
    assert a["wg_waves"] == 4 and b["wg_waves"] == 16
    for key in ("qhat", "scores", "m_final", "m_split"):
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(a["delta"].view(np.uint32), b["delta"].view(np.uint32))
    diff = float(np.abs(a["out"] - b["out"]).max())
    assert diff <= 1e-5, diff
    print(f"pool vs four waves: taps bit-identical, O differs by {diff:.1e}")


def test_pool_rejects_other_wave_counts():
    d = make_decode_inputs(870, B=1, Hq=8, Hkv=1, T=300)
    se, cm, sc = gpu_encode(d["k_bits"].reshape(-1, 64), 0)
    for bad in (8, 12, 5, -1):
        with pytest.raises(pa.PotError):
            gpu_pot_decode(d, se, cm, sc, force_splits=1, wg_waves=bad)
