"""GPU parity of the CU-wide variant of the decode kernels
(pot_debug.force_wg_waves): one workgroup of 16 waves (12 at k = 3, 4 for the
shift-accumulate kernels; 16 or 12 for the decoded-code engines, 12 for the
INT8 comparator) per (split, kv head, batch) whose waves claim the split's
64-key tiles from a counter in LDS. Same bar as the four-wave kernels: q^, Delta, int32 scores,
the final and per-split integer maxima bit-exact against the oracle, O within
2e-3; with ragged lengths, fewer tiles than waves, several splits, every
mantissa width and group size, Hadamard, the fused append, and against the
four-wave kernel on the same inputs (agreement to fp32 rounding: the order of
the sums depends on which wave claimed which tile).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_09208_amd as pa
from parity_util import DEV, O_TOL, assert_pot_parity, gpu_encode, gpu_pot_decode, store_values, to_dev
from test_gpu_values_int8 import assert_v8_parity
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


# the other engines' CU-wide variants: decoded-code engines over fp16 values
@pytest.mark.parametrize("engine,k,waves", [("ds4a", 0, 12), ("dot", 1, 16), ("dot", 4, 16)])
def test_pool_decoded_code_engines(engine, k, waves):
    d = make_decode_inputs(880 + k, B=2, Hq=16, Hkv=2, T=3100)
    err, g = assert_pot_parity(d, mant_bits=k, engine=engine, force_splits=2, wg_waves=waves)
    print(f"pool {engine} k={k} waves={g['wg_waves']} O err {err:.2e}")


# INT8 values: shift-accumulate (engine 0) and byte decode (engine 1), with
# softmax weights and with power-of-two weights
@pytest.mark.parametrize("engine,k,pow2,waves", [(0, 0, False, 16), (0, 4, False, 12),
                                                 (1, 0, False, 16), (0, 1, True, 16),
                                                 (1, 0, True, 12)])
def test_pool_int8_values(engine, k, pow2, waves):
    d = make_decode_inputs(890 + 10 * engine + k, B=2, Hq=16, Hkv=2, T=2700, t_cap=2704)
    err, n = assert_v8_parity(d, engine=engine, mant_bits=k, force_splits=2, pow2=pow2,
                              wg_waves=waves)
    print(f"pool v8 engine={engine} k={k} pow2={pow2} O err {err:.2e}")


def test_pool_int8_comparator():
    B, Hq, Hkv, T = 2, 32, 4, 3000
    d = make_decode_inputs(899, B=B, Hq=Hq, Hkv=Hkv, T=T)
    tc = d["t_cap"]
    rows = d["k_bits"].reshape(-1, 64)
    n = rows.shape[0]
    codes = torch.empty((n, 64), dtype=torch.int8, device=DEV)
    sc = torch.empty(n, dtype=torch.float32, device=DEV)
    pa.pot_int8_encode_keys(to_dev(rows).view(torch.float16), n, 1, 0, sc, codes)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, 2), DEV)
    dbg = pa.pot_debug()
    taps = dict(scores=torch.empty((B, Hq, T), dtype=torch.int32, device=DEV),
                m_final=torch.empty((B, Hq), dtype=torch.int32, device=DEV))
    for k_, t_ in taps.items():
        setattr(dbg, k_, t_.data_ptr())
    dbg.force_splits = 2
    dbg.force_wg_waves = 12
    pa.pot_int8_decode_attention(to_dev(d["q"]), codes, sc, store_values(d["v_bits"], B, Hkv, tc),
                                 tc, d["kv_head_of_q"], B, Hq, Hkv, T, 0, out, ws, dbg=dbg)
    torch.cuda.synchronize()
    assert dbg.wg_waves == 12
    oc, osc = oracle.int8_encode_keys(rows)
    r = oracle.int8_decode(d["q"], oc, osc, d["v_bits"], tc, d["kv_head_of_q"], B, Hq, Hkv, T)
    assert np.array_equal(taps["scores"].cpu().numpy(), r["scores"])
    assert np.array_equal(taps["m_final"].cpu().numpy(), r["m_final"])
    err = float(np.abs(out.cpu().numpy() - r["out"]).max())
    assert err <= O_TOL, err
    print(f"pool INT8 comparator O err {err:.2e}")
