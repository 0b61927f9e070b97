"""GPU parity of the byte-decode score path (pot_ds4a_decode_attention).

The path decodes PoT-4 code nibbles to int8 sigma 2^(6-e) bytes and scores
them with v_dot4 (a software form of the packed shift-dot of Sec. III,
eq. ds4a). Its int32 scores must be exactly those of the shift-accumulate
definition, so the bar is the same as for pot_decode_attention: codes,
q^, Delta, scores and integer maxima bit-exact against the oracle, O within
2e-3, at sizes spanning several tiles and ragged tails, with the edge cases.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_09208_amd as pa
from parity_util import DEV, O_TOL, assert_pot_parity, gpu_encode, gpu_pot_decode
from workloads import make_decode_inputs, make_decode_inputs_device

pytestmark = pytest.mark.gpu


def test_ds4a_tinyllama_layer_t4096():
    d = make_decode_inputs(2, B=1, Hq=32, Hkv=4, T=4096)
    err, g = assert_pot_parity(d, engine="ds4a")
    print(f"ds4a T=4096 splits={g['n_splits']} O err {err:.3e}")


@pytest.mark.parametrize("T,t_cap", [(1, 8), (255, 256), (257, 320), (4099, 4104)])
def test_ds4a_ragged(T, t_cap):
    d = make_decode_inputs(60 + T, B=2, Hq=8, Hkv=2, T=T, t_cap=t_cap)
    assert_pot_parity(d, engine="ds4a")


@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (4, 2), (8, 2), (16, 16)])
def test_ds4a_group_sizes(Hq, Hkv):
    d = make_decode_inputs(70 + Hq, B=2, Hq=Hq, Hkv=Hkv, T=300)
    assert_pot_parity(d, engine="ds4a")


@pytest.mark.parametrize("F", [6, 12])
def test_ds4a_head_room(F):
    d = make_decode_inputs(80 + F, B=1, Hq=8, Hkv=1, T=600)
    assert_pot_parity(d, frac_bits=F, engine="ds4a")


def test_ds4a_hadamard_and_forced_splits():
    d = make_decode_inputs(90, B=2, Hq=8, Hkv=1, T=2000)
    assert_pot_parity(d, hadamard=True, force_splits=3, engine="ds4a")


def test_ds4a_degenerate_rows_and_query():
    d = make_decode_inputs(91, B=2, Hq=8, Hkv=1, T=300)
    k = d["k_bits"].reshape(2, 1, -1, 64)
    k[0, 0, 5] = 0          # all-zero key row (s = 0, all zero codes)
    k[1, 0, :50] = 0
    d["q"][1, 3] = 0.0      # zero query (q^ = 0, Delta = 0)
    assert_pot_parity(d, engine="ds4a")


def test_ds4a_scores_equal_shift_path():
    d = make_decode_inputs(92, B=2, Hq=32, Hkv=4, T=1500)
    rows = d["k_bits"].reshape(-1, 64)
    se, _, sc = gpu_encode(rows)
    a = gpu_pot_decode(d, se, None, sc, engine="sac")
    b = gpu_pot_decode(d, se, None, sc, engine="ds4a")
    assert np.array_equal(a["scores"], b["scores"])
    assert np.array_equal(a["m_final"], b["m_final"])
    assert float(np.abs(a["out"] - b["out"]).max()) <= 1e-5


def test_ds4a_full_size_b64_t32768_sampled():
    """Full-size launch as the benchmark times it; sampled slices vs the oracle."""
    B, T, Hq, Hkv = 64, 32768, 32, 4
    d = make_decode_inputs_device(12, B, Hq, Hkv, T, DEV)
    fmt = pa.make_format()
    cache = pa.alloc_pot_cache(B, Hkv, T, 0, DEV)
    pa.pot_encode_keys(fmt, d["k"], B * Hkv * T, 1, 0, cache["key_scale"], cache["codes_se"],
                       None)
    v = pa.alloc_value_cache(B, Hkv, T, DEV)
    pa.pot_store_values(d["v"], B * Hkv, T, T, 0, v)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    pa.pot_ds4a_decode_attention(fmt, d["q"], cache["codes_se"], cache["key_scale"], v, T,
                                 d["kv_head_of_q"], B, Hq, Hkv, T, out, ws)
    torch.cuda.synchronize()
    G = Hq // Hkv
    worst = 0.0
    for (b, h) in [(0, 0), (31, 1), (63, 3)]:
        kb = d["k"][b, h].view(torch.uint16).cpu().numpy()
        vb = d["v"][b, h].view(torch.uint16).cpu().numpy()
        qs = d["q"][b, h * G:(h + 1) * G].cpu().numpy()
        o_se, _, o_sc = oracle.encode_keys(kb)
        r = oracle.pot_decode(qs[None], o_se, None, o_sc, vb, T, np.zeros(G, np.int32),
                              1, G, 1, T)
        worst = max(worst, float(np.abs(out[b, h * G:(h + 1) * G].cpu().numpy()
                                        - r["out"][0]).max()))
    assert worst <= O_TOL, worst
    print(f"ds4a B=64 T=32768 sampled O err {worst:.3e}")
