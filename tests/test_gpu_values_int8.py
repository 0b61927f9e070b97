"""GPU parity of the INT8 value cache (pot_store_values_int8) and of decode
attention over it (pot_decode_attention_v8, both score engines).

Bar: the stored value bytes and exponents equal the oracle's quantiser bit for
bit; q^, Delta, int32 scores and integer maxima equal the oracle's (they do
not depend on the values); O is within 2e-3 of the oracle's fp64 decode over
the dequantised values v^ 2^-g. Rows with very different magnitudes inside
one split exercise the per-workgroup reference exponent g_ref: with every
row at or below unit scale the bar is the same 2e-3; with rows up to 2^12
times larger, O itself reaches 1e4, where one fp32 ulp is already 1e-3, so
the bar there is V8_REL_TOL times the largest value magnitude.
Tokens past T hold poison values in every sequence.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_09208_amd as pa
from parity_util import DEV, O_TOL, gpu_encode, to_dev
from workloads import make_decode_inputs, make_decode_inputs_device

pytestmark = pytest.mark.gpu

# Bound on |O - O_oracle| / max|v| when the values are far from unit scale:
# fp32 resolves 2^-24 of max|v|; the sums carry the byte-to-fp16 offset 1152
# next to codes of at most 127 (a factor of 9), and the weights are split in
# two fp16 parts whose products and sums round a few times more: 2^-24 * 9 * 4.
V8_REL_TOL = 2.0e-6


def _deinterleave(v_u8, B, Hkv, t_cap):
    """[B, Hkv, t_cap, 64] token-interleaved bytes -> row-major int8 codes."""
    a = v_u8.reshape(B * Hkv, t_cap // 8, 64, 8).transpose(0, 1, 3, 2)
    return (a.reshape(B * Hkv * t_cap, 64).astype(np.int16) - 128).astype(np.int8)


def gpu_store_int8(v_bits, B, Hkv, t_cap):
    src = to_dev(np.ascontiguousarray(v_bits).reshape(B * Hkv, t_cap, 64)).view(torch.float16)
    vu, ve = pa.alloc_value_cache_int8(B, Hkv, t_cap, DEV)
    pa.pot_store_values_int8(src, B * Hkv, t_cap, t_cap, 0, vu, ve)
    return vu, ve


def _taps(B, Hq, T):
    max_s = -(-T // 256)
    bufs = dict(qhat=torch.empty((B, Hq, 64), dtype=torch.int8, device=DEV),
                delta=torch.empty((B, Hq), dtype=torch.float32, device=DEV),
                scores=torch.empty((B, Hq, T), dtype=torch.int32, device=DEV),
                m_final=torch.empty((B, Hq), dtype=torch.int32, device=DEV),
                m_split=torch.empty((B, Hq, max_s), dtype=torch.int32, device=DEV))
    dbg = pa.pot_debug()
    for k, t in bufs.items():
        setattr(dbg, k, t.data_ptr())
    return dbg, bufs


def assert_v8_parity(d, engine=0, mant_bits=0, hadamard=False, force_splits=0, tol=O_TOL,
                     pow2=False, wg_waves=0):
    B, Hq, Hkv, T, t_cap = d["B"], d["Hq"], d["Hkv"], d["T"], d["t_cap"]
    rows = d["k_bits"].reshape(-1, 64)
    se, cm, sc = gpu_encode(rows, mant_bits, hadamard)
    o_se, o_cm, o_sc = oracle.encode_keys(rows, mant_bits=mant_bits, hadamard=hadamard)
    assert np.array_equal(se, o_se)
    # values: bytes and exponents against the oracle quantiser
    vu, ve = gpu_store_int8(d["v_bits"], B, Hkv, t_cap)
    torch.cuda.synchronize()
    o_vh, o_g = oracle.quantize_values(d["v_bits"].reshape(-1, 64))
    assert np.array_equal(_deinterleave(vu.cpu().numpy(), B, Hkv, t_cap), o_vh), "value codes"
    assert np.array_equal(ve.cpu().numpy().reshape(-1), o_g), "value exponents"
    fmt = pa.make_format(mant_bits, 7, hadamard)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    nws = pa.pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, force_splits) \
        if force_splits else pa.pot_decode_workspace_bytes(B, Hq, Hkv, T)
    ws = pa.alloc_workspace(nws, DEV)
    dbg, bufs = _taps(B, Hq, T)
    dbg.force_splits = force_splits
    dbg.force_wg_waves = wg_waves
    call = pa.pot_decode_attention_v8_pow2 if pow2 else pa.pot_decode_attention_v8
    call(fmt, engine, to_dev(d["q"]), to_dev(se), to_dev(cm) if cm is not None else None,
         to_dev(sc), vu, ve, t_cap, d["kv_head_of_q"], B, Hq, Hkv, T, out, ws, dbg=dbg)
    torch.cuda.synchronize()
    if wg_waves:
        assert dbg.wg_waves == wg_waves, (dbg.wg_waves, wg_waves)
    o = oracle.pot_decode_v8(d["q"], o_se, o_cm, o_sc, o_vh, o_g, t_cap, d["kv_head_of_q"],
                             B, Hq, Hkv, T, mant_bits=mant_bits, hadamard=hadamard,
                             split_len=dbg.split_len, pow2=pow2)
    assert np.array_equal(bufs["qhat"].cpu().numpy(), o["qhat"])
    assert np.array_equal(bufs["scores"].cpu().numpy(), o["scores"]), "int32 scores"
    assert np.array_equal(bufs["m_final"].cpu().numpy(), o["m_final"]), "M"
    ms = bufs["m_split"].cpu().numpy().reshape(-1)[:B * Hq * dbg.n_splits]
    assert np.array_equal(ms.reshape(B, Hq, dbg.n_splits), o["m_split"]), "per-split M"
    err = float(np.abs(out.cpu().numpy() - o["out"]).max())
    assert err <= tol, (err, tol)
    return err, dbg.n_splits


def test_store_int8_partial_range_leaves_the_rest():
    B, Hkv, t_cap = 2, 2, 64
    d = make_decode_inputs(500, B=B, Hq=4, Hkv=Hkv, T=t_cap)
    vu, ve = gpu_store_int8(d["v_bits"], B, Hkv, t_cap)
    before_u, before_e = vu.clone(), ve.clone()
    new = make_decode_inputs(501, B=B, Hq=4, Hkv=Hkv, T=t_cap)["v_bits"][:, :, 20:27]
    src = to_dev(np.ascontiguousarray(new).reshape(B * Hkv, 7, 64)).view(torch.float16)
    pa.pot_store_values_int8(src, B * Hkv, 7, t_cap, 20, vu, ve)
    torch.cuda.synchronize()
    mixed = d["v_bits"].copy()
    mixed[:, :, 20:27] = new
    o_vh, o_g = oracle.quantize_values(mixed.reshape(-1, 64))
    assert np.array_equal(_deinterleave(vu.cpu().numpy(), B, Hkv, t_cap), o_vh)
    assert np.array_equal(ve.cpu().numpy().reshape(-1), o_g)
    keep = np.ones((B, Hkv, t_cap), bool)
    keep[:, :, 20:27] = False
    assert np.array_equal(ve.cpu().numpy()[keep], before_e.cpu().numpy()[keep])


def test_store_int8_extreme_rows():
    B, Hkv, t_cap = 1, 1, 16
    v = np.zeros((B, Hkv, t_cap, 64), np.float16)
    v[0, 0, 0] = 65504.0                     # g = -10
    v[0, 0, 1, 3] = np.float16(2.0 ** -24)   # one subnormal: g = 30
    v[0, 0, 2] = -np.float16(2.0 ** -14)     # smallest normal
    v[0, 0, 3, :8] = [127, 2.5, 3.5, -2.5, 0.5, 1.5, 126.5, -127]  # ties at g = 0
    v[0, 0, 4] = np.linspace(-1000, 1000, 64).astype(np.float16)
    # row 5 stays all zero: g = 0, codes 0
    rng = np.random.default_rng(3)
    v[0, 0, 6:] = (rng.standard_normal((10, 64)) * 2.0 ** rng.integers(-20, 12, (10, 1)))
    bits = v.view(np.uint16)
    vu, ve = gpu_store_int8(bits, B, Hkv, t_cap)
    torch.cuda.synchronize()
    o_vh, o_g = oracle.quantize_values(bits.reshape(-1, 64))
    assert np.array_equal(_deinterleave(vu.cpu().numpy(), B, Hkv, t_cap), o_vh)
    assert np.array_equal(ve.cpu().numpy().reshape(-1), o_g)
    assert o_g[0] == -10 and o_g[1] == 30 and o_g[5] == 0


def test_v8_tinyllama_layer_t4096():
    d = make_decode_inputs(502, B=1, Hq=32, Hkv=4, T=4096)
    err, s = assert_v8_parity(d)
    print(f"INT8-V T=4096 splits={s} O err {err:.3e}")


@pytest.mark.parametrize("engine", [0, 1])
@pytest.mark.parametrize("T,t_cap", [(1, 8), (255, 264), (1000, 1024), (4099, 4104)])
def test_v8_ragged(engine, T, t_cap):
    d = make_decode_inputs(510 + T, B=2, Hq=8, Hkv=2, T=T, t_cap=t_cap)
    assert_v8_parity(d, engine=engine)


@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (4, 2), (16, 4), (32, 4)])
def test_v8_group_sizes(Hq, Hkv):
    d = make_decode_inputs(520 + Hq, B=2, Hq=Hq, Hkv=Hkv, T=700)
    assert_v8_parity(d)


@pytest.mark.parametrize("mant_bits,hadamard", [(1, False), (4, True)])
def test_v8_mantissa_and_hadamard(mant_bits, hadamard):
    d = make_decode_inputs(530 + mant_bits, B=2, Hq=32, Hkv=4, T=1500)
    assert_v8_parity(d, mant_bits=mant_bits, hadamard=hadamard)


@pytest.mark.parametrize("splits", [1, 3, 16])
def test_v8_forced_splits(splits):
    d = make_decode_inputs(540 + splits, B=1, Hq=32, Hkv=4, T=4000)
    assert_v8_parity(d, engine=1, force_splits=splits)


def _mixed_magnitudes(seed, lo, hi, zero_row=False):
    """Rows of the decode inputs scaled by 2^lo .. 2^hi (one power per row)."""
    T = 2000
    d = make_decode_inputs(seed, B=2, Hq=8, Hkv=2, T=T)
    rng = np.random.default_rng(seed + 1)
    v = d["v_bits"].view(np.float16).astype(np.float32)
    sc = np.exp2(rng.integers(lo, hi + 1, size=(2, 2, d["t_cap"], 1))).astype(np.float32)
    v[:, :, :T] = v[:, :, :T] * sc[:, :, :T]
    if zero_row:
        v[0, 0, 5] = 0.0      # an all-zero value row
    d["v_bits"] = v.astype(np.float16).view(np.uint16)
    return d, float(np.abs(v[:, :, :T]).max())


@pytest.mark.parametrize("engine", [0, 1])
def test_v8_mixed_magnitudes_across_a_split(engine):
    """Rows scaled by 2^-20 .. 2^12 inside one split: exponents g from about 30
    down to -10, so the weights p 2^(g_ref - g) span the whole range."""
    d, vmax = _mixed_magnitudes(550, -20, 12, zero_row=True)
    err, _ = assert_v8_parity(d, engine=engine, tol=max(O_TOL, V8_REL_TOL * vmax),
                              force_splits=2)
    print(f"INT8-V mixed magnitudes: O err {err:.3e} = {err / vmax:.2e} of max |v|")


@pytest.mark.parametrize("engine", [0, 1])
def test_v8_mixed_magnitudes_unit_scale(engine):
    """Rows scaled by 2^-20 .. 2^0 inside one split, held to the plain 2e-3."""
    d, vmax = _mixed_magnitudes(560, -20, 0, zero_row=True)
    err, _ = assert_v8_parity(d, engine=engine, force_splits=2)
    print(f"INT8-V unit-scale mixed magnitudes: O err {err:.3e}, max |v| {vmax:.2f}")


def test_v8_full_size_b64_t32768_sampled():
    """B = 64, T = 32768 with the planner's splits (the benchmark's launch),
    sampled (b, kv-head) slices against the oracle."""
    B, Hq, Hkv, T = 64, 32, 4, 32768
    d = make_decode_inputs_device(560, B, Hq, Hkv, T, DEV)
    fmt = pa.make_format(0)
    cache = pa.alloc_pot_cache(B, Hkv, T, 0, DEV)
    pa.pot_encode_keys(fmt, d["k"], B * Hkv * T, 1, 0, cache["key_scale"], cache["codes_se"],
                       None)
    vu, ve = pa.alloc_value_cache_int8(B, Hkv, T, DEV)
    pa.pot_store_values_int8(d["v"], B * Hkv, T, T, 0, vu, ve)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    G = Hq // Hkv
    worst = 0.0
    for engine in (0, 1):
        out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
        pa.pot_decode_attention_v8(fmt, engine, d["q"], cache["codes_se"], None,
                                   cache["key_scale"], vu, ve, T, d["kv_head_of_q"], B, Hq, Hkv,
                                   T, out, ws)
        torch.cuda.synchronize()
        for (b, h) in [(0, 0), (31, 1), (63, 3)]:
            vb = d["v"][b, h].view(torch.uint16).cpu().numpy()
            o_vh, o_g = oracle.quantize_values(vb)
            assert np.array_equal(_deinterleave(vu[b, h].cpu().numpy(), 1, 1, T), o_vh)
            assert np.array_equal(ve[b, h].cpu().numpy(), o_g)
            o_se, _, o_sc = oracle.encode_keys(d["k"][b, h].view(torch.uint16).cpu().numpy())
            qs = d["q"][b, h * G:(h + 1) * G].cpu().numpy()
            r = oracle.pot_decode_v8(qs[None], o_se, None, o_sc, o_vh, o_g, T,
                                     np.zeros(G, np.int32), 1, G, 1, T)
            err = float(np.abs(out[b, h * G:(h + 1) * G].cpu().numpy() - r["out"][0]).max())
            worst = max(worst, err)
    assert worst <= O_TOL, worst
    print(f"INT8-V B=64 T=32768 sampled O err {worst:.3e}")


# ---- power-of-two weights (eq. logsm A~ = 2^-k) over the INT8 values ----------------
@pytest.mark.parametrize("engine", [0, 1])
def test_pow2_tinyllama_layer_t4096(engine):
    d = make_decode_inputs(570 + engine, B=1, Hq=32, Hkv=4, T=4096)
    err, s = assert_v8_parity(d, engine=engine, pow2=True)
    print(f"pow2 weights engine {engine} T=4096 splits={s} O err {err:.3e}")


@pytest.mark.parametrize("T,t_cap", [(1, 8), (255, 264), (4099, 4104)])
def test_pow2_ragged(T, t_cap):
    d = make_decode_inputs(580 + T, B=2, Hq=8, Hkv=2, T=T, t_cap=t_cap)
    assert_v8_parity(d, pow2=True)


@pytest.mark.parametrize("splits", [1, 5, 16])
def test_pow2_forced_splits(splits):
    d = make_decode_inputs(590 + splits, B=1, Hq=32, Hkv=4, T=4000)
    assert_v8_parity(d, engine=1, force_splits=splits, pow2=True)


def test_pow2_mantissa_hadamard_and_groups():
    d = make_decode_inputs(600, B=2, Hq=16, Hkv=4, T=1500)
    assert_v8_parity(d, mant_bits=4, hadamard=True, pow2=True)


def test_pow2_mixed_magnitudes():
    d, vmax = _mixed_magnitudes(610, -20, 12)
    err, _ = assert_v8_parity(d, tol=max(O_TOL, V8_REL_TOL * vmax), force_splits=2,
                              pow2=True)
    print(f"INT8-V pow2 mixed magnitudes: O err {err:.3e} = {err / vmax:.2e} of max |v|")


def test_pow2_mixed_magnitudes_unit_scale():
    d, vmax = _mixed_magnitudes(620, -20, 0)
    err, _ = assert_v8_parity(d, force_splits=2, pow2=True)
    print(f"INT8-V pow2 unit-scale mixed magnitudes: O err {err:.3e}")


def test_pow2_full_size_b64_t32768_sampled():
    B, Hq, Hkv, T = 64, 32, 4, 32768
    d = make_decode_inputs_device(620, B, Hq, Hkv, T, DEV)
    fmt = pa.make_format(0)
    cache = pa.alloc_pot_cache(B, Hkv, T, 0, DEV)
    pa.pot_encode_keys(fmt, d["k"], B * Hkv * T, 1, 0, cache["key_scale"], cache["codes_se"],
                       None)
    vu, ve = pa.alloc_value_cache_int8(B, Hkv, T, DEV)
    pa.pot_store_values_int8(d["v"], B * Hkv, T, T, 0, vu, ve)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    pa.pot_decode_attention_v8_pow2(fmt, 0, d["q"], cache["codes_se"], None, cache["key_scale"],
                                    vu, ve, T, d["kv_head_of_q"], B, Hq, Hkv, T, out, ws)
    torch.cuda.synchronize()
    G = Hq // Hkv
    worst = 0.0
    for (b, h) in [(0, 0), (40, 2)]:
        vb = d["v"][b, h].view(torch.uint16).cpu().numpy()
        o_vh, o_g = oracle.quantize_values(vb)
        o_se, _, o_sc = oracle.encode_keys(d["k"][b, h].view(torch.uint16).cpu().numpy())
        qs = d["q"][b, h * G:(h + 1) * G].cpu().numpy()
        r = oracle.pot_decode_v8(qs[None], o_se, None, o_sc, o_vh, o_g, T, np.zeros(G, np.int32),
                                 1, G, 1, T, pow2=True)
        worst = max(worst, float(np.abs(out[b, h * G:(h + 1) * G].cpu().numpy() -
                                        r["out"][0]).max()))
    assert worst <= O_TOL, worst
    print(f"pow2 weights B=64 T=32768 sampled O err {worst:.3e}")
