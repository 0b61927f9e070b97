"""Helpers for the GPU parity tests: run the HIP path through the C ABI and the
oracle on the same seeded inputs. The oracle never sees a GPU output: it gets
the generator's inputs (keys, values, queries) and encodes them itself."""
from __future__ import annotations

import numpy as np
import torch

import oracle
import paper_2609_09208_amd as pa

DEV = "cuda:0"
O_TOL = 2e-3  # max-abs bound on O against the fp64 oracle (the kernels accumulate in fp32)


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype)
    return t.to(DEV)


def store_values(v_bits, B, Hkv, t_cap):
    """Row-major fp16 values [B, Hkv, t_cap, 64] (host) -> device value cache."""
    src = to_dev(np.ascontiguousarray(v_bits).reshape(B * Hkv, t_cap, 64)).view(torch.float16)
    cache = pa.alloc_value_cache(B, Hkv, t_cap, DEV)
    pa.pot_store_values(src, B * Hkv, t_cap, t_cap, 0, cache)
    return cache


def gpu_encode(k_bits, mant_bits=0, hadamard=False, key_scale=None, frac_bits=7):
    """k_bits: uint16 [rows, 64] host. Returns numpy (codes_se, codes_m, scale)."""
    rows = k_bits.reshape(-1, 64).shape[0]
    k = to_dev(k_bits.reshape(rows, 64)).view(torch.float16)
    fmt = pa.make_format(mant_bits, frac_bits, hadamard)
    se = torch.zeros((rows, 32), dtype=torch.uint8, device=DEV)
    cm = torch.zeros((rows, 8 * mant_bits), dtype=torch.uint8, device=DEV) if mant_bits else None
    if key_scale is None:
        sc = torch.zeros(rows, dtype=torch.float32, device=DEV)
        mode = 0
    else:
        sc = to_dev(np.asarray(key_scale, np.float32).reshape(rows))
        mode = 1
    pa.pot_encode_keys(fmt, k, rows, 1, mode, sc, se, cm)
    torch.cuda.synchronize()
    return (se.cpu().numpy(), cm.cpu().numpy() if cm is not None else None,
            sc.cpu().numpy())


def gpu_pot_decode(d, codes_se, codes_m, key_scale, mant_bits=0, frac_bits=7,
                   hadamard=False, taps=True, force_splits=0, engine="sac", wg_waves=0):
    """d: workloads.make_decode_inputs dict; cache arrays are host numpy in the
    row layout. engine "sac" runs pot_decode_attention (shift-accumulate),
    "ds4a" pot_ds4a_decode_attention (byte decode + v_dot4), "dot"
    pot_dot_decode_attention (codes decoded to dot-unit weights, any k).
    Returns dict of numpy results (taps when requested)."""
    B, Hq, Hkv, T, t_cap = d["B"], d["Hq"], d["Hkv"], d["T"], d["t_cap"]
    fmt = pa.make_format(mant_bits, frac_bits, hadamard)
    q = to_dev(d["q"])
    se = to_dev(codes_se)
    cm = to_dev(codes_m) if codes_m is not None else None
    sc = to_dev(key_scale)
    v = store_values(d["v_bits"], B, Hkv, t_cap)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    nws = pa.pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, force_splits) \
        if force_splits else pa.pot_decode_workspace_bytes(B, Hq, Hkv, T)
    ws = pa.alloc_workspace(nws, DEV)
    res = {}
    dbg = pa.pot_debug()
    dbg.force_splits = force_splits
    dbg.force_wg_waves = wg_waves
    bufs = {}
    if taps:
        max_s = -(-T // 256)
        bufs = dict(qhat=torch.empty((B, Hq, 64), dtype=torch.int8, device=DEV),
                    delta=torch.empty((B, Hq), dtype=torch.float32, device=DEV),
                    scores=torch.empty((B, Hq, T), dtype=torch.int32, device=DEV),
                    m_final=torch.empty((B, Hq), dtype=torch.int32, device=DEV),
                    m_split=torch.empty((B, Hq, max_s), dtype=torch.int32, device=DEV))
        for k_, t_ in bufs.items():
            setattr(dbg, k_, t_.data_ptr())
    if engine == "sac":
        pa.pot_decode_attention(fmt, q, se, cm, sc, v, t_cap, d["kv_head_of_q"], B,
                                Hq, Hkv, T, out, ws, dbg=dbg)
    elif engine == "dot":
        pa.pot_dot_decode_attention(fmt, q, se, cm, sc, v, t_cap, d["kv_head_of_q"], B,
                                    Hq, Hkv, T, out, ws, dbg=dbg)
    else:
        assert engine == "ds4a" and cm is None
        pa.pot_ds4a_decode_attention(fmt, q, se, sc, v, t_cap, d["kv_head_of_q"], B,
                                     Hq, Hkv, T, out, ws, dbg=dbg)
    torch.cuda.synchronize()
    res["out"] = out.cpu().numpy()
    res["n_splits"], res["split_len"] = dbg.n_splits, dbg.split_len
    res["wg_waves"] = dbg.wg_waves
    for k_, t_ in bufs.items():
        res[k_] = t_.cpu().numpy()
    if taps:
        # m_split is [B, Hq, n_splits] densely packed at the start of the buffer
        flat = res["m_split"].reshape(-1)[:B * Hq * dbg.n_splits]
        res["m_split"] = flat.reshape(B, Hq, dbg.n_splits)
    return res


def oracle_pot(d, mant_bits=0, frac_bits=7, hadamard=False, split_len=None,
               key_scale=None):
    rows = d["k_bits"].reshape(-1, 64)
    se, cm, sc = oracle.encode_keys(rows, mant_bits=mant_bits, hadamard=hadamard,
                                    key_scale=key_scale)
    r = oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], d["t_cap"],
                          d["kv_head_of_q"], d["B"], d["Hq"], d["Hkv"], d["T"],
                          mant_bits=mant_bits, frac_bits=frac_bits,
                          hadamard=hadamard, split_len=split_len)
    return se, cm, sc, r


def assert_pot_parity(d, mant_bits=0, frac_bits=7, hadamard=False, force_splits=0,
                      key_scale=None, taps=True, engine="sac", wg_waves=0):
    """Full parity: codes, scales, q^, Delta, scores, M (final and per split)
    bit-exact; O within O_TOL. Returns the max-abs O error."""
    rows = d["k_bits"].reshape(-1, 64)
    g_se, g_cm, g_sc = gpu_encode(rows, mant_bits, hadamard, key_scale)
    o_se, o_cm, o_sc, _ = oracle_pot(d, mant_bits, frac_bits, hadamard,
                                     key_scale=key_scale)
    assert np.array_equal(g_se, o_se), "codes_se differ"
    if mant_bits:
        assert np.array_equal(g_cm, o_cm), "codes_m differ"
    assert np.array_equal(g_sc.view(np.uint32), o_sc.view(np.uint32)), "key_scale differ"
    g = gpu_pot_decode(d, g_se, g_cm, g_sc, mant_bits, frac_bits, hadamard,
                       taps=taps, force_splits=force_splits, engine=engine, wg_waves=wg_waves)
    if wg_waves:
        assert g["wg_waves"] == wg_waves, (g["wg_waves"], wg_waves)
    _, _, _, o = oracle_pot(d, mant_bits, frac_bits, hadamard,
                            split_len=g["split_len"], key_scale=key_scale)
    if taps:
        assert np.array_equal(g["qhat"], o["qhat"]), "q^ differ"
        assert np.array_equal(g["delta"].view(np.uint32), o["delta"].view(np.uint32))
        assert np.array_equal(g["scores"], o["scores"]), "int32 scores differ"
        assert np.array_equal(g["m_final"], o["m_final"]), "M differs"
        assert np.array_equal(g["m_split"], o["m_split"]), "per-split M differs"
    err = float(np.abs(g["out"] - o["out"]).max())
    assert err <= O_TOL, err
    return err, g
