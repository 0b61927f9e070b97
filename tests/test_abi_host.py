"""Host-only checks of the C ABI (no GPU needed).

* libpotattn.so loads and exports every function include/pot_attn.h declares;
* every argument check returns its status before any HIP call, so these calls
  run with fake (never dereferenced) device addresses on a machine without a
  GPU;
* host-only helpers (bytes per row, workspace sizes, split plan) are right.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_09208_amd as pa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pot_attn.h")
FAKE = 0x7F0000001000  # 4 KiB-aligned, never dereferenced by host checks


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pot_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 11
    lib = ctypes.CDLL(pa.LIBRARY_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    assert pa.pot_status_string(0) == "POT_OK"
    assert pa.pot_status_string(3) == "POT_ERR_WORKSPACE"


def test_code_bytes_per_row():
    assert pa.pot_code_bytes_per_row(pa.make_format(0)) == 32     # 4 bits/element
    assert pa.pot_code_bytes_per_row(pa.make_format(1)) == 40     # 5 bits
    assert pa.pot_code_bytes_per_row(pa.make_format(4)) == 64     # 8 bits (Sec. II-D)
    assert pa.pot_code_bytes_per_row(pa.make_format(0, frac_bits=5)) == 0


def test_workspace_sizes():
    # B=64 kv units=256 -> 4 splits of 8192 keys at T=32768
    w = pa.pot_decode_workspace_bytes(64, 32, 4, 32768)
    # sized for the most splits the planner can pick: 2048 resident slots / 256
    # (batch, kv head) pairs = 8 splits
    per = 64 * 32 * 8                       # partials (m, l, o[64]) per (b, q head, split)
    # prepared query words per decode workgroup (one slot per (batch, kv
    # head, split); G = 8): 32 operand words and one score factor per head,
    # rounded up to 64 words
    qwords = -(-(32 + 1) * 8 // 64) * 64
    need = per * (64 + 2) * 4 + 64 * 4 * 8 * qwords * 4
    assert need <= w < need + 4 * 256
    assert pa.pot_decode_workspace_bytes(0, 32, 4, 10) == 0
    assert pa.pot_decode_workspace_bytes(1, 32, 4, 0) == 0
    # forcing more splits needs more workspace; one split needs only counters
    assert (pa.pot_decode_workspace_bytes_for_splits(1, 32, 4, 32768, 128)
            > pa.pot_decode_workspace_bytes(64, 32, 4, 32768) // 100)


def _decode(fmt=None, **over):
    args = dict(q=FAKE, codes_se=FAKE, codes_m=None, key_scale=FAKE, v=FAKE,
                t_cap=4096, heads=np.arange(32, dtype=np.int32) // 8, B=1,
                Hq=32, Hkv=4, T=4096, out=FAKE, ws=FAKE, ws_bytes=1 << 30)
    args.update(over)
    fmt = fmt or pa.make_format()
    hm = np.ascontiguousarray(args["heads"], dtype=np.int32) \
        if args["heads"] is not None else None
    return pa._lib.pot_decode_attention(
        ctypes.byref(fmt), args["q"], args["codes_se"], args["codes_m"],
        args["key_scale"], args["v"], args["t_cap"],
        hm.ctypes.data_as(ctypes.c_void_p) if hm is not None else None,
        args["B"], args["Hq"], args["Hkv"], args["T"], args["out"], args["ws"],
        args["ws_bytes"], None, None)


@pytest.mark.parametrize("fmt,code", [
    (pa.make_format(head_dim=128), pa.POT_ERR_UNSUPPORTED),
    (pa.make_format(exp_bits=2), pa.POT_ERR_UNSUPPORTED),
    (pa.make_format(mant_bits=5), pa.POT_ERR_UNSUPPORTED),
    (pa.make_format(frac_bits=5), pa.POT_ERR_INVALID_ARG),   # F < E
    (pa.make_format(frac_bits=13), pa.POT_ERR_UNSUPPORTED),
    (pa.pot_format(64, 3, 0, 7, 2), pa.POT_ERR_INVALID_ARG),
])
def test_decode_rejects_bad_format(fmt, code):
    assert _decode(fmt) == code


@pytest.mark.parametrize("over,code", [
    (dict(q=None), pa.POT_ERR_INVALID_ARG),
    (dict(codes_se=None), pa.POT_ERR_INVALID_ARG),
    (dict(key_scale=None), pa.POT_ERR_INVALID_ARG),
    (dict(v=None), pa.POT_ERR_INVALID_ARG),
    (dict(out=None), pa.POT_ERR_INVALID_ARG),
    (dict(ws=None), pa.POT_ERR_INVALID_ARG),
    (dict(codes_m=FAKE), pa.POT_ERR_INVALID_ARG),        # k = 0 takes no planes
    (dict(q=FAKE + 4), pa.POT_ERR_INVALID_ARG),          # misaligned
    (dict(T=0), pa.POT_ERR_INVALID_ARG),
    (dict(T=4097), pa.POT_ERR_INVALID_ARG),              # T > t_cap
    (dict(B=0), pa.POT_ERR_INVALID_ARG),
    (dict(heads=None), pa.POT_ERR_INVALID_ARG),
    (dict(heads=np.full(32, 4)), pa.POT_ERR_INVALID_ARG),  # outside [0, Hkv)
    (dict(heads=np.r_[np.zeros(9), np.ones(7), np.full(8, 2), np.full(8, 3)]),
     pa.POT_ERR_UNSUPPORTED),                             # unequal groups
    (dict(Hq=24, Hkv=4, heads=np.arange(24) // 6), pa.POT_ERR_UNSUPPORTED),  # G=6
    (dict(Hq=256, Hkv=32, heads=np.arange(256) // 8), pa.POT_ERR_UNSUPPORTED),
    (dict(ws_bytes=1000), pa.POT_ERR_WORKSPACE),
    (dict(T=1 << 24, t_cap=1 << 24), pa.POT_ERR_UNSUPPORTED),  # past 2^24 - 8 keys
])
def test_decode_rejects_bad_arguments(over, code):
    assert _decode(**over) == code
    assert pa.pot_last_error() != ""


def test_decode_mantissa_needs_planes():
    assert _decode(pa.make_format(mant_bits=1)) == pa.POT_ERR_INVALID_ARG


def test_encode_rejects_bad_arguments():
    f = pa.make_format()
    E = pa._lib.pot_encode_keys
    assert E(ctypes.byref(pa.make_format(frac_bits=4)), FAKE, 10, 1, 0, FAKE,
             FAKE, None, None) == pa.POT_ERR_INVALID_ARG
    assert E(ctypes.byref(f), FAKE, -1, 1, 0, FAKE, FAKE, None, None) == pa.POT_ERR_INVALID_ARG
    assert E(ctypes.byref(f), FAKE, 10, 0, 0, FAKE, FAKE, None, None) == pa.POT_ERR_INVALID_ARG
    assert E(ctypes.byref(f), FAKE, 10, 1, 2, FAKE, FAKE, None, None) == pa.POT_ERR_INVALID_ARG
    assert E(ctypes.byref(f), None, 10, 1, 0, FAKE, FAKE, None, None) == pa.POT_ERR_INVALID_ARG
    assert E(ctypes.byref(pa.make_format(2)), FAKE, 10, 1, 0, FAKE, FAKE, None,
             None) == pa.POT_ERR_INVALID_ARG
    # zero rows is a no-op that needs no pointers at all
    assert E(ctypes.byref(f), None, 0, 1, 0, None, None, None, None) == pa.POT_OK


def test_int8_and_fp16_reject_bad_arguments():
    hm = (np.arange(32, dtype=np.int32) // 8)
    hp = hm.ctypes.data_as(ctypes.c_void_p)
    I = pa._lib.pot_int8_decode_attention
    assert I(FAKE, FAKE, FAKE, FAKE, 64, hp, 1, 32, 4, 64, 2, FAKE, FAKE,
             1 << 20, None, None) == pa.POT_ERR_INVALID_ARG
    assert I(FAKE, None, FAKE, FAKE, 64, hp, 1, 32, 4, 64, 0, FAKE, FAKE,
             1 << 20, None, None) == pa.POT_ERR_INVALID_ARG
    F = pa._lib.pot_fp16_decode_attention
    assert F(FAKE, None, FAKE, 64, hp, 1, 32, 4, 64, FAKE, FAKE, 1 << 20,
             None) == pa.POT_ERR_INVALID_ARG
    assert F(FAKE, FAKE, FAKE, 64, hp, 1, 32, 4, 64, FAKE, FAKE, 16,
             None) == pa.POT_ERR_WORKSPACE
    assert pa._lib.pot_int8_encode_keys(FAKE, 5, 1, 3, FAKE, FAKE, None) == pa.POT_ERR_INVALID_ARG


def test_binding_raises_pot_error():
    with pytest.raises(pa.PotError) as ei:
        pa._check(pa.POT_ERR_WORKSPACE)
    assert ei.value.status == pa.POT_ERR_WORKSPACE


def test_store_values_rejects_bad_arguments():
    S = pa._lib.pot_store_values
    assert S(FAKE, 2, 5, 12, 0, FAKE, None) == pa.POT_ERR_INVALID_ARG   # t_cap % 8
    assert S(FAKE, 2, 5, 16, 12, FAKE, None) == pa.POT_ERR_INVALID_ARG  # past t_cap
    assert S(FAKE, 2, 5, 16, -1, FAKE, None) == pa.POT_ERR_INVALID_ARG
    assert S(FAKE, -1, 5, 16, 0, FAKE, None) == pa.POT_ERR_INVALID_ARG
    assert S(None, 2, 5, 16, 0, FAKE, None) == pa.POT_ERR_INVALID_ARG
    assert S(FAKE + 2, 2, 5, 16, 0, FAKE, None) == pa.POT_ERR_INVALID_ARG
    assert S(None, 0, 5, 16, 0, None, None) == pa.POT_OK  # nothing to store


def test_decode_needs_t_cap_multiple_of_8():
    assert _decode(t_cap=4100) == pa.POT_ERR_INVALID_ARG


def test_ds4a_rejects_bad_arguments():
    hm = (np.arange(32, dtype=np.int32) // 8)
    hp = hm.ctypes.data_as(ctypes.c_void_p)
    D = pa._lib.pot_ds4a_decode_attention
    args = lambda fmt, se=FAKE: (ctypes.byref(fmt), FAKE, se, FAKE, FAKE, 4096, hp, 1, 32, 4,
                                 4096, FAKE, FAKE, 1 << 30, None, None)
    assert D(*args(pa.make_format(mant_bits=1))) == pa.POT_ERR_UNSUPPORTED
    assert D(*args(pa.make_format(frac_bits=5))) == pa.POT_ERR_INVALID_ARG
    assert D(*args(pa.make_format(), se=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(pa.make_format(), se=FAKE + 4)) == pa.POT_ERR_INVALID_ARG


def test_dot_rejects_bad_arguments():
    hm = (np.arange(32, dtype=np.int32) // 8)
    hp = hm.ctypes.data_as(ctypes.c_void_p)
    D = pa._lib.pot_dot_decode_attention

    def args(fmt=None, se=FAKE, cm=None, sc=FAKE, T=4096, t_cap=4096, ws=1 << 30):
        fmt = fmt if fmt is not None else pa.make_format()
        return (ctypes.byref(fmt), FAKE, se, cm, sc, FAKE, t_cap, hp, 1, 32, 4, T, FAKE, FAKE,
                ws, None, None)
    assert D(*args(se=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(sc=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(se=FAKE + 4)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(fmt=pa.make_format(mant_bits=4))) == pa.POT_ERR_INVALID_ARG  # planes NULL
    assert D(*args(cm=FAKE)) == pa.POT_ERR_INVALID_ARG  # planes given for PoT-4
    assert D(*args(fmt=pa.make_format(mant_bits=2), cm=FAKE + 4)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(fmt=pa.make_format(mant_bits=5), cm=FAKE)) == pa.POT_ERR_UNSUPPORTED
    assert D(*args(fmt=pa.make_format(frac_bits=5))) == pa.POT_ERR_INVALID_ARG
    assert D(*args(T=0)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(T=4097)) == pa.POT_ERR_INVALID_ARG  # beyond t_cap
    assert D(*args(ws=16)) == pa.POT_ERR_WORKSPACE


def test_append_rejects_bad_arguments():
    hm = (np.arange(32, dtype=np.int32) // 8)
    hp = hm.ctypes.data_as(ctypes.c_void_p)
    D = pa._lib.pot_append_decode_attention

    def args(fmt=None, kn=FAKE, vn=FAKE, se=FAKE, cm=None, sc=FAKE, T=4096, t_cap=4096,
             ws=1 << 30):
        fmt = fmt if fmt is not None else pa.make_format()
        return (ctypes.byref(fmt), FAKE, kn, vn, se, cm, sc, FAKE, t_cap, hp, 1, 32, 4, T,
                FAKE, FAKE, ws, None, None)
    assert D(*args(kn=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(vn=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(kn=FAKE + 2)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(vn=FAKE + 8)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(se=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(sc=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(fmt=pa.make_format(mant_bits=1))) == pa.POT_ERR_INVALID_ARG  # planes NULL
    assert D(*args(cm=FAKE)) == pa.POT_ERR_INVALID_ARG  # planes given for PoT-4
    assert D(*args(fmt=pa.make_format(mant_bits=5))) == pa.POT_ERR_UNSUPPORTED
    assert D(*args(fmt=pa.make_format(frac_bits=5))) == pa.POT_ERR_INVALID_ARG
    assert D(*args(T=0)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(T=4097)) == pa.POT_ERR_INVALID_ARG  # beyond t_cap
    assert D(*args(t_cap=4100, T=4097)) == pa.POT_ERR_INVALID_ARG  # t_cap not a multiple of 8
    assert D(*args(ws=16)) == pa.POT_ERR_WORKSPACE


def test_int8_values_reject_bad_arguments():
    S = pa._lib.pot_store_values_int8
    assert S(FAKE, 1, 1, 12, 0, FAKE, FAKE, None) == pa.POT_ERR_INVALID_ARG   # t_cap % 8
    assert S(FAKE, 1, 2, 8, 7, FAKE, FAKE, None) == pa.POT_ERR_INVALID_ARG    # past t_cap
    assert S(FAKE, -1, 1, 8, 0, FAKE, FAKE, None) == pa.POT_ERR_INVALID_ARG
    assert S(FAKE, 1, 1, 8, 0, FAKE, None, None) == pa.POT_ERR_INVALID_ARG
    assert S(FAKE, 1, 1, 8, 0, FAKE + 8, FAKE, None) == pa.POT_ERR_INVALID_ARG
    assert S(None, 0, 1, 8, 0, None, None, None) == pa.POT_OK                 # empty: no-op
    hm = (np.arange(32, dtype=np.int32) // 8)
    hp = hm.ctypes.data_as(ctypes.c_void_p)
    D = pa._lib.pot_decode_attention_v8

    def args(fmt=None, engine=0, vu=FAKE, ve=FAKE, T=4096, ws=1 << 30):
        fmt = fmt if fmt is not None else pa.make_format()
        return (ctypes.byref(fmt), engine, FAKE, FAKE, None, FAKE, vu, ve, 4096, hp, 1, 32, 4,
                T, FAKE, FAKE, ws, None, None)
    assert D(*args(engine=2)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(engine=-1)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(vu=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(ve=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(ve=FAKE + 4)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(T=0)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(ws=16)) == pa.POT_ERR_WORKSPACE
    # byte-decode engine: PoT-4 only
    assert D(*args(fmt=pa.make_format(mant_bits=1), engine=1)) == pa.POT_ERR_UNSUPPORTED


def test_pow2_rejects_bad_arguments():
    hm = (np.arange(32, dtype=np.int32) // 8)
    hp = hm.ctypes.data_as(ctypes.c_void_p)
    D = pa._lib.pot_decode_attention_v8_pow2

    def args(fmt=None, engine=0, vu=FAKE, ve=FAKE, T=4096):
        fmt = fmt if fmt is not None else pa.make_format()
        return (ctypes.byref(fmt), engine, FAKE, FAKE, None, FAKE, vu, ve, 4096, hp, 1, 32, 4,
                T, FAKE, FAKE, 1 << 30, None, None)
    assert D(*args(engine=3)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(vu=None)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(ve=FAKE + 2)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(T=4097)) == pa.POT_ERR_INVALID_ARG
    assert D(*args(fmt=pa.make_format(mant_bits=2), engine=1)) == pa.POT_ERR_UNSUPPORTED


def test_noalloc_rejects_shapes_beyond_its_scratch():
    # the workspace bound is checked on the host before any HIP call
    with pytest.raises(pa.PotError) as e:
        pa.pot_decode_attention_noalloc(pa.make_format(0), FAKE, FAKE, None, FAKE, FAKE, 4096,
                                        np.arange(32, dtype=np.int32) // 8, 4096, 32, 4, 4096,
                                        FAKE)
    assert e.value.status == pa.POT_ERR_WORKSPACE
    assert "static scratch" in pa.pot_last_error()
    # forced splits count against the same bound
    dbg = pa.pot_debug()
    dbg.force_splits = 4096
    with pytest.raises(pa.PotError) as e:
        pa.pot_decode_attention_noalloc(pa.make_format(0), FAKE, FAKE, None, FAKE, FAKE,
                                        1 << 20, np.arange(32, dtype=np.int32) // 8, 16, 32, 4,
                                        1 << 20, FAKE, dbg=dbg)
    assert e.value.status == pa.POT_ERR_WORKSPACE
