"""CPU oracle for power-of-two-key decode attention (arXiv 2609.09208).

TEST INFRASTRUCTURE ONLY: the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` are the only callers allowed. The product path
(``paper_2609_09208_amd``) never imports this package, and this package never
imports the product path. It wraps ``pot_oracle.c`` (plain scalar C, fp64 where
the paper leaves precision open) through ctypes on numpy arrays.

Sections cited: Sec. II-A eq. (pot) key code and INT8 query; Sec. II-B eq. (sac)
score; Sec. II-C eq. (exact) head-room; Sec. II-D eq. (mant) mantissa family;
Sec. II-E eq. (logsm) integer-log2 softmax maximum, and INT8 values with a
power-of-two per-token scale; Sec. I-A / V-A Hadamard.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pot_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
DIM = 64

_lib = None


def build_oracle() -> str:
    """Compile pot_oracle.c with gcc (-O2, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-Wall", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or (
            os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC)):
        build_oracle()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int, ctypes.c_int64
    lib.oracle_half_to_float.argtypes = [ctypes.c_uint16]
    lib.oracle_half_to_float.restype = ctypes.c_float
    lib.oracle_float_to_half.argtypes = [ctypes.c_float]
    lib.oracle_float_to_half.restype = ctypes.c_uint16
    lib.oracle_fwht_query.argtypes = [P, P]
    lib.oracle_rotate_keys.argtypes = [P, i64, P]
    lib.oracle_quantize_query.argtypes = [i32, P, i64, P, P, P]
    lib.oracle_encode_keys.argtypes = [i32, i32, P, i64, i32, P, P, P]
    lib.oracle_encode_keys.restype = i32
    lib.oracle_pot_decode.argtypes = [i32, i32, i32, P, P, P, P, P, i64, P,
                                      i32, i32, i32, i32, i32, i32,
                                      P, P, P, P, P, P, P]
    lib.oracle_pot_decode.restype = i32
    lib.oracle_pot_decode_v8.argtypes = [i32, i32, i32, P, P, P, P, P, P, i64, P,
                                         i32, i32, i32, i32, i32, i32,
                                         P, P, P, P, P, P, P]
    lib.oracle_pot_decode_v8.restype = i32
    lib.oracle_pot_decode_v8_pow2.argtypes = lib.oracle_pot_decode_v8.argtypes
    lib.oracle_pot_decode_v8_pow2.restype = i32
    lib.oracle_attend_x.argtypes = [P, P, P, i32, i32, i32, i32, P, P]
    lib.oracle_attend_x.restype = i32
    lib.oracle_quantize_values.argtypes = [P, i64, P, P]
    lib.oracle_quantize_values.restype = i32
    lib.oracle_int8_encode_keys.argtypes = [i32, P, i64, P, P]
    lib.oracle_int8_encode_keys.restype = i32
    lib.oracle_int8_decode.argtypes = [i32, P, P, P, P, i64, P, i32, i32, i32,
                                       i32, i32, P, P, P, P, P, P]
    lib.oracle_int8_decode.restype = i32
    lib.oracle_fp16_decode.argtypes = [P, P, P, i64, P, i32, i32, i32, i32, P]
    lib.oracle_fp16_decode.restype = i32
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# --------------------------------------------------------------------------
def half_to_float(bits: int) -> float:
    return float(_load().oracle_half_to_float(bits))


def float_to_half(x: float) -> int:
    return int(_load().oracle_float_to_half(x))


def fwht_query(q):
    """fp64 radix-2 Walsh-Hadamard butterfly of one 64-vector, /8, to fp32."""
    q = _c(q, np.float32)
    out = np.empty(DIM, np.float32)
    _load().oracle_fwht_query(_ptr(q), _ptr(out))
    return out


def rotate_keys(k_fp16_bits):
    """fl32(H K / 8) per row of fp16 keys (exact fp64 sum, one rounding)."""
    k = _c(k_fp16_bits, np.uint16).reshape(-1, DIM)
    out = np.empty(k.shape, np.float32)
    _load().oracle_rotate_keys(_ptr(k), k.shape[0], _ptr(out))
    return out


def quantize_query(q, hadamard=False):
    """INT8 query with per-vector step (Sec. II-A). q: [..., 64] fp32.

    Returns (qhat int8 [..., 64], delta fp32 [...], q_rot fp32 [..., 64])."""
    q = _c(q, np.float32)
    shape = q.shape[:-1]
    n = int(np.prod(shape)) if shape else 1
    qh = np.empty(q.shape, np.int8)
    dl = np.empty(shape, np.float32)
    qr = np.empty(q.shape, np.float32)
    _load().oracle_quantize_query(int(hadamard), _ptr(q), n, _ptr(qh),
                                  _ptr(dl), _ptr(qr))
    return qh, dl, qr


def encode_keys(k_fp16_bits, mant_bits=0, hadamard=False, key_scale=None):
    """PoT / PoT-Mk key codes (Sec. II-A, II-D).

    k_fp16_bits: uint16 [rows, 64] (fp16 bit patterns).
    key_scale: None (per-row absmax, scale mode 0) or fp32 [rows] (mode 1).
    Returns (codes_se uint8 [rows, 32], codes_m uint8 [rows, 8k] or None,
    key_scale fp32 [rows])."""
    k = _c(k_fp16_bits, np.uint16).reshape(-1, DIM)
    rows = k.shape[0]
    se = np.zeros((rows, DIM // 2), np.uint8)
    cm = np.zeros((rows, 8 * mant_bits), np.uint8) if mant_bits else None
    if key_scale is None:
        sc = np.zeros(rows, np.float32)
        mode = 0
    else:
        sc = _c(key_scale, np.float32).reshape(rows).copy()
        mode = 1
    rc = _load().oracle_encode_keys(int(mant_bits), int(hadamard), _ptr(k),
                                    rows, mode, _ptr(sc), _ptr(se), _ptr(cm))
    if rc:
        raise ValueError(f"oracle_encode_keys failed: {rc}")
    return se, cm, sc


def pot_decode(q, codes_se, codes_m, key_scale, v_fp16_bits, t_cap,
               kv_head_of_q, B, Hq, Hkv, T, mant_bits=0, frac_bits=7,
               hadamard=False, split_len=None, tile=0, want_out=True):
    """Decode attention with PoT keys (Sec. II-B, II-E).

    Cache arrays use the row layout row = (b*Hkv + h)*t_cap + t.
    Returns a dict with qhat, delta, scores (int32 [B,Hq,T]), x (fp32
    log2-domain scores), m_final, m_split and out (fp64 [B,Hq,64])."""
    split_len = T if split_len is None else int(split_len)
    n_split = -(-T // split_len)
    q = _c(q, np.float32)
    se = _c(codes_se, np.uint8)
    cm = None if codes_m is None else _c(codes_m, np.uint8)
    sc = _c(key_scale, np.float32)
    v = _c(v_fp16_bits, np.uint16)
    hm = _c(kv_head_of_q, np.int32)
    res = dict(qhat=np.empty((B, Hq, DIM), np.int8),
               delta=np.empty((B, Hq), np.float32),
               scores=np.empty((B, Hq, T), np.int32),
               x=np.empty((B, Hq, T), np.float32),
               m_final=np.empty((B, Hq), np.int32),
               m_split=np.empty((B, Hq, n_split), np.int32),
               out=np.empty((B, Hq, DIM), np.float64) if want_out else None)
    rc = _load().oracle_pot_decode(
        int(mant_bits), int(frac_bits), int(hadamard), _ptr(q), _ptr(se),
        _ptr(cm), _ptr(sc), _ptr(v), int(t_cap), _ptr(hm), B, Hq, Hkv, T,
        split_len, int(tile), _ptr(res["qhat"]), _ptr(res["delta"]),
        _ptr(res["scores"]), _ptr(res["x"]), _ptr(res["m_final"]),
        _ptr(res["m_split"]), _ptr(res["out"]))
    if rc:
        raise ValueError(f"oracle_pot_decode failed: {rc}")
    return res


def quantize_values(v_fp16_bits):
    """INT8 values with a power-of-two per-token scale (Sec. II-E).

    v_fp16_bits: uint16 [..., 64]. Per row: g = largest integer with
    max|v| * 2^g <= 127 (0 for a zero row), v^ = round-half-even(v * 2^g).
    Returns (v^ int8 [rows, 64], g int8 [rows]); the value is v^ * 2^-g."""
    v = _c(v_fp16_bits, np.uint16).reshape(-1, DIM)
    rows = v.shape[0]
    vh = np.empty((rows, DIM), np.int8)
    g = np.empty(rows, np.int8)
    rc = _load().oracle_quantize_values(_ptr(v), rows, _ptr(vh), _ptr(g))
    if rc:
        raise ValueError(f"oracle_quantize_values failed: {rc}")
    return vh, g


def pot_decode_v8(q, codes_se, codes_m, key_scale, v8, v_exp, t_cap, kv_head_of_q, B, Hq,
                  Hkv, T, mant_bits=0, frac_bits=7, hadamard=False, split_len=None,
                  tile=0, want_out=True, pow2=False):
    """pot_decode with the values given as INT8 codes v8 [rows, 64] and
    exponents v_exp [rows] (value v8 * 2^-v_exp, Sec. II-E). pow2: the
    power-of-two weights 2^-k of eq. logsm (k = M - ceil(x - 1/2)) instead of
    the softmax weights."""
    split_len = T if split_len is None else int(split_len)
    n_split = -(-T // split_len)
    res = dict(qhat=np.empty((B, Hq, DIM), np.int8),
               delta=np.empty((B, Hq), np.float32),
               scores=np.empty((B, Hq, T), np.int32),
               x=np.empty((B, Hq, T), np.float32),
               m_final=np.empty((B, Hq), np.int32),
               m_split=np.empty((B, Hq, n_split), np.int32),
               out=np.empty((B, Hq, DIM), np.float64) if want_out else None)
    cm = None if codes_m is None else _c(codes_m, np.uint8)
    fn = _load().oracle_pot_decode_v8_pow2 if pow2 else _load().oracle_pot_decode_v8
    rc = fn(
        int(mant_bits), int(frac_bits), int(hadamard), _ptr(_c(q, np.float32)),
        _ptr(_c(codes_se, np.uint8)), _ptr(cm), _ptr(_c(key_scale, np.float32)),
        _ptr(_c(v8, np.int8)), _ptr(_c(v_exp, np.int8)), int(t_cap),
        _ptr(_c(kv_head_of_q, np.int32)), B, Hq, Hkv, T, split_len, int(tile),
        _ptr(res["qhat"]), _ptr(res["delta"]), _ptr(res["scores"]), _ptr(res["x"]),
        _ptr(res["m_final"]), _ptr(res["m_split"]), _ptr(res["out"]))
    if rc:
        raise ValueError(f"oracle_pot_decode_v8 failed: {rc}")
    return res


def attend_x(x, v8, v_exp, split_len=None, tile=0, pow2=False):
    """One query's attention over given log2-domain scores x [T] (fp32) and
    INT8 value rows v8 [T, 64] with exponents v_exp [T]. Returns (out fp64
    [64], M)."""
    x = _c(x, np.float32)
    T = x.shape[0]
    out = np.empty(DIM, np.float64)
    m = np.empty(1, np.int32)
    rc = _load().oracle_attend_x(_ptr(x), _ptr(_c(v8, np.int8)), _ptr(_c(v_exp, np.int8)), T,
                                 T if split_len is None else int(split_len), int(tile),
                                 int(pow2), _ptr(m), _ptr(out))
    if rc:
        raise ValueError(f"oracle_attend_x failed: {rc}")
    return out, int(m[0])


def int8_encode_keys(k_fp16_bits, hadamard=False):
    k = _c(k_fp16_bits, np.uint16).reshape(-1, DIM)
    rows = k.shape[0]
    codes = np.empty((rows, DIM), np.int8)
    sc = np.empty(rows, np.float32)
    _load().oracle_int8_encode_keys(int(hadamard), _ptr(k), rows, _ptr(sc),
                                    _ptr(codes))
    return codes, sc


def int8_decode(q, codes, key_scale, v_fp16_bits, t_cap, kv_head_of_q, B, Hq,
                Hkv, T, hadamard=False, split_len=None):
    split_len = T if split_len is None else int(split_len)
    n_split = -(-T // split_len)
    res = dict(qhat=np.empty((B, Hq, DIM), np.int8),
               delta=np.empty((B, Hq), np.float32),
               scores=np.empty((B, Hq, T), np.int32),
               m_final=np.empty((B, Hq), np.int32),
               m_split=np.empty((B, Hq, n_split), np.int32),
               out=np.empty((B, Hq, DIM), np.float64))
    rc = _load().oracle_int8_decode(
        int(hadamard), _ptr(_c(q, np.float32)), _ptr(_c(codes, np.int8)),
        _ptr(_c(key_scale, np.float32)), _ptr(_c(v_fp16_bits, np.uint16)),
        int(t_cap), _ptr(_c(kv_head_of_q, np.int32)), B, Hq, Hkv, T,
        split_len, _ptr(res["qhat"]), _ptr(res["delta"]), _ptr(res["scores"]),
        _ptr(res["m_final"]), _ptr(res["m_split"]), _ptr(res["out"]))
    if rc:
        raise ValueError(f"oracle_int8_decode failed: {rc}")
    return res


def fp16_decode(q, k_fp16_bits, v_fp16_bits, t_cap, kv_head_of_q, B, Hq, Hkv,
                T):
    out = np.empty((B, Hq, DIM), np.float64)
    rc = _load().oracle_fp16_decode(
        _ptr(_c(q, np.float32)), _ptr(_c(k_fp16_bits, np.uint16)),
        _ptr(_c(v_fp16_bits, np.uint16)), int(t_cap),
        _ptr(_c(kv_head_of_q, np.int32)), B, Hq, Hkv, T, _ptr(out))
    if rc:
        raise ValueError(f"oracle_fp16_decode failed: {rc}")
    return out
