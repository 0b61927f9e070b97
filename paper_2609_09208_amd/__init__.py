"""Python binding of libpotattn: PoT-key decode attention for AMD MI355X.

Argument marshalling only. Every entry point has the name of the C function in
``include/pot_attn.h`` and forwards device pointers, sizes and the current HIP
stream through ctypes; every step of the computation runs in the library's
gfx950 kernels. Tensors are torch device tensors (torch is used for device
memory and streams). A missing or unloadable library raises at import time:
there is no fallback path.

Method: "Shift-Accumulate Attention: Multiplier-Free Query-Key Products for
Transformer Decoding" (arXiv 2609.09208), Sec. II.
"""
from __future__ import annotations

import ctypes
import os

HEAD_DIM = 64
_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpotattn.so")

POT_OK = 0
POT_ERR_INVALID_ARG = 1
POT_ERR_UNSUPPORTED = 2
POT_ERR_WORKSPACE = 3
POT_ERR_HIP = 4


class PotError(RuntimeError):
    def __init__(self, status: int, name: str, detail: str):
        super().__init__(f"{name}: {detail}")
        self.status = status


class pot_format(ctypes.Structure):
    _fields_ = [("head_dim", ctypes.c_int32), ("exp_bits", ctypes.c_int32),
                ("mant_bits", ctypes.c_int32), ("frac_bits", ctypes.c_int32),
                ("hadamard", ctypes.c_int32)]


class pot_debug(ctypes.Structure):
    _fields_ = [("qhat", ctypes.c_void_p), ("delta", ctypes.c_void_p),
                ("scores", ctypes.c_void_p), ("m_final", ctypes.c_void_p),
                ("m_split", ctypes.c_void_p), ("force_splits", ctypes.c_int32),
                ("n_splits", ctypes.c_int32), ("split_len", ctypes.c_int32),
                ("decode_begin", ctypes.c_void_p), ("decode_end", ctypes.c_void_p),
                ("force_wg_waves", ctypes.c_int32), ("wg_waves", ctypes.c_int32)]


def make_format(mant_bits: int = 0, frac_bits: int = 7, hadamard: bool = False,
                exp_bits: int = 3, head_dim: int = HEAD_DIM) -> pot_format:
    return pot_format(head_dim, exp_bits, mant_bits, frac_bits, int(bool(hadamard)))


def _load_library():
    # torch ships its own HIP runtime with the same soname as ROCm's; load it
    # first so that this library binds to the one runtime torch uses for the
    # device memory and streams it hands over (two runtimes in one process do
    # not share devices).
    import torch  # noqa: F401
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is not built; run __graft_entry__.build() (hipcc, gfx950)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, S = ctypes.c_void_p, ctypes.c_size_t
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    fmt_p = ctypes.POINTER(pot_format)
    dbg_p = ctypes.POINTER(pot_debug)
    sig = {
        "pot_status_string": (ctypes.c_char_p, [i32]),
        "pot_last_error": (ctypes.c_char_p, []),
        "pot_code_bytes_per_row": (S, [fmt_p]),
        "pot_encode_keys": (i32, [fmt_p, P, i64, i64, i32, P, P, P, P]),
        "pot_decode_workspace_bytes": (S, [i32, i32, i32, i32]),
        "pot_decode_workspace_bytes_for_splits": (S, [i32, i32, i32, i32, i32]),
        "pot_workspace_init": (i32, [P, S, P]),
        "pot_store_values": (i32, [P, i64, i64, i64, i64, P, P]),
        "pot_store_values_int8": (i32, [P, i64, i64, i64, i64, P, P, P]),
        "pot_decode_attention_v8": (i32, [fmt_p, i32, P, P, P, P, P, P, i64, P, i32, i32,
                                          i32, i32, P, P, S, dbg_p, P]),
        "pot_decode_attention_v8_pow2": (i32, [fmt_p, i32, P, P, P, P, P, P, i64, P, i32, i32,
                                               i32, i32, P, P, S, dbg_p, P]),
        "pot_decode_attention": (i32, [fmt_p, P, P, P, P, P, i64, P, i32, i32,
                                       i32, i32, P, P, S, dbg_p, P]),
        "pot_append_decode_attention": (i32, [fmt_p, P, P, P, P, P, P, P, i64, P, i32, i32,
                                              i32, i32, P, P, S, dbg_p, P]),
        "pot_append_decode_attention_v8": (i32, [fmt_p, i32, P, P, P, P, P, P, P, P, i64, P,
                                                 i32, i32, i32, i32, P, P, S, dbg_p, P]),
        "pot_decode_attention_noalloc": (i32, [fmt_p, P, P, P, P, P, i64, P, i32, i32,
                                               i32, i32, P, dbg_p, P]),
        "pot_ds4a_decode_attention": (i32, [fmt_p, P, P, P, P, i64, P, i32, i32, i32, i32, P, P,
                                            S, dbg_p, P]),
        "pot_dot_decode_attention": (i32, [fmt_p, P, P, P, P, P, i64, P, i32, i32, i32, i32,
                                           P, P, S, dbg_p, P]),
        "pot_int8_encode_keys": (i32, [P, i64, i64, i32, P, P, P]),
        "pot_int8_decode_attention": (i32, [P, P, P, P, i64, P, i32, i32, i32,
                                            i32, i32, P, P, S, dbg_p, P]),
        "pot_fp16_decode_attention": (i32, [P, P, P, i64, P, i32, i32, i32,
                                            i32, P, P, S, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load_library()
LIBRARY_PATH = _LIB_PATH


def _check(status: int) -> None:
    if status != POT_OK:
        name = _lib.pot_status_string(status).decode()
        raise PotError(status, name, _lib.pot_last_error().decode())


def _ptr(t) -> int | None:
    """Device pointer of a torch tensor, an int address, or None."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    if not torch.cuda.is_available():
        return None
    return torch.cuda.current_stream().cuda_stream


def _heads(kv_head_of_q):
    import numpy as np
    arr = np.ascontiguousarray(kv_head_of_q, dtype=np.int32)
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


# ---- C ABI mirrors ---------------------------------------------------------
def pot_status_string(status: int) -> str:
    return _lib.pot_status_string(status).decode()


def pot_last_error() -> str:
    return _lib.pot_last_error().decode()


def pot_code_bytes_per_row(fmt: pot_format) -> int:
    return int(_lib.pot_code_bytes_per_row(ctypes.byref(fmt)))


def pot_decode_workspace_bytes(B: int, Hq: int, Hkv: int, T: int) -> int:
    return int(_lib.pot_decode_workspace_bytes(B, Hq, Hkv, T))


def pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, n_splits) -> int:
    return int(_lib.pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, n_splits))


def pot_workspace_init(workspace, ws_bytes: int | None = None, stream=None) -> None:
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_workspace_init(_ptr(workspace), nbytes, _stream(stream)))


def pot_store_values(v_fp16, n_seq: int, n_tok: int, t_cap: int, t0: int, v_cache,
                     stream=None) -> None:
    _check(_lib.pot_store_values(_ptr(v_fp16), int(n_seq), int(n_tok), int(t_cap),
                                 int(t0), _ptr(v_cache), _stream(stream)))


def pot_store_values_int8(v_fp16, n_seq: int, n_tok: int, t_cap: int, t0: int, v_u8, v_exp,
                          stream=None) -> None:
    _check(_lib.pot_store_values_int8(_ptr(v_fp16), int(n_seq), int(n_tok), int(t_cap),
                                      int(t0), _ptr(v_u8), _ptr(v_exp), _stream(stream)))


def pot_decode_attention_v8(fmt: pot_format, engine: int, q, codes_se, codes_m, key_scale,
                            v_u8, v_exp, t_cap: int, kv_head_of_q, B: int, Hq: int, Hkv: int,
                            T: int, out, workspace, ws_bytes=None,
                            dbg: pot_debug | None = None, stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_decode_attention_v8(
        ctypes.byref(fmt), int(engine), _ptr(q), _ptr(codes_se), _ptr(codes_m),
        _ptr(key_scale), _ptr(v_u8), _ptr(v_exp), int(t_cap), hp, B, Hq, Hkv, T, _ptr(out),
        _ptr(workspace), nbytes, ctypes.byref(dbg) if dbg is not None else None,
        _stream(stream)))


def pot_decode_attention_v8_pow2(fmt: pot_format, engine: int, q, codes_se, codes_m, key_scale,
                                 v_u8, v_exp, t_cap: int, kv_head_of_q, B: int, Hq: int,
                                 Hkv: int, T: int, out, workspace, ws_bytes=None,
                                 dbg: pot_debug | None = None, stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_decode_attention_v8_pow2(
        ctypes.byref(fmt), int(engine), _ptr(q), _ptr(codes_se), _ptr(codes_m),
        _ptr(key_scale), _ptr(v_u8), _ptr(v_exp), int(t_cap), hp, B, Hq, Hkv, T, _ptr(out),
        _ptr(workspace), nbytes, ctypes.byref(dbg) if dbg is not None else None,
        _stream(stream)))


def pot_encode_keys(fmt: pot_format, k_fp16, n_rows: int, out_row_stride: int,
                    scale_mode: int, key_scale, codes_se, codes_m=None,
                    stream=None) -> None:
    _check(_lib.pot_encode_keys(ctypes.byref(fmt), _ptr(k_fp16), int(n_rows),
                                int(out_row_stride), int(scale_mode),
                                _ptr(key_scale), _ptr(codes_se), _ptr(codes_m),
                                _stream(stream)))


def pot_decode_attention(fmt: pot_format, q, codes_se, codes_m, key_scale,
                         v_fp16, t_cap: int, kv_head_of_q, B: int, Hq: int,
                         Hkv: int, T: int, out, workspace, ws_bytes=None,
                         dbg: pot_debug | None = None, stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_decode_attention(
        ctypes.byref(fmt), _ptr(q), _ptr(codes_se), _ptr(codes_m),
        _ptr(key_scale), _ptr(v_fp16), int(t_cap), hp, B, Hq, Hkv, T,
        _ptr(out), _ptr(workspace), nbytes,
        ctypes.byref(dbg) if dbg is not None else None, _stream(stream)))


def pot_decode_attention_noalloc(fmt: pot_format, q, codes_se, codes_m, key_scale,
                                 v_fp16, t_cap: int, kv_head_of_q, B: int, Hq: int,
                                 Hkv: int, T: int, out, dbg: pot_debug | None = None,
                                 stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    _check(_lib.pot_decode_attention_noalloc(
        ctypes.byref(fmt), _ptr(q), _ptr(codes_se), _ptr(codes_m),
        _ptr(key_scale), _ptr(v_fp16), int(t_cap), hp, B, Hq, Hkv, T,
        _ptr(out), ctypes.byref(dbg) if dbg is not None else None, _stream(stream)))


def pot_append_decode_attention(fmt: pot_format, q, k_new, v_new, codes_se, codes_m,
                                key_scale, v_cache, t_cap: int, kv_head_of_q, B: int, Hq: int,
                                Hkv: int, T: int, out, workspace, ws_bytes=None,
                                dbg: pot_debug | None = None, stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_append_decode_attention(
        ctypes.byref(fmt), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(codes_se), _ptr(codes_m),
        _ptr(key_scale), _ptr(v_cache), int(t_cap), hp, B, Hq, Hkv, T, _ptr(out),
        _ptr(workspace), nbytes, ctypes.byref(dbg) if dbg is not None else None,
        _stream(stream)))


def pot_append_decode_attention_v8(fmt: pot_format, engine: int, q, k_new, v_new, codes_se,
                                   codes_m, key_scale, v_u8, v_exp, t_cap: int, kv_head_of_q,
                                   B: int, Hq: int, Hkv: int, T: int, out, workspace,
                                   ws_bytes=None, dbg: pot_debug | None = None,
                                   stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_append_decode_attention_v8(
        ctypes.byref(fmt), int(engine), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(codes_se),
        _ptr(codes_m), _ptr(key_scale), _ptr(v_u8), _ptr(v_exp), int(t_cap), hp, B, Hq, Hkv, T,
        _ptr(out), _ptr(workspace), nbytes, ctypes.byref(dbg) if dbg is not None else None,
        _stream(stream)))


def pot_ds4a_decode_attention(fmt: pot_format, q, codes_se, key_scale, v_fp16, t_cap: int,
                              kv_head_of_q, B: int, Hq: int, Hkv: int, T: int, out,
                              workspace, ws_bytes=None, dbg: pot_debug | None = None,
                              stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_ds4a_decode_attention(
        ctypes.byref(fmt), _ptr(q), _ptr(codes_se), _ptr(key_scale), _ptr(v_fp16),
        int(t_cap), hp, B, Hq, Hkv, T, _ptr(out), _ptr(workspace), nbytes,
        ctypes.byref(dbg) if dbg is not None else None, _stream(stream)))


def pot_dot_decode_attention(fmt: pot_format, q, codes_se, codes_m, key_scale, v_fp16,
                             t_cap: int, kv_head_of_q, B: int, Hq: int, Hkv: int, T: int, out,
                             workspace, ws_bytes=None, dbg: pot_debug | None = None,
                             stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_dot_decode_attention(
        ctypes.byref(fmt), _ptr(q), _ptr(codes_se), _ptr(codes_m), _ptr(key_scale),
        _ptr(v_fp16), int(t_cap), hp, B, Hq, Hkv, T, _ptr(out), _ptr(workspace), nbytes,
        ctypes.byref(dbg) if dbg is not None else None, _stream(stream)))


def pot_int8_encode_keys(k_fp16, n_rows: int, out_row_stride: int, hadamard: int,
                         key_scale, codes, stream=None) -> None:
    _check(_lib.pot_int8_encode_keys(_ptr(k_fp16), int(n_rows),
                                     int(out_row_stride), int(hadamard),
                                     _ptr(key_scale), _ptr(codes),
                                     _stream(stream)))


def pot_int8_decode_attention(q, codes, key_scale, v_fp16, t_cap: int,
                              kv_head_of_q, B: int, Hq: int, Hkv: int, T: int,
                              hadamard: int, out, workspace, ws_bytes=None,
                              dbg: pot_debug | None = None, stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_int8_decode_attention(
        _ptr(q), _ptr(codes), _ptr(key_scale), _ptr(v_fp16), int(t_cap), hp,
        B, Hq, Hkv, T, int(hadamard), _ptr(out), _ptr(workspace), nbytes,
        ctypes.byref(dbg) if dbg is not None else None, _stream(stream)))


def pot_fp16_decode_attention(q, k_fp16, v_fp16, t_cap: int, kv_head_of_q,
                              B: int, Hq: int, Hkv: int, T: int, out, workspace,
                              ws_bytes=None, stream=None) -> None:
    _, hp = _heads(kv_head_of_q)
    nbytes = workspace.numel() * workspace.element_size() if ws_bytes is None else ws_bytes
    _check(_lib.pot_fp16_decode_attention(
        _ptr(q), _ptr(k_fp16), _ptr(v_fp16), int(t_cap), hp, B, Hq, Hkv, T,
        _ptr(out), _ptr(workspace), nbytes, _stream(stream)))


# ---- buffer helpers (allocation only, torch device memory) -----------------
def alloc_pot_cache(B: int, Hkv: int, t_cap: int, mant_bits: int, device):
    """Zeroed cache buffers in the library's row layout.

    Returns dict(codes_se uint8 [B,Hkv,t_cap,32], codes_m uint8
    [B,Hkv,t_cap,8k] or None, key_scale fp32 [B,Hkv,t_cap])."""
    import torch
    se = torch.zeros((B, Hkv, t_cap, HEAD_DIM // 2), dtype=torch.uint8, device=device)
    cm = (torch.zeros((B, Hkv, t_cap, 8 * mant_bits), dtype=torch.uint8, device=device)
          if mant_bits else None)
    sc = torch.zeros((B, Hkv, t_cap), dtype=torch.float32, device=device)
    return dict(codes_se=se, codes_m=cm, key_scale=sc)


def alloc_value_cache(B: int, Hkv: int, t_cap: int, device):
    """Value cache of B*Hkv sequences of t_cap tokens (token-interleaved)."""
    import torch
    return torch.zeros((B, Hkv, t_cap, HEAD_DIM), dtype=torch.float16, device=device)


def alloc_value_cache_int8(B: int, Hkv: int, t_cap: int, device):
    """INT8 value cache: (value bytes uint8 [B,Hkv,t_cap,64] token-interleaved,
    exponents int8 [B,Hkv,t_cap])."""
    import torch
    return (torch.zeros((B, Hkv, t_cap, HEAD_DIM), dtype=torch.uint8, device=device),
            torch.zeros((B, Hkv, t_cap), dtype=torch.int8, device=device))


def alloc_workspace(nbytes: int, device):
    """Workspace buffer for the decode calls (zero-filled; the kernels write
    every word they read, so any contents would do)."""
    import torch
    return torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=device)
