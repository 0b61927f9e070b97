"""The decode step under HIP graph capture.

A layer's call launches only kernels on the caller's stream (no allocation,
no memset, no host synchronisation), so a whole multi-layer decode step can be
captured once and replayed. The test captures a three-layer step (append the
new token's key and values, then decode, per layer; PoT-4, PoT-M1 and the INT8
value cache) with torch.cuda.CUDAGraph, replays it several times with eager
calls of the same library and synchronisations in between, and checks every
replay bit for bit against the eager step: outputs and the appended cache
rows. The append writes the same row T - 1 each time, so replays are
idempotent.
"""
import numpy as np
import pytest
import torch

import paper_2609_09208_amd as pa
from workloads import make_decode_inputs_device

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _layer(seed, B, Hq, Hkv, T, mant_bits, int8_values):
    d = make_decode_inputs_device(seed, B, Hq, Hkv, T, DEV)
    fmt = pa.make_format(mant_bits)
    c = pa.alloc_pot_cache(B, Hkv, T, mant_bits, DEV)
    pa.pot_encode_keys(fmt, d["k"], B * Hkv * T, 1, 0, c["key_scale"], c["codes_se"],
                       c["codes_m"])
    lay = dict(fmt=fmt, q=d["q"], heads=d["kv_head_of_q"], int8=int8_values,
               new_k=d["k"][:, :, T - 1].contiguous(), new_v=d["v"][:, :, T - 1].contiguous(),
               out=torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV),
               ws=pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV), **c)
    if int8_values:
        vu, ve = pa.alloc_value_cache_int8(B, Hkv, T, DEV)
        pa.pot_store_values_int8(d["v"], B * Hkv, T, T, 0, vu, ve)
        lay.update(vu=vu, ve=ve)
    else:
        v = pa.alloc_value_cache(B, Hkv, T, DEV)
        pa.pot_store_values(d["v"], B * Hkv, T, T, 0, v)
        lay.update(v=v)
    return lay


def _call(c, B, Hq, Hkv, T):
    if c["int8"]:
        pa.pot_append_decode_attention_v8(c["fmt"], 0, c["q"], c["new_k"], c["new_v"],
                                          c["codes_se"], c["codes_m"], c["key_scale"], c["vu"],
                                          c["ve"], T, c["heads"], B, Hq, Hkv, T, c["out"],
                                          c["ws"])
    else:
        pa.pot_append_decode_attention(c["fmt"], c["q"], c["new_k"], c["new_v"], c["codes_se"],
                                       c["codes_m"], c["key_scale"], c["v"], T, c["heads"], B,
                                       Hq, Hkv, T, c["out"], c["ws"])


def _snapshot(layers, T):
    snap = []
    for c in layers:
        s = dict(out=c["out"].cpu().numpy().copy(),
                 se=c["codes_se"][:, :, T - 1].cpu().numpy().copy(),
                 sc=c["key_scale"][:, :, T - 1].cpu().numpy().copy())
        if c["codes_m"] is not None:
            s["cm"] = c["codes_m"][:, :, T - 1].cpu().numpy().copy()
        snap.append(s)
    return snap


def _equal(a, b):
    return all(np.array_equal(x[k], y[k]) for x, y in zip(a, b) for k in x)


def test_graph_replays_equal_the_eager_step():
    B, Hq, Hkv, T = 4, 32, 4, 2000
    layers = [_layer(70, B, Hq, Hkv, T, 0, False), _layer(71, B, Hq, Hkv, T, 1, False),
              _layer(72, B, Hq, Hkv, T, 0, True)]

    def step():
        for c in layers:
            _call(c, B, Hq, Hkv, T)

    step()  # eager; also fills the library's per-variant occupancy cache
    torch.cuda.synchronize()
    eager = _snapshot(layers, T)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(4):
        for c in layers:
            c["out"].fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert _equal(_snapshot(layers, T), eager), f"replay {rep} differs from the eager step"
        # eager work of the same library between replays
        step()
        torch.cuda.synchronize()
        assert _equal(_snapshot(layers, T), eager), f"eager step after replay {rep} differs"
