"""Seeded synthetic inputs shaped like the paper's decode workloads.

TinyLlama-1.1B-shaped decode attention (Sec. IV): 32 query heads, 4 KV heads,
head dimension 64, one query token per sequence, a KV cache of T tokens.
Captured post-RoPE tensors, model weights and WikiText are not available, so
keys are drawn as N(0, 1) times a per-channel scale from U[0.5, 4] (outlier
channels), values as N(0, 1), queries as N(0, 1).

This module holds no arithmetic of the method (no rotation, quantisation or
encoding): it is the one place both the GPU path's tests and the oracle get
their inputs from. Host generation uses numpy's PCG64 (``default_rng(seed)``)
in a fixed draw order; large device-resident workloads use torch's seeded
device generator, and the oracle then reads back the slices it checks.
"""
from __future__ import annotations

import numpy as np

HEAD_DIM = 64
# Value written into cache rows at positions t >= T (never attended): a key or
# value from these rows leaking into a result shows up as a gross error.
POISON_V = 60000.0
POISON_K = 30000.0


def head_map(Hq: int, Hkv: int) -> np.ndarray:
    """Contiguous GQA map: query head i is served by kv head i // (Hq/Hkv)."""
    G = Hq // Hkv
    return (np.arange(Hq, dtype=np.int32) // G).astype(np.int32)


def make_decode_inputs(seed: int, B: int, Hq: int, Hkv: int, T: int,
                       t_cap: int | None = None, channel_scale: bool = True,
                       v_dist: str = "normal") -> dict:
    """Host (numpy) inputs for one decode-attention call.

    Draw order: channel scale c [Hkv, 64] ~ U[0.5, 4] (if channel_scale),
    z [B, Hkv, T, 64] ~ N(0, 1), v [B, Hkv, T, 64] ~ N(0, 1),
    q [B, Hq, 64] ~ N(0, 1). K = fp16(z * c), V = fp16(v).
    Rows T..t_cap-1 of each sequence hold POISON values; t_cap defaults to T
    rounded up to a multiple of 8 (the value cache's token groups).

    Returns q (fp32), k_bits / v_bits (uint16 fp16 bit patterns,
    [B, Hkv, t_cap, 64]), kv_head_of_q (int32 [Hq]) and the shape fields."""
    t_cap = max(8, -(-T // 8) * 8) if t_cap is None else int(t_cap)
    assert t_cap >= T >= 0
    rng = np.random.default_rng(seed)
    if channel_scale:
        c = rng.uniform(0.5, 4.0, size=(Hkv, HEAD_DIM)).astype(np.float32)
    else:
        c = np.ones((Hkv, HEAD_DIM), np.float32)
    z = rng.standard_normal((B, Hkv, T, HEAD_DIM), dtype=np.float32)
    if v_dist == "normal":
        v = rng.standard_normal((B, Hkv, T, HEAD_DIM), dtype=np.float32)
    else:
        raise ValueError(v_dist)
    q = rng.standard_normal((B, Hq, HEAD_DIM), dtype=np.float32)
    k16 = np.full((B, Hkv, t_cap, HEAD_DIM), POISON_K, np.float16)
    v16 = np.full((B, Hkv, t_cap, HEAD_DIM), POISON_V, np.float16)
    k16[:, :, :T] = (z * c[None, :, None, :]).astype(np.float16)
    v16[:, :, :T] = v.astype(np.float16)
    return dict(q=q, k_bits=k16.view(np.uint16), v_bits=v16.view(np.uint16),
                kv_head_of_q=head_map(Hq, Hkv), B=B, Hq=Hq, Hkv=Hkv, T=T,
                t_cap=t_cap)


def make_query(seed: int, B: int, Hq: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.standard_normal((B, Hq, HEAD_DIM), dtype=np.float32)


def make_decode_inputs_device(seed: int, B: int, Hq: int, Hkv: int, T: int,
                              device, t_cap: int | None = None,
                              channel_scale: bool = True):
    """Device-resident inputs for large workloads (torch seeded generator).

    Same distributions as make_decode_inputs; positions >= T are poisoned.
    Returns torch tensors q (fp32 [B,Hq,64]), k, v (fp16 [B,Hkv,t_cap,64]),
    and kv_head_of_q (numpy int32)."""
    import torch
    t_cap = T if t_cap is None else int(t_cap)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    if channel_scale:
        c = torch.rand((Hkv, HEAD_DIM), generator=g, device=device) * 3.5 + 0.5
    else:
        c = torch.ones((Hkv, HEAD_DIM), device=device)
    k = torch.full((B, Hkv, t_cap, HEAD_DIM), POISON_K, dtype=torch.float16,
                   device=device)
    v = torch.full((B, Hkv, t_cap, HEAD_DIM), POISON_V, dtype=torch.float16,
                   device=device)
    for b in range(B):  # per batch row keeps the fp32 staging buffer small
        z = torch.randn((Hkv, T, HEAD_DIM), generator=g, device=device)
        k[b, :, :T] = (z * c[:, None, :]).to(torch.float16)
        vv = torch.randn((Hkv, T, HEAD_DIM), generator=g, device=device)
        v[b, :, :T] = vv.to(torch.float16)
        del z, vv
    q = torch.randn((B, Hq, HEAD_DIM), generator=g, device=device)
    return dict(q=q, k=k, v=v, kv_head_of_q=head_map(Hq, Hkv), B=B, Hq=Hq,
                Hkv=Hkv, T=T, t_cap=t_cap)
