"""GPU parity at full size, in the launch configuration the benchmark times.

B = 64, T = 32768, PoT-4 (the headline shape) and B = 8, T = 32768 with
Hadamard + PoT-M4: the planner's key splits, through both decode entry points
(pot_decode_attention and the benchmark's pot_append_decode_attention, which
appends the token at T - 1 first); the decoded-weight entry point
pot_dot_decode_attention at Hadamard + PoT-M4 (B = 8) and PoT-M1 (B = 64). Each call runs twice on the same inputs:
plain (the timed kernel) and with the score taps on (the instrumented build
of the same kernel source, same split plan). Checked:
* the two outputs are bit-identical with four-wave workgroups; the CU-wide
  variant (one workgroup per CU, tiles claimed from a counter) sums each
  wave's tiles in the order it claimed them, so there the two agree to
  fp32 rounding (1e-5);
* on sampled (batch, kv head) slices: q^, Delta, the int32 scores of all G
  query heads over all T keys, the final integer maximum and the maximum of
  every split equal the oracle's bit for bit, and O is within 2e-3.
The oracle encodes the slice's fp16 keys itself (the appended key included).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_09208_amd as pa
from parity_util import DEV, O_TOL
from workloads import POISON_K, POISON_V, make_decode_inputs_device

pytestmark = pytest.mark.gpu

HQ, HKV = 32, 4
G = HQ // HKV


def _run(fmt, d, cache, v, append, dbg, engine="sac"):
    B, T = d["B"], d["T"]
    out = torch.empty((B, HQ, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, HQ, HKV, T), DEV)
    if engine == "dot":
        assert not append
        pa.pot_dot_decode_attention(fmt, d["q"], cache["codes_se"], cache["codes_m"],
                                    cache["key_scale"], v, T, d["kv_head_of_q"], B, HQ, HKV,
                                    T, out, ws, dbg=dbg)
    elif append:
        pa.pot_append_decode_attention(fmt, d["q"], d["k_new"], d["v_new"], cache["codes_se"],
                                       cache["codes_m"], cache["key_scale"], v, T,
                                       d["kv_head_of_q"], B, HQ, HKV, T, out, ws, dbg=dbg)
    else:
        pa.pot_decode_attention(fmt, d["q"], cache["codes_se"], cache["codes_m"],
                                cache["key_scale"], v, T, d["kv_head_of_q"], B, HQ, HKV, T,
                                out, ws, dbg=dbg)
    return out


def _check(B, T, mant_bits, hadamard, append, samples, seed, engine="sac"):
    print(f"full-size taps B={B} T={T} k={mant_bits} had={hadamard} append={append} "
          f"engine={engine}", flush=True)
    d = make_decode_inputs_device(seed, B, HQ, HKV, T, DEV)
    fmt = pa.make_format(mant_bits, 7, hadamard)
    rows = B * HKV * T

    def fresh_cache():
        cache = pa.alloc_pot_cache(B, HKV, T, mant_bits, DEV)
        k = d["k"]
        if append:  # row T - 1 starts as a poison key the call must overwrite
            k = k.clone()
            k[:, :, T - 1] = POISON_K
        pa.pot_encode_keys(fmt, k, rows, 1, 0, cache["key_scale"], cache["codes_se"],
                           cache["codes_m"])
        v = pa.alloc_value_cache(B, HKV, T, DEV)
        vs = d["v"]
        if append:
            vs = vs.clone()
            vs[:, :, T - 1] = POISON_V
        pa.pot_store_values(vs, B * HKV, T, T, 0, v)
        return cache, v

    if append:
        d["k_new"] = d["k"][:, :, T - 1].contiguous()
        d["v_new"] = d["v"][:, :, T - 1].contiguous()
    # the plain call, as timed; the planner's split length comes back in dbg
    cache, v = fresh_cache()
    plan = pa.pot_debug()
    out_plain = _run(fmt, d, cache, v, append, plan, engine)
    torch.cuda.synchronize()
    n_splits, split_len = plan.n_splits, plan.split_len
    del cache, v
    # the instrumented call on a fresh copy of the same cache
    cache, v = fresh_cache()
    taps = dict(qhat=torch.empty((B, HQ, 64), dtype=torch.int8, device=DEV),
                delta=torch.empty((B, HQ), dtype=torch.float32, device=DEV),
                scores=torch.empty((B, HQ, T), dtype=torch.int32, device=DEV),
                m_final=torch.empty((B, HQ), dtype=torch.int32, device=DEV),
                m_split=torch.empty((B * HQ * n_splits,), dtype=torch.int32, device=DEV))
    dbg = pa.pot_debug()
    for name, t in taps.items():
        setattr(dbg, name, t.data_ptr())
    out_taps = _run(fmt, d, cache, v, append, dbg, engine)
    torch.cuda.synchronize()
    assert (dbg.n_splits, dbg.split_len, dbg.wg_waves) == (n_splits, split_len, plan.wg_waves)
    if plan.wg_waves == 4:
        assert torch.equal(out_plain.view(torch.int32), out_taps.view(torch.int32)), \
            "instrumented build differs from the timed one"
    else:
        diff = float((out_plain - out_taps).abs().max())
        assert diff <= 1e-5, f"instrumented build differs from the timed one by {diff}"
    m_split = taps["m_split"].view(B, HQ, n_splits)
    worst = 0.0
    for (b, h) in samples:
        kb = d["k"][b, h].view(torch.uint16).cpu().numpy()
        vb = d["v"][b, h].view(torch.uint16).cpu().numpy()
        qs = d["q"][b, h * G:(h + 1) * G].cpu().numpy()
        o_se, o_cm, o_sc = oracle.encode_keys(kb, mant_bits=mant_bits, hadamard=hadamard)
        assert np.array_equal(cache["codes_se"][b, h].cpu().numpy(), o_se)
        if mant_bits:
            assert np.array_equal(cache["codes_m"][b, h].cpu().numpy(), o_cm)
        assert np.array_equal(cache["key_scale"][b, h].cpu().numpy().view(np.uint32),
                              o_sc.view(np.uint32))
        r = oracle.pot_decode(qs[None], o_se, o_cm, o_sc, vb, T, np.zeros(G, np.int32),
                              1, G, 1, T, mant_bits=mant_bits, hadamard=hadamard,
                              split_len=split_len)
        hs = slice(h * G, (h + 1) * G)
        assert np.array_equal(taps["qhat"][b, hs].cpu().numpy(), r["qhat"][0])
        assert np.array_equal(taps["delta"][b, hs].cpu().numpy().view(np.uint32),
                              r["delta"][0].view(np.uint32))
        g_sc = taps["scores"][b, hs].cpu().numpy()
        bad = np.argwhere(g_sc != r["scores"][0])
        assert bad.size == 0, f"{len(bad)} int32 scores differ, first {bad[:3].tolist()}"
        assert np.array_equal(taps["m_final"][b, hs].cpu().numpy(), r["m_final"][0])
        assert np.array_equal(m_split[b, hs].cpu().numpy(), r["m_split"][0])
        err = float(np.abs(out_plain[b, hs].cpu().numpy() - r["out"][0]).max())
        worst = max(worst, err)
    assert worst <= O_TOL, worst
    print(f"  splits={n_splits} x {split_len} keys, {plan.wg_waves} waves per workgroup, "
          f"{len(samples)} slices x {G} heads x "
          f"{T} scores bit-exact, O err {worst:.3e}", flush=True)
    del d, cache, v, taps
    torch.cuda.empty_cache()


@pytest.mark.parametrize("append", [False, True])
def test_full_size_b64_t32768_pot4_taps(append):
    _check(64, 32768, 0, False, append, [(0, 0), (31, 1), (63, 3)], 40 + append)


@pytest.mark.parametrize("append", [False, True])
def test_full_size_b8_t32768_hadamard_potm4_taps(append):
    _check(8, 32768, 4, True, append, [(0, 2), (7, 3)], 50 + append)


# the decoded-weight engine (pot_dot_decode_attention) at the PoT-Mk shapes
def test_full_size_b8_t32768_hadamard_potm4_dot_taps():
    _check(8, 32768, 4, True, False, [(1, 0), (6, 3)], 52, engine="dot")


def test_full_size_b64_t32768_potm1_dot_taps():
    _check(64, 32768, 1, False, False, [(0, 1), (40, 2), (63, 0)], 53, engine="dot")
