"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bar: codes, key scales, q^, Delta, int32 scores and integer maxima (final and
per split) bit-exact; O within max-abs 2e-3 (fp32 accumulation). Workloads
follow the paper's TinyLlama-1.1B decode shape (32 query heads, 4 kv heads,
d = 64) with seeded synthetic inputs (workloads.py)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_09208_amd as pa
from parity_util import (DEV, O_TOL, assert_pot_parity, gpu_encode, gpu_pot_decode,
                         oracle_pot, store_values, to_dev)
from workloads import head_map, make_decode_inputs, make_decode_inputs_device

pytestmark = pytest.mark.gpu


def _all_fp16_rows():
    return np.arange(65536, dtype=np.uint32).astype(np.uint16).reshape(1024, 64)


# ---- encoder ----------------------------------------------------------------
@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
def test_encode_every_fp16_pattern(k):
    rows = _all_fp16_rows()
    for s in (1.0, 0.001, 3.7, 65504.0, 2.0 ** -20, 0.0):
        sc = np.full(1024, s, np.float32)
        g = gpu_encode(rows, k, key_scale=sc)
        o = oracle.encode_keys(rows, mant_bits=k, key_scale=sc)
        assert np.array_equal(g[0], o[0]), (k, s)
        if k:
            assert np.array_equal(g[1], o[1]), (k, s)


def _f32(bits):
    return np.array(bits, np.uint32).view(np.float32)


# Scales at the edges of the one-reciprocal path: all-ones mantissas (where a
# Newton step from the hardware reciprocal can land on a tie), the ends of the
# normal-reciprocal range [2^-126, 2^126] and one ulp past them, subnormal,
# largest finite, infinite, NaN and negative scales.
_EDGE_SCALES = _f32([0x3FFFFFFF, 0x3F7FFFFF, 0x4B7FFFFF, 0x37FFFFFF, 0x00FFFFFF, 0x7E7FFFFF,
                     0x7E800000, 0x7E800001, 0x00800000, 0x007FFFFF, 0x00000001, 0x7F7FFFFF,
                     0x7F800000, 0x7FC00000, 0xBF800000])


@pytest.mark.parametrize("k", [0, 1, 4])
def test_encode_every_fp16_pattern_edge_scales(k):
    rows = _all_fp16_rows()
    for s in _EDGE_SCALES:
        sc = np.full(1024, s, np.float32)
        g = gpu_encode(rows, k, key_scale=sc)
        o = oracle.encode_keys(rows, mant_bits=k, key_scale=sc)
        assert np.array_equal(g[0], o[0]), (k, hex(int(np.float32(s).view(np.uint32))))
        if k:
            assert np.array_equal(g[1], o[1]), (k, s)


@pytest.mark.parametrize("k", [0, 2])
def test_encode_every_fp16_pattern_random_scales(k):
    # one log-uniform scale per row: many distinct reciprocals on the fast path
    rng = np.random.default_rng(11 + k)
    rows = _all_fp16_rows()[rng.permutation(1024)]
    sc = np.exp2(rng.uniform(-30.0, 20.0, 1024)).astype(np.float32)
    sc[::7] = (sc[::7].view(np.uint32) | np.uint32(0x7FFFFF)).view(np.float32)
    g = gpu_encode(rows, k, key_scale=sc)
    o = oracle.encode_keys(rows, mant_bits=k, key_scale=sc)
    assert np.array_equal(g[0], o[0])
    if k:
        assert np.array_equal(g[1], o[1])


@pytest.mark.parametrize("k", [0, 1, 4])
def test_encode_hadamard_with_caller_scales(k):
    # the rotation followed by caller scales (scale mode 1): one log-uniform
    # scale per row, every fp16 pattern, shuffled into rows; ratios of the
    # rotated elements span [0, 2) and beyond
    rng = np.random.default_rng(31 + k)
    flat = _all_fp16_rows().reshape(-1)
    rows = flat[rng.permutation(flat.size)].reshape(1024, 64)
    sc = np.exp2(rng.uniform(-12.0, 16.0, 1024)).astype(np.float32)
    g = gpu_encode(rows, k, True, key_scale=sc)
    o = oracle.encode_keys(rows, mant_bits=k, hadamard=True, key_scale=sc)
    assert np.array_equal(g[0], o[0])
    if k:
        assert np.array_equal(g[1], o[1])


@pytest.mark.parametrize("k,had", [(0, False), (0, True), (1, False), (4, True)])
def test_encode_absmax_every_fp16_pattern(k, had):
    # row scales from the rows themselves, over every fp16 pattern: in order
    # (rows of only NaNs, a row holding infinity and NaNs, rows of subnormals)
    # and shuffled (NaN and infinity mixed into ordinary rows)
    rng = np.random.default_rng(23)
    flat = _all_fp16_rows().reshape(-1)
    for rows in (flat.reshape(1024, 64), flat[rng.permutation(flat.size)].reshape(1024, 64)):
        g = gpu_encode(rows, k, had)
        o = oracle.encode_keys(rows, mant_bits=k, hadamard=had)
        assert np.array_equal(g[0], o[0])
        if k:
            assert np.array_equal(g[1], o[1])
        assert np.array_equal(g[2].view(np.uint32), o[2].view(np.uint32))


@pytest.mark.parametrize("k,had", [(0, False), (1, False), (4, False), (0, True),
                                   (1, True), (4, True)])
def test_encode_absmax_rows(k, had):
    d = make_decode_inputs(100 + k, B=2, Hq=8, Hkv=4, T=1000)
    rows = d["k_bits"].reshape(-1, 64)
    g = gpu_encode(rows, k, had)
    o = oracle.encode_keys(rows, mant_bits=k, hadamard=had)
    assert np.array_equal(g[0], o[0])
    if k:
        assert np.array_equal(g[1], o[1])
    assert np.array_equal(g[2].view(np.uint32), o[2].view(np.uint32))


def test_encode_append_with_row_stride():
    # append one token (position t) to each of B*Hkv sequences of a t_cap cache
    B, Hkv, t_cap, t, k = 3, 4, 50, 17, 2
    rng = np.random.default_rng(5)
    new = rng.standard_normal((B * Hkv, 64)).astype(np.float16).view(np.uint16)
    fmt = pa.make_format(k)
    cache = pa.alloc_pot_cache(B, Hkv, t_cap, k, DEV)
    kd = to_dev(new).view(torch.float16)
    se, cm, sc = cache["codes_se"], cache["codes_m"], cache["key_scale"]
    pa.pot_encode_keys(fmt, kd, B * Hkv, t_cap, 0,
                       sc.view(-1)[t:], se.view(-1, 32)[t:], cm.view(-1, 8 * k)[t:])
    torch.cuda.synchronize()
    o_se, o_cm, o_sc = oracle.encode_keys(new, mant_bits=k)
    g_se = se.cpu().numpy().reshape(B * Hkv, t_cap, 32)
    g_cm = cm.cpu().numpy().reshape(B * Hkv, t_cap, 8 * k)
    g_sc = sc.cpu().numpy().reshape(B * Hkv, t_cap)
    assert np.array_equal(g_se[:, t], o_se) and np.array_equal(g_cm[:, t], o_cm)
    assert np.array_equal(g_sc[:, t], o_sc)
    # nothing else written
    others = np.ones(t_cap, bool)
    others[t] = False
    assert not g_se[:, others].any() and not g_sc[:, others].any()


@pytest.mark.parametrize("had", [False, True])
def test_int8_encode(had):
    d = make_decode_inputs(7, B=1, Hq=8, Hkv=4, T=700)
    rows = d["k_bits"].reshape(-1, 64)
    n = rows.shape[0]
    codes = torch.empty((n, 64), dtype=torch.int8, device=DEV)
    sc = torch.empty(n, dtype=torch.float32, device=DEV)
    pa.pot_int8_encode_keys(to_dev(rows).view(torch.float16), n, 1, int(had), sc, codes)
    torch.cuda.synchronize()
    oc, osc = oracle.int8_encode_keys(rows, hadamard=had)
    assert np.array_equal(codes.cpu().numpy(), oc)
    assert np.array_equal(sc.cpu().numpy().view(np.uint32), osc.view(np.uint32))


def test_store_values_layout_and_append():
    # token t, dim m of sequence q at (q*t_cap + (t//8)*8)*64 + m*8 + t%8
    rng = np.random.default_rng(6)
    n_seq, t_cap, T = 3, 48, 37
    v = rng.standard_normal((n_seq, T, 64)).astype(np.float16)
    cache = torch.full((n_seq * t_cap * 64,), 7.0, dtype=torch.float16, device=DEV)
    pa.pot_store_values(to_dev(v), n_seq, T, t_cap, 0, cache)
    new = rng.standard_normal((n_seq, 1, 64)).astype(np.float16)
    pa.pot_store_values(to_dev(new), n_seq, 1, t_cap, T, cache)  # append token T
    torch.cuda.synchronize()
    got = cache.cpu().numpy().reshape(n_seq, t_cap // 8, 64, 8)
    logical = got.transpose(0, 1, 3, 2).reshape(n_seq, t_cap, 64)
    assert np.array_equal(logical[:, :T], v)
    assert np.array_equal(logical[:, T], new[:, 0])
    assert (logical[:, T + 1:] == 7.0).all()  # untouched


# ---- decode: the paper's configurations ---------------------------------------
def test_tiny_single_head_pot4():
    # d = 64, T = 256, batch 1, one head; K and q N(0, 1), V fp16 N(0, 1)
    d = make_decode_inputs(0, B=1, Hq=1, Hkv=1, T=256, channel_scale=False)
    err, _ = assert_pot_parity(d)
    print(f"tiny PoT-4 O max-abs err {err:.3e}")


def test_tiny_single_head_head_wide_scale():
    # one caller-given scale per head (scale mode 1): the head's absmax
    d = make_decode_inputs(1, B=1, Hq=1, Hkv=1, T=256, channel_scale=False)
    kf = d["k_bits"].view(np.float16).astype(np.float32)
    s = np.full(256, np.abs(kf).max(), np.float32)
    err, _ = assert_pot_parity(d, key_scale=s)
    print(f"tiny head-scale O max-abs err {err:.3e}")


def test_tinyllama_layer_t4096_pot4():
    d = make_decode_inputs(2, B=1, Hq=32, Hkv=4, T=4096)
    err, g = assert_pot_parity(d)
    print(f"T=4096 PoT-4 splits={g['n_splits']} O err {err:.3e}")


def test_tinyllama_layer_t32768_potm1():
    d = make_decode_inputs(3, B=1, Hq=32, Hkv=4, T=32768)
    err, g = assert_pot_parity(d, mant_bits=1)
    print(f"T=32768 PoT-M1 splits={g['n_splits']} O err {err:.3e}")


def test_batch8_hadamard_potm4_reduced_T():
    d = make_decode_inputs(4, B=8, Hq=32, Hkv=4, T=2048)
    err, g = assert_pot_parity(d, mant_bits=4, hadamard=True)
    print(f"B=8 T=2048 H+PoT-M4 O err {err:.3e}")


def _sampled_full_size(B, T, mant_bits, hadamard, samples, seed):
    """Full-size launch as the benchmark times it (planner splits, no taps);
    sampled (b, kv-head) slices checked against the oracle."""
    Hq, Hkv = 32, 4
    d = make_decode_inputs_device(seed, B, Hq, Hkv, T, DEV)
    fmt = pa.make_format(mant_bits, 7, hadamard)
    cache = pa.alloc_pot_cache(B, Hkv, T, mant_bits, DEV)
    rows = B * Hkv * T
    pa.pot_encode_keys(fmt, d["k"], rows, 1, 0, cache["key_scale"], cache["codes_se"],
                       cache["codes_m"])
    vcache = pa.alloc_value_cache(B, Hkv, T, DEV)
    pa.pot_store_values(d["v"], B * Hkv, T, T, 0, vcache)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    pa.pot_decode_attention(fmt, d["q"], cache["codes_se"], cache["codes_m"],
                            cache["key_scale"], vcache, T, d["kv_head_of_q"], B, Hq, Hkv,
                            T, out, ws)
    torch.cuda.synchronize()
    G = Hq // Hkv
    worst = 0.0
    for (b, h) in samples:
        kb = d["k"][b, h].view(torch.uint16).cpu().numpy()
        vb = d["v"][b, h].view(torch.uint16).cpu().numpy()
        qs = d["q"][b, h * G:(h + 1) * G].cpu().numpy()
        o_se, o_cm, o_sc = oracle.encode_keys(kb, mant_bits=mant_bits, hadamard=hadamard)
        assert np.array_equal(cache["codes_se"][b, h].cpu().numpy(), o_se)
        if mant_bits:
            assert np.array_equal(cache["codes_m"][b, h].cpu().numpy(), o_cm)
        assert np.array_equal(cache["key_scale"][b, h].cpu().numpy(), o_sc)
        r = oracle.pot_decode(qs[None], o_se, o_cm, o_sc, vb, T, np.zeros(G, np.int32),
                              1, G, 1, T, mant_bits=mant_bits, hadamard=hadamard)
        err = float(np.abs(out[b, h * G:(h + 1) * G].cpu().numpy() - r["out"][0]).max())
        worst = max(worst, err)
    assert worst <= O_TOL, worst
    return worst


def test_full_size_b64_t32768_pot4_sampled():
    err = _sampled_full_size(64, 32768, 0, False, [(0, 0), (17, 3), (63, 2)], 10)
    print(f"B=64 T=32768 PoT-4 sampled O err {err:.3e}")


def test_longest_context_b1_t1m_pot4_sampled():
    # 2^20 keys per sequence (4096 tiles of 256 keys): the longest ranges per
    # split the planner makes, and the largest cache of the suite (4 * 2^20
    # rows, 512 MiB of values)
    err = _sampled_full_size(1, 1 << 20, 0, False, [(0, 0), (0, 3)], 12)
    print(f"B=1 T=2^20 PoT-4 sampled O err {err:.3e}")


def test_cache_offsets_beyond_4gib():
    # t_cap = 2^24 keys per sequence: the last sequences' rows start past
    # 2^27 rows, so their value bytes lie beyond 16 GiB and their code bytes
    # beyond 4 GiB (64-bit address arithmetic in every kernel); only the first
    # T keys of each sequence are attended
    B, Hq, Hkv, T, t_cap = 2, 32, 4, 1000, 1 << 24
    d = make_decode_inputs_device(13, B, Hq, Hkv, T, DEV, t_cap=t_cap)
    fmt = pa.make_format(1)
    cache = pa.alloc_pot_cache(B, Hkv, t_cap, 1, DEV)
    pa.pot_encode_keys(fmt, d["k"], B * Hkv * t_cap, 1, 0, cache["key_scale"],
                       cache["codes_se"], cache["codes_m"])
    vcache = pa.alloc_value_cache(B, Hkv, t_cap, DEV)
    pa.pot_store_values(d["v"], B * Hkv, t_cap, t_cap, 0, vcache)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    pa.pot_decode_attention(fmt, d["q"], cache["codes_se"], cache["codes_m"],
                            cache["key_scale"], vcache, t_cap, d["kv_head_of_q"], B, Hq, Hkv,
                            T, out, ws)
    torch.cuda.synchronize()
    G = Hq // Hkv
    for (b, h) in [(0, 0), (1, 3)]:
        kb = d["k"][b, h, :T].view(torch.uint16).cpu().numpy()
        vb = d["v"][b, h, :T].view(torch.uint16).cpu().numpy()
        qs = d["q"][b, h * G:(h + 1) * G].cpu().numpy()
        o_se, o_cm, o_sc = oracle.encode_keys(kb, mant_bits=1)
        assert np.array_equal(cache["codes_se"][b, h, :T].cpu().numpy(), o_se)
        assert np.array_equal(cache["codes_m"][b, h, :T].cpu().numpy(), o_cm)
        r = oracle.pot_decode(qs[None], o_se, o_cm, o_sc, vb, T, np.zeros(G, np.int32),
                              1, G, 1, T, mant_bits=1)
        err = float(np.abs(out[b, h * G:(h + 1) * G].cpu().numpy() - r["out"][0]).max())
        assert err <= O_TOL, err
    del d, cache, vcache
    torch.cuda.empty_cache()


def test_full_size_b8_t32768_hadamard_potm4_sampled():
    err = _sampled_full_size(8, 32768, 4, True, [(0, 1), (7, 3)], 11)
    print(f"B=8 T=32768 H+PoT-M4 sampled O err {err:.3e}")


# ---- edge cases ------------------------------------------------------------------
@pytest.mark.parametrize("T,t_cap", [(1, 8), (5, 16), (255, 256), (257, 320), (1000, 1032),
                                     (4099, 4104)])
def test_ragged_lengths_and_padding(T, t_cap):
    d = make_decode_inputs(20 + T, B=2, Hq=8, Hkv=2, T=T, t_cap=t_cap)
    assert_pot_parity(d, mant_bits=1)


@pytest.mark.parametrize("Hq,Hkv", [(1, 1), (4, 2), (8, 2), (32, 4), (16, 16)])
def test_group_sizes(Hq, Hkv):
    d = make_decode_inputs(30 + Hq, B=2, Hq=Hq, Hkv=Hkv, T=300)
    assert_pot_parity(d)


@pytest.mark.parametrize("k", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("G", [1, 2, 4, 8])
def test_every_mantissa_width_and_group(k, G):
    # every PoT / PoT-Mk score variant of the decode kernel (one per k and
    # group size), a ragged tail of 700 = 2 * 256 + 188 keys
    d = make_decode_inputs(60 + 8 * k + G, B=2, Hq=2 * G, Hkv=2, T=700, t_cap=704)
    assert_pot_parity(d, mant_bits=k)


def test_interleaved_head_map():
    d = make_decode_inputs(41, B=2, Hq=8, Hkv=2, T=300)
    d["kv_head_of_q"] = (np.arange(8) % 2).astype(np.int32)
    assert_pot_parity(d, mant_bits=2)


@pytest.mark.parametrize("F", [6, 12])
def test_head_room(F):
    d = make_decode_inputs(42, B=1, Hq=8, Hkv=1, T=600)
    assert_pot_parity(d, mant_bits=4 if F == 12 else 0, frac_bits=F)


def test_degenerate_rows_and_query():
    d = make_decode_inputs(43, B=2, Hq=8, Hkv=2, T=300)
    k = d["k_bits"].view(np.float16)
    k[0, 0, 10] = 0            # all-zero key row: s = 0, every code zero
    k[1, 1, 50:60] = 0
    k[0, 1, 7, :32] = 0        # half-zero row
    d["q"][1, 3] = 0           # zero query: Delta = 0, uniform weights
    assert_pot_parity(d, mant_bits=1)


@pytest.mark.parametrize("engine", ["sac", "ds4a"])
def test_scores_reach_the_bound(engine):
    # q^ = +-127 everywhere and keys of equal magnitudes (every code e = 0)
    # with the signs of the query (and the opposite ones): the scores are the
    # printed bound +-64 * 127 * 2^7 = +-1 040 384 (Sec. II-C); a third row
    # runs through every exponent and the zero code, a fourth is all zero
    d = make_decode_inputs(46, B=1, Hq=8, Hkv=1, T=64)
    rng = np.random.default_rng(46)
    sgn = np.where(rng.random(64) < 0.5, -1.0, 1.0)
    d["q"][0, 0] = sgn.astype(np.float32)
    k = d["k_bits"].view(np.float16)
    k[0, 0, 0] = sgn.astype(np.float16)
    k[0, 0, 1] = (-sgn).astype(np.float16)
    k[0, 0, 2] = (sgn * np.exp2(-(np.arange(64) % 8))).astype(np.float16)
    k[0, 0, 3] = 0
    _, g = assert_pot_parity(d, engine=engine)
    assert g["scores"][0, 0, 0] == 1040384 and g["scores"][0, 0, 1] == -1040384
    assert g["scores"][0, 0, 3] == 0


@pytest.mark.parametrize("S", [1, 2, 3, 7, 16])
def test_forced_splits(S):
    d = make_decode_inputs(44, B=1, Hq=32, Hkv=4, T=4000)
    err, g = assert_pot_parity(d, force_splits=S)
    tiles = -(-4000 // 256)
    split_len = -(-tiles // min(S, tiles)) * 256  # whole tiles per split
    assert g["split_len"] == split_len and g["n_splits"] == -(-4000 // split_len)


def test_split_invariance_and_determinism():
    d = make_decode_inputs(45, B=2, Hq=32, Hkv=4, T=3000)
    se, cm, sc = gpu_encode(d["k_bits"].reshape(-1, 64), 0)
    ms = []
    outs = []
    for S in (1, 4, 12, 12):
        g = gpu_pot_decode(d, se, cm, sc, force_splits=S)
        ms.append(g["m_final"])
        outs.append(g["out"])
    for m in ms[1:]:
        assert np.array_equal(m, ms[0])
    assert np.array_equal(outs[2], outs[3])  # run to run bit-identical
    assert np.abs(outs[0] - outs[1]).max() < 1e-5


@pytest.mark.parametrize("S", [1, 4])
def test_decode_kernel_events(S):
    # pot_debug.decode_begin / decode_end: the library records the caller's
    # events around the decode kernel alone; the output is unchanged and the
    # kernel's time lies inside the call's
    d = make_decode_inputs(47, B=4, Hq=32, Hkv=4, T=4096)
    B, Hq, Hkv, T = 4, 32, 4, 4096
    se, _, sc = gpu_encode(d["k_bits"].reshape(-1, 64), 0)
    fmt = pa.make_format(0)
    q, se_d, sc_d = to_dev(d["q"]), to_dev(se), to_dev(sc)
    v = store_values(d["v_bits"], B, Hkv, d["t_cap"])
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes_for_splits(B, Hq, Hkv, T, S), DEV)
    outs = []
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for with_events in (False, True):
        out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
        dbg = pa.pot_debug()
        dbg.force_splits = S
        if with_events:
            for e in ev:
                e.record()  # creates the HIP events
            dbg.decode_begin, dbg.decode_end = ev[1].cuda_event, ev[2].cuda_event
            ev[0].record()
        pa.pot_decode_attention(fmt, q, se_d, None, sc_d, v, d["t_cap"], d["kv_head_of_q"], B,
                                Hq, Hkv, T, out, ws, dbg=dbg)
        if with_events:
            ev[3].record()
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
        assert dbg.n_splits == S
    assert np.array_equal(outs[0], outs[1])
    call_ms, kern_ms = ev[0].elapsed_time(ev[3]), ev[1].elapsed_time(ev[2])
    assert 0 < kern_ms <= call_ms
    assert ev[0].elapsed_time(ev[1]) >= 0 and ev[2].elapsed_time(ev[3]) >= 0


# ---- comparison kernels ------------------------------------------------------------
@pytest.mark.parametrize("had", [False, True])
def test_int8_decode_parity(had):
    B, Hq, Hkv, T = 2, 32, 4, 2500
    d = make_decode_inputs(50, B=B, Hq=Hq, Hkv=Hkv, T=T)
    tc = d["t_cap"]
    rows = d["k_bits"].reshape(-1, 64)
    n = rows.shape[0]
    codes = torch.empty((n, 64), dtype=torch.int8, device=DEV)
    sc = torch.empty(n, dtype=torch.float32, device=DEV)
    pa.pot_int8_encode_keys(to_dev(rows).view(torch.float16), n, 1, int(had), sc, codes)
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    dbg = pa.pot_debug()
    taps = dict(qhat=torch.empty((B, Hq, 64), dtype=torch.int8, device=DEV),
                delta=torch.empty((B, Hq), dtype=torch.float32, device=DEV),
                scores=torch.empty((B, Hq, T), dtype=torch.int32, device=DEV),
                m_final=torch.empty((B, Hq), dtype=torch.int32, device=DEV))
    for k_, t_ in taps.items():
        setattr(dbg, k_, t_.data_ptr())
    pa.pot_int8_decode_attention(to_dev(d["q"]), codes, sc, store_values(d["v_bits"], B, Hkv, tc),
                                 tc, d["kv_head_of_q"], B, Hq, Hkv, T, int(had), out, ws, dbg=dbg)
    torch.cuda.synchronize()
    oc, osc = oracle.int8_encode_keys(rows, hadamard=had)
    r = oracle.int8_decode(d["q"], oc, osc, d["v_bits"], tc, d["kv_head_of_q"], B, Hq, Hkv, T,
                           hadamard=had)
    assert np.array_equal(taps["qhat"].cpu().numpy(), r["qhat"])
    assert np.array_equal(taps["scores"].cpu().numpy(), r["scores"])
    assert np.array_equal(taps["m_final"].cpu().numpy(), r["m_final"])
    assert np.abs(out.cpu().numpy() - r["out"]).max() <= O_TOL


def test_fp16_decode_parity():
    d = make_decode_inputs(51, B=2, Hq=32, Hkv=4, T=2500, t_cap=2600)
    assert d["t_cap"] % 8 == 0
    B, Hq, Hkv, T = 2, 32, 4, 2500
    out = torch.empty((B, Hq, 64), dtype=torch.float32, device=DEV)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
    pa.pot_fp16_decode_attention(to_dev(d["q"]), to_dev(d["k_bits"]).view(torch.float16),
                                 store_values(d["v_bits"], B, Hkv, 2600), 2600,
                                 d["kv_head_of_q"], B, Hq, Hkv, T, out, ws)
    torch.cuda.synchronize()
    r = oracle.fp16_decode(d["q"], d["k_bits"], d["v_bits"], 2600, d["kv_head_of_q"], B, Hq,
                           Hkv, T)
    err = float(np.abs(out.cpu().numpy() - r).max())
    assert err <= O_TOL, err
    print(f"fp16 O err {err:.3e}")
    # T = 2500 < t_cap = 2600: the tail group's tokens past T are never used


def test_status_errors_do_not_launch():
    # invalid arguments are rejected on the host even with real buffers
    d = make_decode_inputs(52, B=1, Hq=8, Hkv=1, T=10)
    q = to_dev(d["q"])
    with pytest.raises(pa.PotError) as ei:
        pa.pot_decode_attention(pa.make_format(frac_bits=3), q, q, None, q, q, 10,
                                d["kv_head_of_q"], 1, 8, 1, 10, q,
                                pa.alloc_workspace(1 << 16, DEV))
    assert ei.value.status == pa.POT_ERR_INVALID_ARG
