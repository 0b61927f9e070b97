"""Benchmark: TinyLlama-1.1B-shaped decode step with PoT-4 key caches.

One step = 22 layers, each: append the new token's key and value to that
layer's cache (pot_encode_keys and pot_store_values, one row per (batch, kv
head)) and run single-token decode attention over T keys
(pot_decode_attention). 32 query heads, 4 kv
heads, d = 64, fp16 values, synthetic seeded inputs resident in HBM before the
timed region. Every layer has its own cache, so consecutive calls never hit
the previous layer's data in the 256 MB last-level cache.

Prints one JSON line: keys scored per second (B * Hq * T * layers per step),
the roofline of the decode kernel (algorithmic bytes per launch / mean launch
time from HIP events on the launch stream), speed-up over the in-repo fp16
and INT8 kernels, and the CPU oracle timed on host cores on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HQ, HKV, D = 32, 4, 64
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "decode_pot4_b64_t32768_traffic.txt")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_09208_amd", "csrc", "decode.hip")


def row_bytes(mant_bits: int) -> int:
    """Algorithmic HBM bytes per cache row: codes + fp32 scale + fp16 V."""
    return 32 + 8 * mant_bits + 4 + 2 * D


def algorithmic_bytes(B: int, T: int, mant_bits: int) -> int:
    return B * HKV * T * row_bytes(mant_bits) + B * HQ * D * 4 * 2  # + q in, O out


def source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(os.path.dirname(KERNEL_SRC))):
        with open(os.path.join(os.path.dirname(KERNEL_SRC), name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def read_traffic():
    """HBM bytes per launch measured with rocprofv3 counters, if they were
    taken on the current kernel sources; otherwise None."""
    if not os.path.exists(PROFILE_TRAFFIC):
        return None
    vals = {}
    for line in open(PROFILE_TRAFFIC):
        if ":" in line:
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_digest") != source_digest():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(T: int, budget_s: float) -> dict:
    """The oracle (plain C, one thread) on (batch, kv-head) slices of the same
    workload: append-encode one key row, then decode attention of the G = 8
    query heads over T PoT-4 keys. Slices repeat until budget_s is spent."""
    import numpy as np

    import oracle
    from workloads import make_decode_inputs

    G = HQ // HKV
    d = make_decode_inputs(1234, B=1, Hq=G, Hkv=1, T=T)
    rows = d["k_bits"].reshape(-1, D)
    se, cm, sc = oracle.encode_keys(rows)
    n = 0
    t0 = time.perf_counter()
    while True:
        oracle.encode_keys(rows[-1:])
        oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], T, np.zeros(G, np.int32),
                          1, G, 1, T)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return {"value": n * G * T / el, "unit": "keys/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} (batch, kv-head) slices of T={T}: 1 appended key + "
                      f"{G} query heads over {T} PoT-4 keys, {el:.1f} s, 1 thread"}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--seq", type=int, default=32768)
    ap.add_argument("--layers", type=int, default=22)
    ap.add_argument("--mant-bits", type=int, default=0)
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--no-compare", action="store_true")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run device-to-device copies of BYTES bytes (calibrates "
                         "the FETCH_SIZE / WRITE_SIZE counters against a known size)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the decode path shards over (batch, kv head) with no communication; "
              "see DESIGN.md)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import paper_2609_09208_amd as pa
    from workloads import make_decode_inputs_device

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.copy_probe:
        n = args.copy_probe
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "copies": 3}), flush=True)
        return 0
    B, T, L, k = args.batch, args.seq, args.layers, args.mant_bits
    G = HQ // HKV
    fmt = pa.make_format(mant_bits=k, frac_bits=7)
    layers = []
    for layer in range(L):
        d = make_decode_inputs_device(1000 + layer, B, HQ, HKV, T, dev)
        cache = pa.alloc_pot_cache(B, HKV, T, k, dev)
        pa.pot_encode_keys(fmt, d["k"], B * HKV * T, 1, 0, cache["key_scale"],
                           cache["codes_se"], cache["codes_m"])
        vcache = pa.alloc_value_cache(B, HKV, T, dev)
        pa.pot_store_values(d["v"], B * HKV, T, T, 0, vcache)
        new_k = d["k"][:, :, T - 1].contiguous()  # the appended token's key
        new_v = d["v"][:, :, T - 1].contiguous()  # and value
        keep_k16 = d["k"] if (not args.no_compare and layer < 4) else None
        layers.append(dict(q=d["q"], v=vcache, new_k=new_k, new_v=new_v, k16=keep_k16,
                           **cache))
        del d
    heads = np.arange(HQ, dtype=np.int32) // G
    out = torch.empty((B, HQ, D), dtype=torch.float32, device=dev)
    ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, HQ, HKV, T), dev)
    torch.cuda.synchronize()

    def step(events=None):
        for i, c in enumerate(layers):
            pos = T - 1
            pa.pot_encode_keys(fmt, c["new_k"], B * HKV, T, 0, c["key_scale"].view(-1)[pos:],
                               c["codes_se"].view(-1, 32)[pos:],
                               c["codes_m"].view(-1, 8 * k)[pos:] if k else None)
            pa.pot_store_values(c["new_v"], B * HKV, 1, T, pos, c["v"])
            if events is not None:
                events[i][0].record()
            pa.pot_decode_attention(fmt, c["q"], c["codes_se"], c["codes_m"], c["key_scale"],
                                    c["v"], T, heads, B, HQ, HKV, T, out, ws)
            if events is not None:
                events[i][1].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(L)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(ev[s])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    kern_ms = [a.elapsed_time(b) for row in ev for (a, b) in row]
    kern_s = float(np.mean(kern_ms)) / 1e3
    ms_step = elapsed / args.steps * 1e3
    keys_per_step = B * HQ * T * L
    value = keys_per_step * args.steps / elapsed
    alg = algorithmic_bytes(B, T, k)
    achieved = alg / kern_s / 1e9
    traffic = read_traffic()

    result = {
        "metric": "decode-attention keys scored/s and achieved HBM GB/s at T=32k (PoT-4)",
        "value": value, "unit": "keys/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int32+fp32",
        "data": "synthetic",
        "config": {"workload": f"TinyLlama-1.1B-shaped {L}-layer decode step, "
                               f"PoT-{'4' if k == 0 else 'M%d' % k} keys (append + attend), "
                               f"fp16 V, B={B}, T={T}, Hq={HQ}, Hkv={HKV}, d={D}",
                   "B": B, "T": T, "layers": L, "Hq": HQ, "Hkv": HKV, "head_dim": D,
                   "mant_bits": k, "frac_bits": 7, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic,
                     "kernel": "potattn::decode_kernel<PoT,G=8>",
                     "alg_bytes_per_launch": alg, "launch_us": kern_s * 1e6,
                     "keys_scored_per_s_kernel": B * HQ * T / kern_s},
    }

    if not args.no_compare:
        # in-repo comparators on the same shape, rotating over 4 layer caches
        comp = {}
        cl = layers[:4]
        n8 = B * HKV * T
        i8 = [dict(codes=torch.empty((n8, D), dtype=torch.int8, device=dev),
                   sc=torch.empty(n8, dtype=torch.float32, device=dev)) for _ in cl]
        for c, x in zip(cl, i8):
            pa.pot_int8_encode_keys(c["k16"], n8, 1, 0, x["sc"], x["codes"])

        def timed(fn, reps=10):
            for _ in range(2):
                for c_i in range(len(cl)):
                    fn(c_i)
            torch.cuda.synchronize()
            s_ev, e_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s_ev.record()
            for _ in range(reps):
                for c_i in range(len(cl)):
                    fn(c_i)
            e_ev.record()
            torch.cuda.synchronize()
            return s_ev.elapsed_time(e_ev) / (reps * len(cl)) * 1e3  # us

        pot_us = timed(lambda i: pa.pot_decode_attention(
            fmt, cl[i]["q"], cl[i]["codes_se"], cl[i]["codes_m"], cl[i]["key_scale"],
            cl[i]["v"], T, heads, B, HQ, HKV, T, out, ws))
        f16_us = timed(lambda i: pa.pot_fp16_decode_attention(
            cl[i]["q"], cl[i]["k16"], cl[i]["v"], T, heads, B, HQ, HKV, T, out, ws))
        i8_us = timed(lambda i: pa.pot_int8_decode_attention(
            cl[i]["q"], i8[i]["codes"], i8[i]["sc"], cl[i]["v"], T, heads, B, HQ, HKV, T, 0,
            out, ws))
        comp = {"pot_us_per_layer": pot_us, "fp16_us_per_layer": f16_us,
                "int8_us_per_layer": i8_us, "speedup_vs_fp16": f16_us / pot_us,
                "speedup_vs_int8": i8_us / pot_us,
                "fp16_hbm_frac": (B * HKV * T * 256 + B * HQ * D * 8) / (f16_us * 1e-6) / 1e9
                / HBM_PEAK_GBS,
                "int8_hbm_frac": (B * HKV * T * 196 + B * HQ * D * 8) / (i8_us * 1e-6) / 1e9
                / HBM_PEAK_GBS}
        result["comparators"] = comp

    if args.cpu_budget > 0:
        result["cpu_baseline"] = cpu_baseline(T, args.cpu_budget)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
