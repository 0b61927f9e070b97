"""Benchmark: TinyLlama-1.1B-shaped decode steps over PoT key caches.

Default (the headline JSON line): one step = 22 layers at B = 64, T = 32768,
PoT-4 keys, fp16 values. Each layer makes one call,
pot_append_decode_attention, which appends the new token's key (encoded to
PoT codes) and values at position T - 1 of every (batch, kv head) sequence of
that layer's cache and runs single-token decode attention over the T keys.

32 query heads, 4 kv heads, d = 64. Inputs are synthetic, seeded, and resident
in HBM before the timed region. Every layer has its own cache, so consecutive
calls never hit the previous layer's data in the 256 MB last-level cache. Each
timed phase starts with about 0.3 s of untimed steps, so that the GPU runs at
the clocks of back-to-back steps rather than those it drops to while the host
sets a phase up, then the warm-up steps.

The line reports:
- keys scored per second (B * Hq * T * layers per step);
- the roofline of the decode kernel: algorithmic bytes per launch over its
  mean time from HIP events that the library records on the launch stream
  right before and after that kernel (pot_debug.decode_begin / decode_end),
  with median and best; the whole call (query prep with the append, decode,
  split combine) is reported beside it as call_us / frac_call;
- the same step captured once as a HIP graph and replayed (graph);
- speed-up over the in-repo fp16 and INT8 kernels on the same shape (each
  engine timed as HIP graph replays of a pass over the layers);
- the CPU oracle timed on host cores on a bounded sample, with one thread and
  with all threads.

--sweep prints one JSON line per point instead:
- the 22-layer step for B in {1, 16, 64} x T in {1k, 4k, 16k, 32k}, PoT-4 and
  PoT-M4;
- the single-layer configurations (B = 1, T = 4096 PoT-4; B = 1, T = 32768
  PoT-M1; B = 8, T = 32768 Hadamard + PoT-M4 with the fp16 and INT8
  comparators on the same seeds).
--sweep-point B,T,k (repeatable) and --sweep-layers N restrict the sweep to
those 22-layer points and change their layer count (one point per process for
counter runs).

--cpu-configs times only the CPU oracle, on the four single-layer
configurations in full (every key encoded, every query head attended), on one
thread and on every host thread; no GPU use.
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
G = HQ // HKV
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak
LLC_BYTES = 256 << 20  # last-level (MALL) cache
COMPARE_ROUNDS = 3  # interleaved timing rounds per comparator engine
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "decode_pot4_b64_t32768_traffic.txt")
PROFILE_READ_CEILING = os.path.join(ROOT, "profiles", "stream_read_ceiling.md")
PROFILE_VALU = os.path.join(ROOT, "profiles", "decode_valu_counters.txt")
# wave64 VALU instructions per ns per CU that shifts, v_perm, v_dot2 / v_dot4,
# packed 16-bit ops and SGPR-operand forms issue at (profiles/valu_issue_rates.md):
# the issue term of the roofline for the score cores
ISSUE_RATE = 2.2
N_CU = 256
CSRC = os.path.join(ROOT, "paper_2609_09208_amd", "csrc")
METRIC = "decode-attention keys scored/s and achieved HBM GB/s at T=32k (PoT-4)"


def row_bytes(mant_bits: int) -> int:
    """Algorithmic HBM bytes per cache row: codes + fp32 scale + fp16 V."""
    return 32 + 8 * mant_bits + 4 + 2 * D


def row_bytes_v8(mant_bits: int) -> int:
    """The same with INT8 values: 64 value bytes + 1 exponent byte."""
    return 32 + 8 * mant_bits + 4 + D + 1


def algorithmic_bytes(B: int, T: int, per_row: int) -> int:
    return B * HKV * T * per_row + B * HQ * D * 4 * 2  # + q in, O out


def source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def read_profile(path):
    """key: value lines of a committed counter summary, if its counters were
    taken on the current kernel sources; otherwise None."""
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_digest") != source_digest():
        return None
    return vals


def read_traffic():
    """HBM bytes per launch measured with rocprofv3 counters, if they were
    taken on the current kernel sources; otherwise None."""
    vals = read_profile(PROFILE_TRAFFIC)
    if vals is None:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def lane_ops_per_key(engine: str, mant_bits: int):
    """VALU lane-ops per cache row of a decode kernel (SQ_INSTS_VALU * 64 /
    rows, rocprofv3 counters on the current sources), or None."""
    vals = read_profile(PROFILE_VALU)
    try:
        return float(vals[f"lane_ops_per_key.{engine}.k{mant_bits}"]) if vals else None
    except (KeyError, ValueError):
        return None


def issue_term(lane_ops, rows: int, us: float):
    """The VALU issue term of the roofline (Sec. III, eq. roofline) for one
    launch: wave64 instructions / (ISSUE_RATE * N_CU) against the measured
    kernel time."""
    if lane_ops is None:
        return None
    wave_instr = lane_ops * rows / 64.0
    floor_us = wave_instr / (ISSUE_RATE * N_CU) / 1e3
    return {"lane_ops_per_key": lane_ops, "wave_instr_per_launch": wave_instr,
            "issue_floor_us": floor_us, "achieved_rate": wave_instr / (us * 1e3) / N_CU,
            "peak_rate": ISSUE_RATE, "rate_unit": "wave64 VALU instr/ns/CU",
            "frac": floor_us / us,
            "source": "SQ_INSTS_VALU from profiles/decode_valu_counters.txt; issue rate of "
                      "the shift / dot / SGPR-operand class from profiles/valu_issue_rates.md"}


def read_ceiling():
    """Best measured stream-read bandwidth (GB/s) of this device model, from the
    committed probe summary; None if absent."""
    try:
        for line in open(PROFILE_READ_CEILING):
            if line.startswith("read_ceiling_gbs:"):
                return float(line.split(":", 1)[1])
    except (OSError, ValueError):
        pass
    return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_threads() -> int:
    """Host threads the oracle may use: every CPU this process may run on,
    capped by the host's per-job share when the environment sets one
    (OMP_NUM_THREADS; a one-GPU job's share of a shared host)."""
    n = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    share = os.environ.get("OMP_NUM_THREADS")
    if share and share.isdigit() and int(share) > 0:
        n = min(n, int(share))
    return max(1, n)


def host_info() -> dict:
    return {"cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity")
            else None, "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def cpu_baseline(T: int, budget_s: float) -> dict:
    """The oracle (plain C) on (batch, kv-head) slices of the same workload:
    append-encode one key row, then decode attention of the G = 8 query heads
    over T PoT-4 keys. Half the budget runs one thread, half runs one slice per
    thread on every available host thread (the oracle holds no shared state and
    its ctypes calls release the interpreter lock)."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    from workloads import make_decode_inputs

    d = make_decode_inputs(1234, B=1, Hq=G, Hkv=1, T=T)
    rows = d["k_bits"].reshape(-1, D)
    se, cm, sc = oracle.encode_keys(rows)
    zeros = np.zeros(G, np.int32)

    def one_slice(_=None):
        oracle.encode_keys(rows[-1:])
        oracle.pot_decode(d["q"], se, cm, sc, d["v_bits"], T, zeros, 1, G, 1, T)

    def run(threads: int, budget: float):
        n, t0 = 0, time.perf_counter()
        with ThreadPoolExecutor(max_workers=threads) as ex:
            while True:
                list(ex.map(one_slice, range(threads)))
                n += threads
                el = time.perf_counter() - t0
                if el >= budget:
                    return n, el

    n1, e1 = run(1, budget_s / 2)
    threads = host_threads()
    nt, et = run(threads, budget_s / 2)
    info = host_info()
    return {"value": nt * G * T / et, "unit": "keys/s", "cores": threads, "kind": "oracle",
            "value_1thread": n1 * G * T / e1, **info,
            "sample": f"(batch, kv-head) slices of T={T}: 1 appended key + {G} query heads over "
                      f"{T} PoT-4 keys; {n1} slices in {e1:.1f} s on 1 thread, {nt} slices in "
                      f"{et:.1f} s on {threads} threads; host CPU {info['cpu_model']}, "
                      f"{info['nproc']} logical CPUs, {info['affinity_cpus']} available"}


# The four single-layer configurations (name, B, T, mant_bits, hadamard,
# query heads; one head means one kv head and no channel scale): tiny single head, TinyLlama layer at T=4096 (PoT-4), at
# T=32768 (PoT-M1), and B=8 T=32768 with Hadamard + PoT-M4.
CPU_CONFIGS = [("C1 tiny single head", 1, 256, 0, False, 1),
               ("C2 TinyLlama layer", 1, 4096, 0, False, HQ),
               ("C3 TinyLlama layer, PoT-M1", 1, 32768, 1, False, HQ),
               ("C4 B=8, Hadamard + PoT-M4", 8, 32768, 4, True, HQ)]


def cpu_configs() -> None:
    """The oracle timed on each single-layer configuration in full: encode
    every key row and run decode attention for every (batch, query head),
    once on one thread and once split over (batch, kv head) units on every
    host thread. One JSON line per configuration."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle
    from workloads import make_decode_inputs

    threads = host_threads()
    info = host_info()
    for name, B, T, k, had, hq in CPU_CONFIGS:
        hkv = 1 if hq == 1 else HKV
        g = hq // hkv
        d = make_decode_inputs(7, B=B, Hq=hq, Hkv=hkv, T=T, channel_scale=hq > 1)
        units = [(b, h) for b in range(B) for h in range(hkv)]

        def unit(bh):
            b, h = bh
            rows = d["k_bits"][b, h]
            se, cm, sc = oracle.encode_keys(rows, mant_bits=k, hadamard=had)
            oracle.pot_decode(d["q"][b, h * g:(h + 1) * g][None], se, cm, sc, d["v_bits"][b, h],
                              d["t_cap"], np.zeros(g, np.int32), 1, g, 1, T, mant_bits=k,
                              hadamard=had)

        t0 = time.perf_counter()
        for u in units:
            unit(u)
        t1 = time.perf_counter() - t0
        t0 = time.perf_counter()
        with ThreadPoolExecutor(max_workers=threads) as ex:
            list(ex.map(unit, units))
        tn = time.perf_counter() - t0
        keys = B * hq * T
        print(json.dumps({"config": name, "B": B, "T": T, "Hq": hq, "Hkv": hkv,
                          "mant_bits": k, "hadamard": had, "kind": "oracle",
                          "seconds_1thread": t1, "seconds_all_threads": tn,
                          "threads": threads, "units": len(units),
                          "keys_scored_per_s_1thread": keys / t1,
                          "keys_scored_per_s_all_threads": keys / tn,
                          "rows_per_s_all_threads": B * hkv * T / tn,
                          "work": "encode every key row, then decode attention of every "
                                  "(batch, query head)", **info}), flush=True)


class Layers:
    """Per-layer PoT caches (codes, scales, interleaved V) plus the appended
    token of each layer, all resident on the device. With distinct=False the
    layers hold copies of one drawn K/V (separate buffers, fresh queries)."""

    def __init__(self, pa, B, T, L, mant_bits, hadamard, dev, distinct=True, keep_k16=0):
        import numpy as np
        import torch

        from workloads import make_decode_inputs_device
        self.pa, self.B, self.T, self.L, self.k = pa, B, T, L, mant_bits
        self.fmt = pa.make_format(mant_bits=mant_bits, frac_bits=7, hadamard=hadamard)
        self.layers = []
        shared = None
        for layer in range(L):
            if distinct or shared is None:
                d = make_decode_inputs_device(1000 + layer, B, HQ, HKV, T, dev)
                if not distinct:
                    shared = d
            else:
                d = dict(shared, q=torch.randn((B, HQ, D), device=dev))
            cache = pa.alloc_pot_cache(B, HKV, T, mant_bits, dev)
            pa.pot_encode_keys(self.fmt, d["k"], B * HKV * T, 1, 0, cache["key_scale"],
                               cache["codes_se"], cache["codes_m"])
            v = pa.alloc_value_cache(B, HKV, T, dev)
            pa.pot_store_values(d["v"], B * HKV, T, T, 0, v)
            rec = dict(q=d["q"], v=v, new_k=d["k"][:, :, T - 1].contiguous(),
                       new_v=d["v"][:, :, T - 1].contiguous(), **cache)
            if layer < keep_k16:
                rec["k16"] = d["k"] if distinct else d["k"].clone()
                rec["v16"] = d["v"] if distinct else d["v"].clone()
            self.layers.append(rec)
            del d
        del shared
        self.heads = np.arange(HQ, dtype=np.int32) // G
        self.out = torch.empty((B, HQ, D), dtype=torch.float32, device=dev)
        self.ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, HQ, HKV, T), dev)

    def decode(self, c):
        self.pa.pot_decode_attention(self.fmt, c["q"], c["codes_se"], c["codes_m"],
                                     c["key_scale"], c["v"], self.T, self.heads, self.B, HQ,
                                     HKV, self.T, self.out, self.ws)

    def step(self, events=None, kernel_events=None):
        """events[i]: HIP events recorded around layer i's call; kernel_events[i]:
        pot_debug structs whose decode_begin / decode_end events the library
        records around the decode kernel alone."""
        pa, T, B = self.pa, self.T, self.B
        for i, c in enumerate(self.layers):
            if events is not None:
                events[i][0].record()
            pa.pot_append_decode_attention(self.fmt, c["q"], c["new_k"], c["new_v"],
                                           c["codes_se"], c["codes_m"], c["key_scale"], c["v"],
                                           T, self.heads, B, HQ, HKV, T, self.out, self.ws,
                                           dbg=kernel_events[i] if kernel_events else None)
            if events is not None:
                events[i][1].record()


PREHEAT_S = 0.3  # seconds of steps before the warm-up steps of each timed phase


def collect_garbage():
    """A full collection of Python's cyclic garbage, before a phase's untimed
    steps (so that the idle gap it leaves falls before them, not between them
    and the timed region)."""
    import gc
    gc.collect()


class no_gc:
    """Python's cyclic garbage collector off inside a timed region (as timeit
    does): a full collection over the host objects of a run can stall the
    launch thread for tens of ms while the GPU idles."""

    def __enter__(self):
        import gc
        gc.disable()

    def __exit__(self, *exc):
        import gc
        gc.enable()


def preheat(lay, seconds=PREHEAT_S):
    """Runs whole steps for about `seconds` and waits for them: the GPU leaves
    the clock state it drops to while the host prepares a phase (after an
    idle gap of tens of ms the first ~40 decode calls run 10-20% slower than
    the steady state of back-to-back steps)."""
    import torch
    collect_garbage()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        lay.step()
        torch.cuda.synchronize()


def time_plain(lay, steps, warmup):
    """Wall time of `steps` steps with only the library's calls in the timed
    region (no timing events: each event record costs the step time on the
    device, about 5% for the four per layer of the instrumented pass)."""
    import torch
    preheat(lay)
    for _ in range(warmup):
        lay.step()
    torch.cuda.synchronize()
    with no_gc():
        t0 = time.perf_counter()
        for _ in range(steps):
            lay.step()
        torch.cuda.synchronize()
        return time.perf_counter() - t0


def time_steps(lay, steps, warmup, kernel_times=False):
    """Wall time of `steps` steps and the per-call decode times (us) from HIP
    events recorded on the launch stream around each call (query prep with
    the append, decode kernel, split combine). With kernel_times, also the
    decode kernel's own times (us), from events the library records on the
    same stream right before and after that kernel."""
    import numpy as np
    import torch
    for _ in range(warmup):
        lay.step()
    torch.cuda.synchronize()
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(lay.L)] for _ in range(steps)]
    kev = kdbg = None
    if kernel_times:
        kev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(lay.L)] for _ in range(steps)]
        kdbg = []
        for row in kev:
            dl = []
            for a, b in row:
                a.record()  # creates the HIP events behind the handles
                b.record()
                d = lay.pa.pot_debug()
                d.decode_begin, d.decode_end = a.cuda_event, b.cuda_event
                dl.append(d)
            kdbg.append(dl)
        torch.cuda.synchronize()
    preheat(lay)
    with no_gc():
        t0 = time.perf_counter()
        for s in range(steps):
            lay.step(ev[s], kdbg[s] if kdbg else None)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    us = np.array([a.elapsed_time(b) for row in ev for (a, b) in row]) * 1e3
    if not kernel_times:
        return elapsed, us
    kus = np.array([a.elapsed_time(b) for row in kev for (a, b) in row]) * 1e3
    return elapsed, us, kus


def time_graph(lay, steps, warmup):
    """Milliseconds per step when the whole step (every layer's call) is
    captured once as a HIP graph and replayed: the launch gaps between the
    kernels shrink, the kernels are the same. Events around all replays."""
    import torch
    collect_garbage()
    lay.step()  # eager first: the library caches its occupancy queries
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lay.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < PREHEAT_S:  # the clocks, as in preheat()
        g.replay()
        torch.cuda.synchronize()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with no_gc():
        s.record()
        for _ in range(steps):
            g.replay()
        e.record()
        torch.cuda.synchronize()
    del g
    return s.elapsed_time(e) / steps


def timed_calls(fn, n_layers, reps=10, warm=2, graph=False):
    """Mean microseconds per call of fn(layer) over reps passes of n_layers
    (no garbage collection before it: the comparators' timed regions follow
    each other back to back, and an idle gap would lower the next engine's
    clocks). graph: one pass over the layers is captured as a HIP graph and
    the timed passes replay it, so the figure is the device's time per call
    even where a call takes less than its Python and ctypes launch path on
    the host (the small single-layer configurations)."""
    import torch
    for _ in range(warm):
        for i in range(n_layers):
            fn(i)
    torch.cuda.synchronize()
    g = None
    if graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(n_layers):
                fn(i)
        for _ in range(warm):
            g.replay()
        torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with no_gc():
        s.record()
        for _ in range(reps):
            if g is not None:
                g.replay()
            else:
                for i in range(n_layers):
                    fn(i)
        e.record()
        torch.cuda.synchronize()
    del g
    return s.elapsed_time(e) / (reps * n_layers) * 1e3


def bulk_encode(pa, lay, dev):
    """The prefill-side bulk key encoder (pot_encode_keys, row scales from the
    rows) over one layer's whole key cache, B * Hkv * T fp16 rows, rotating
    over the layers kept with their fp16 keys."""
    import torch
    cl = [c for c in lay.layers if "k16" in c]
    B, T, k = lay.B, lay.T, lay.k
    n = B * HKV * T
    out = pa.alloc_pot_cache(B, HKV, T, k, dev)
    us = timed_calls(lambda i: pa.pot_encode_keys(lay.fmt, cl[i]["k16"], n, 1, 0,
                                                  out["key_scale"], out["codes_se"],
                                                  out["codes_m"]), len(cl), reps=10, warm=2)
    # bit-identical to the cache encoded when the layer was built
    same = bool(torch.equal(out["codes_se"], cl[-1]["codes_se"]) and
                torch.equal(out["key_scale"], cl[-1]["key_scale"]))
    per_row = 2 * D + D // 2 + 4 + 8 * k  # fp16 row in; codes, planes, scale out
    gbs = n * per_row / (us * 1e-6) / 1e9
    return {"rows": n, "us_per_call": us, "alg_bytes_per_row": per_row, "achieved_gbs": gbs,
            "frac": gbs / HBM_PEAK_GBS, "same_codes_as_cache": same,
            "kernel": f"potattn::encode_pot_kernel<{k}, false>",
            "timing": f"mean of 10 passes over {len(cl)} layers, HIP events around the passes"}


def comparators(pa, lay, dev):
    """fp16 and INT8 kernels and the PoT kernel on the same caches, rotating
    over the layers kept with their fp16 keys."""
    import torch
    cl = [c for c in lay.layers if "k16" in c]
    B, T = lay.B, lay.T
    n8 = B * HKV * T
    i8 = [dict(codes=torch.empty((n8, D), dtype=torch.int8, device=dev),
               sc=torch.empty(n8, dtype=torch.float32, device=dev)) for _ in cl]
    had = int(lay.fmt.hadamard)
    for c, x in zip(cl, i8):
        pa.pot_int8_encode_keys(c["k16"], n8, 1, had, x["sc"], x["codes"])
    # the paper's value cache: INT8 with a power-of-two per-token scale
    v8 = []
    for c in cl:
        vu, ve = pa.alloc_value_cache_int8(B, HKV, T, dev)
        pa.pot_store_values_int8(c["v16"], B * HKV, T, T, 0, vu, ve)
        v8.append((vu, ve))
    out, ws, heads = lay.out, lay.ws, lay.heads
    engines = {
        "pot": lambda i: lay.decode(cl[i]),
        "fp16": lambda i: pa.pot_fp16_decode_attention(
            cl[i]["q"], cl[i]["k16"], cl[i]["v"], T, heads, B, HQ, HKV, T, out, ws),
        "int8": lambda i: pa.pot_int8_decode_attention(
            cl[i]["q"], i8[i]["codes"], i8[i]["sc"], cl[i]["v"], T, heads, B, HQ, HKV, T, had,
            out, ws),
    }
    engines["pot_v8"] = lambda i: pa.pot_decode_attention_v8(
        lay.fmt, 0, cl[i]["q"], cl[i]["codes_se"], cl[i]["codes_m"], cl[i]["key_scale"],
        v8[i][0], v8[i][1], T, heads, B, HQ, HKV, T, out, ws)
    engines["pot_v8_pow2"] = lambda i: pa.pot_decode_attention_v8_pow2(
        lay.fmt, 0, cl[i]["q"], cl[i]["codes_se"], cl[i]["codes_m"], cl[i]["key_scale"],
        v8[i][0], v8[i][1], T, heads, B, HQ, HKV, T, out, ws)
    if lay.k > 0:  # PoT-Mk decoded to 16-bit weights + v_dot2 (a multiply path)
        engines["dot"] = lambda i: pa.pot_dot_decode_attention(
            lay.fmt, cl[i]["q"], cl[i]["codes_se"], cl[i]["codes_m"], cl[i]["key_scale"],
            cl[i]["v"], T, heads, B, HQ, HKV, T, out, ws)
    if lay.k == 0:  # byte decode + v_dot4 on the same PoT-4 caches (a multiply path)
        engines["ds4a"] = lambda i: pa.pot_ds4a_decode_attention(
            lay.fmt, cl[i]["q"], cl[i]["codes_se"], cl[i]["key_scale"], cl[i]["v"], T, heads,
            B, HQ, HKV, T, out, ws)
        engines["ds4a_v8"] = lambda i: pa.pot_decode_attention_v8(
            lay.fmt, 1, cl[i]["q"], cl[i]["codes_se"], None, cl[i]["key_scale"], v8[i][0],
            v8[i][1], T, heads, B, HQ, HKV, T, out, ws)
    # interleaved rounds, each engine warmed before it is timed; median per engine
    runs = {name: [] for name in engines}
    for _ in range(COMPARE_ROUNDS):
        for name, fn in engines.items():
            runs[name].append(timed_calls(fn, len(cl), reps=10, warm=4, graph=True))
    med = {name: float(sorted(v)[len(v) // 2]) for name, v in runs.items()}
    pot_us, f16_us, i8_us, ds4a_us = med["pot"], med["fp16"], med["int8"], med.get("ds4a")
    pv8_us, dv8_us, pw_us = med["pot_v8"], med.get("ds4a_v8"), med["pot_v8_pow2"]
    dot_us = med.get("dot")

    def frac(per_row, us):
        return algorithmic_bytes(B, T, per_row) / (us * 1e-6) / 1e9 / HBM_PEAK_GBS

    return {"pot_us_per_layer": pot_us, "fp16_us_per_layer": f16_us, "int8_us_per_layer": i8_us,
            "speedup_vs_fp16": f16_us / pot_us, "speedup_vs_int8": i8_us / pot_us,
            "pot_hbm_frac": frac(row_bytes(lay.k), pot_us), "fp16_hbm_frac": frac(256, f16_us),
            "int8_hbm_frac": frac(196, i8_us), "layers_rotated": len(cl),
            "ds4a_us_per_layer": ds4a_us,
            "ds4a_hbm_frac": frac(row_bytes(0), ds4a_us) if ds4a_us else None,
            "ds4a_speedup_vs_fp16": f16_us / ds4a_us if ds4a_us else None,
            "ds4a_note": "PoT-4 codes decoded to int8 bytes by v_perm and scored by v_dot4 "
                         "(software packed shift-dot, a multiply path)",
            "dot_us_per_layer": dot_us,
            "dot_hbm_frac": frac(row_bytes(lay.k), dot_us) if dot_us else None,
            "dot_speedup_vs_fp16": f16_us / dot_us if dot_us else None,
            "dot_speedup_vs_sac": pot_us / dot_us if dot_us else None,
            "dot_note": "PoT-Mk codes decoded to 16-bit weights sigma (2^k + j) 2^(7-e) and "
                        "scored by v_dot2 (pot_dot_decode_attention, a multiply path)",
            "int8_values": {
                "bytes_per_row": row_bytes_v8(lay.k),
                "pot_us_per_layer": pv8_us,
                "pot_hbm_frac": frac(row_bytes_v8(lay.k), pv8_us),
                "pot_speedup_vs_fp16": f16_us / pv8_us,
                "ds4a_us_per_layer": dv8_us,
                "ds4a_hbm_frac": frac(row_bytes_v8(0), dv8_us) if dv8_us else None,
                "ds4a_speedup_vs_fp16": f16_us / dv8_us if dv8_us else None,
                "pot_pow2_weights_us_per_layer": pw_us,
                "note": "INT8 values with a power-of-two per-token scale (pot_store_values_int8); "
                        "pow2 weights: both products by powers of two "
                        "(pot_decode_attention_v8_pow2)"},
            "timing": f"median of {COMPARE_ROUNDS} interleaved rounds of 10 passes over the "
                      f"{len(cl)} layers per engine, each pass one HIP graph replay (device "
                      "time per call, free of the host's launch path)"}


def fmt_name(k: int, had: bool) -> str:
    return ("Hadamard + " if had else "") + ("PoT-4" if k == 0 else f"PoT-M{k}")


def sweep(pa, dev, steps, warmup, only=None, layers=None, compare_only=False):
    """only: keep the points whose (B, T, k) is in this set; layers: layer
    count override (the counter runs profile one point per process);
    compare_only: only the configurations timed with the comparators."""
    import numpy as np
    import torch
    pts = []
    for B in (1, 16, 64):
        for T in (1024, 4096, 16384, 32768):
            for k in (0, 4):
                pts.append(dict(B=B, T=T, k=k, had=False, L=22, compare=False))
    # the single-layer configurations with the comparators, over 22 layers
    # that all keep their fp16 keys (every engine streams the same layers)
    pts += [dict(B=1, T=4096, k=0, had=False, L=22, compare=True),
            dict(B=1, T=32768, k=1, had=False, L=22, compare=True),
            dict(B=8, T=32768, k=4, had=True, L=22, compare=True),
            dict(B=8, T=32768, k=0, had=False, L=22, compare=True)]
    if only is not None:
        pts = [p for p in pts if (p["B"], p["T"], p["k"]) in only and not p["compare"]]
    if compare_only:
        pts = [p for p in pts if p["compare"]]
    for p in pts:
        if layers is not None:
            p["L"] = layers
        lay = Layers(pa, p["B"], p["T"], p["L"], p["k"], p["had"], dev, distinct=False,
                     keep_k16=p["L"] if p["compare"] else 0)
        elapsed, us = time_steps(lay, steps, warmup)
        graph_ms = time_graph(lay, steps, warmup)
        alg = algorithmic_bytes(p["B"], p["T"], row_bytes(p["k"]))
        foot = p["L"] * alg
        rec = {"B": p["B"], "T": p["T"], "format": fmt_name(p["k"], p["had"]), "layers": p["L"],
               "keys_per_s_step": p["B"] * HQ * p["T"] * p["L"] * steps / elapsed,
               "ms_per_step": elapsed / steps * 1e3, "graph_ms_per_step": graph_ms,
               "decode_us_mean": float(us.mean()), "decode_us_median": float(np.median(us)),
               "decode_us_best": float(us.min()),
               "hbm_frac_mean": alg / (us.mean() * 1e-6) / 1e9 / HBM_PEAK_GBS,
               "step_footprint_bytes": foot, "cache_resident": foot < LLC_BYTES}
        if p["compare"]:
            rec["comparators"] = comparators(pa, lay, dev)
        print(json.dumps(rec), flush=True)
        del lay
        torch.cuda.empty_cache()


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
    ap.add_argument("--sweep", action="store_true",
                    help="one JSON line per workload point instead of the headline line")
    ap.add_argument("--sweep-point", action="append", default=None, metavar="B,T,k",
                    help="with --sweep: run only this 22-layer point (repeatable)")
    ap.add_argument("--sweep-compare", action="store_true",
                    help="with --sweep: only the configurations timed with the comparators")
    ap.add_argument("--sweep-layers", type=int, default=None,
                    help="with --sweep: layers per point instead of 22")
    ap.add_argument("--cpu-configs", action="store_true",
                    help="only time the CPU oracle on the four single-layer configurations "
                         "in full (one thread and all host threads); no GPU use")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run device-to-device copies of BYTES bytes (calibrates "
                         "the FETCH_SIZE / WRITE_SIZE counters against a known size)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU; --gpus {args.gpus} is not supported "
              "(the decode path shards over (batch, kv head) with no communication)",
              file=sys.stderr)
        return 2

    if args.cpu_configs:
        cpu_configs()
        return 0

    import numpy as np
    import torch

    import paper_2609_09208_amd as pa

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
    if args.sweep:
        only = None
        if args.sweep_point:
            only = {tuple(int(v) for v in sp.split(",")) for sp in args.sweep_point}
        sweep(pa, dev, max(2, min(args.steps, 5)), max(1, min(args.warmup, 2)), only,
              args.sweep_layers, args.sweep_compare)
        return 0

    B, T, L, k = args.batch, args.seq, args.layers, args.mant_bits
    lay = Layers(pa, B, T, L, k, False, dev, distinct=True,
                 keep_k16=0 if args.no_compare else 4)
    torch.cuda.synchronize()
    # value: K steps with nothing else in the timed region; then K more steps
    # with HIP events around every call and every decode kernel (roofline)
    elapsed = time_plain(lay, args.steps, args.warmup)
    elapsed_ev, us, kus = time_steps(lay, args.steps, 1, kernel_times=True)
    kern_s = float(kus.mean()) * 1e-6
    call_s = float(us.mean()) * 1e-6
    alg = algorithmic_bytes(B, T, row_bytes(k))
    achieved = alg / kern_s / 1e9

    roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                "traffic": read_traffic() if (B, T, k) == (64, 32768, 0) else None,
                "kernel": f"potattn::decode_kernel<0, 8, {k}, false, 0> (SAC, G = 8, fp16 V: "
                          "products by packed 16-bit shifts, signs and int32 sums by "
                          "v_dot2_i32_i16 with weights -1/0/+1"
                          + (", one sum per mantissa bit plane" if k else "") + ")",
                "note": "score cores built from shifts and adds alone (v_lshl_add_u32, "
                        "SDWA shift + v_xad_u32) measured 0.57-0.60 of 8 TB/s in this "
                        "kernel; the v_dot2 accumulate is the one timed here",
                "alg_bytes_per_launch": alg, "launch_us": kern_s * 1e6,
                "launch_us_median": float(np.median(kus)), "launch_us_best": float(kus.min()),
                "launches_timed": int(kus.size),
                "call_us": call_s * 1e6, "call_us_median": float(np.median(us)),
                "frac_call": alg / call_s / 1e9 / HBM_PEAK_GBS,
                "read_ceiling_gbs": read_ceiling(),
                "frac_of_read_ceiling": achieved / read_ceiling() if read_ceiling() else None,
                "keys_scored_per_s_kernel": B * HQ * T / kern_s,
                "keys_scored_per_s_call": B * HQ * T / call_s}
    issue = issue_term(lane_ops_per_key("sac", k), B * HKV * T, kern_s * 1e6)
    roofline["issue"] = issue
    if k > 0 and issue is not None:
        # PoT-Mk's shift-accumulate core is bound by VALU issue (eq. roofline's
        # second term): the headline fraction is the issue one, HBM beside it
        hbm = {key: roofline.pop(key) for key in ("achieved", "peak", "unit", "frac", "traffic")}
        roofline.pop("bound")
        roofline = {"bound": "valu", "achieved": issue["achieved_rate"], "peak": ISSUE_RATE,
                    "unit": issue["rate_unit"], "frac": issue["frac"], "traffic": None,
                    "hbm": hbm, **roofline}
    result = {
        "metric": METRIC,
        "value": B * HQ * T * L * args.steps / elapsed, "unit": "keys/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int32+fp32", "data": "synthetic",
        "config": {"workload": f"TinyLlama-1.1B-shaped {L}-layer decode step, "
                               f"{fmt_name(k, False)} keys (append + attend), "
                               f"fp16 V, B={B}, T={T}, Hq={HQ}, Hkv={HKV}, d={D}",
                   "B": B, "T": T, "layers": L, "Hq": HQ, "Hkv": HKV, "head_dim": D,
                   "mant_bits": k, "frac_bits": 7, "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "timing": {"value": f"{args.steps} steps after {PREHEAT_S} s of steps and "
                            f"{args.warmup} warm-up steps, no events in the timed region",
                   "roofline": f"{args.steps} further steps with HIP events around every "
                               f"call and every decode kernel, after {PREHEAT_S} s of steps",
                   "ms_per_step_with_events": elapsed_ev / args.steps * 1e3},
    }
    graph_ms = time_graph(lay, args.steps, args.warmup)
    result["graph"] = {"ms_per_step": graph_ms,
                       "keys_per_s": B * HQ * T * L / (graph_ms * 1e-3),
                       "note": "the same step captured once as a HIP graph and replayed"}
    if not args.no_compare:
        result["comparators"] = comparators(pa, lay, dev)
        result["bulk_encode"] = bulk_encode(pa, lay, dev)
    if args.cpu_budget > 0:
        result["cpu_baseline"] = cpu_baseline(T, args.cpu_budget)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
