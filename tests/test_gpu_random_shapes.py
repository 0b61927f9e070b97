"""GPU parity over seeded random shapes and formats.

Each case draws a batch size, group size, kv-head count, key count T (ragged,
with spare cache rows up to t_cap), mantissa width k, Hadamard rotation,
head-room F, score engine and split count, and runs the full parity check
against the oracle: codes, scales, q^, Delta, int32 scores and integer maxima
bit-exact, O within 2e-3. The cases are fixed by their seeds, so the test is
deterministic; together they cover combinations that the hand-written cases
do not. A second set draws the same shapes over the INT8 value cache, with
softmax or power-of-two weights and either score engine, a third the fused
append of the new token, and a fourth the decoded-code entry point
(pot_dot_decode_attention) at every mantissa width.
"""
import numpy as np
import pytest

from parity_util import assert_pot_parity
from workloads import make_decode_inputs

pytestmark = pytest.mark.gpu


def _case(seed):
    rng = np.random.default_rng(9000 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.choice([1, 2, 4]))
    B = int(rng.integers(1, 4))
    T = int(rng.integers(1, 3000))
    t_cap = (T + 7) // 8 * 8 + 8 * int(rng.integers(0, 4))
    engine = "ds4a" if rng.random() < 0.25 else "sac"
    k = 0 if engine == "ds4a" else int(rng.integers(0, 5))
    hadamard = bool(rng.random() < 0.3)
    F = 7 if engine == "ds4a" else int(rng.choice([6, 7, 9, 12]))
    tiles = -(-T // 256)
    splits = 0 if rng.random() < 0.5 else int(rng.integers(1, tiles + 1))
    return dict(G=G, Hkv=Hkv, B=B, T=T, t_cap=t_cap, engine=engine, k=k, hadamard=hadamard,
                F=F, splits=splits)


@pytest.mark.parametrize("seed", range(24))
def test_random_shape(seed):
    c = _case(seed)
    d = make_decode_inputs(7000 + seed, B=c["B"], Hq=c["G"] * c["Hkv"], Hkv=c["Hkv"],
                           T=c["T"], t_cap=c["t_cap"])
    err, g = assert_pot_parity(d, mant_bits=c["k"], frac_bits=c["F"], hadamard=c["hadamard"],
                               force_splits=c["splits"], engine=c["engine"])
    print(f"seed {seed} {c} splits={g['n_splits']} O err {err:.2e}")


@pytest.mark.parametrize("seed", range(12))
def test_random_shape_dot_engine(seed):
    # the decoded-code entry point over the same kind of draws, every k
    c = _case(100 + seed)
    k = int(np.random.default_rng(9300 + seed).integers(0, 5))
    d = make_decode_inputs(7100 + seed, B=c["B"], Hq=c["G"] * c["Hkv"], Hkv=c["Hkv"],
                           T=c["T"], t_cap=c["t_cap"])
    err, g = assert_pot_parity(d, mant_bits=k, frac_bits=c["F"], hadamard=c["hadamard"],
                               force_splits=c["splits"], engine="dot")
    shape = {key: c[key] for key in ("G", "Hkv", "B", "T", "t_cap", "hadamard", "F", "splits")}
    print(f"seed {seed} {shape} k={k} dot splits={g['n_splits']} O err {err:.2e}")


def _case_v8(seed):
    rng = np.random.default_rng(9500 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.choice([1, 2, 4]))
    B = int(rng.integers(1, 4))
    T = int(rng.integers(1, 3000))
    t_cap = (T + 7) // 8 * 8 + 8 * int(rng.integers(0, 4))
    engine = int(rng.random() < 0.3)
    k = 0 if engine else int(rng.integers(0, 5))
    hadamard = bool(rng.random() < 0.3)
    pow2 = bool(rng.random() < 0.5)
    tiles = -(-T // 256)
    splits = 0 if rng.random() < 0.5 else int(rng.integers(1, tiles + 1))
    return dict(G=G, Hkv=Hkv, B=B, T=T, t_cap=t_cap, engine=engine, k=k, hadamard=hadamard,
                pow2=pow2, splits=splits)


@pytest.mark.parametrize("seed", range(16))
def test_random_shape_int8_values(seed):
    """The INT8 value cache (softmax weights, or power-of-two weights) over the
    same kind of random draws: value codes and exponents, q^, scores and M
    bit-exact, O within 2e-3."""
    from test_gpu_values_int8 import assert_v8_parity
    c = _case_v8(seed)
    d = make_decode_inputs(7500 + seed, B=c["B"], Hq=c["G"] * c["Hkv"], Hkv=c["Hkv"],
                           T=c["T"], t_cap=c["t_cap"])
    err, s = assert_v8_parity(d, engine=c["engine"], mant_bits=c["k"], hadamard=c["hadamard"],
                              force_splits=c["splits"], pow2=c["pow2"])
    print(f"seed {seed} {c} splits={s} O err {err:.2e}")


@pytest.mark.parametrize("seed", range(12))
def test_random_shape_fused_append(seed):
    """The fused append + decode call over random draws: the appended row and
    every output and tap equal those of the three separate calls bit for bit,
    and the oracle's."""
    from test_gpu_append import _run
    rng = np.random.default_rng(9800 + seed)
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.choice([1, 2, 4]))
    B = int(rng.integers(1, 4))
    T = int(rng.integers(1, 3000))
    t_cap = (T + 7) // 8 * 8 + 8 * int(rng.integers(0, 4))
    k = int(rng.integers(0, 5))
    hadamard = bool(rng.random() < 0.3)
    err, s = _run(7800 + seed, B, G * Hkv, Hkv, T, t_cap=t_cap, mant_bits=k, hadamard=hadamard)
    print(f"seed {seed} G={G} Hkv={Hkv} B={B} T={T} t_cap={t_cap} k={k} had={hadamard} "
          f"splits={s} O err {err:.2e}")
