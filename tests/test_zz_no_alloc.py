"""GPU test of pot_decode_attention_noalloc, the entry point for callers that
cannot allocate: two calls in a row (the second with a smaller input, both
with several key splits, so the second combine runs over scratch the first
call left behind) against pot_decode_attention with a caller workspace on the
same inputs. Same kernels, so the outputs and the integer maxima must be
bit-identical; O is also checked against the oracle within 2e-3."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_09208_amd as pa
from parity_util import DEV, O_TOL, oracle_pot, store_values, to_dev
from workloads import make_decode_inputs

pytestmark = pytest.mark.gpu


def _run_both(d, mant_bits, hadamard):
    B, Hq, Hkv, T, t_cap = d["B"], d["Hq"], d["Hkv"], d["T"], d["t_cap"]
    fmt = pa.make_format(mant_bits, 7, hadamard)
    se, cm, sc, r = oracle_pot(d, mant_bits, 7, hadamard)
    q = to_dev(d["q"])
    se_d, sc_d = to_dev(se), to_dev(sc)
    cm_d = to_dev(cm) if mant_bits else None
    v = store_values(d["v_bits"], B, Hkv, t_cap)
    outs, maxima, plans = [], [], []
    for noalloc in (False, True):
        out = torch.full((B, Hq, 64), float("nan"), dtype=torch.float32, device=DEV)
        m_final = torch.full((B, Hq), -7, dtype=torch.int32, device=DEV)
        dbg = pa.pot_debug()
        dbg.m_final = m_final.data_ptr()
        if noalloc:
            pa.pot_decode_attention_noalloc(fmt, q, se_d, cm_d, sc_d, v, t_cap,
                                            d["kv_head_of_q"], B, Hq, Hkv, T, out, dbg=dbg)
        else:
            ws = pa.alloc_workspace(pa.pot_decode_workspace_bytes(B, Hq, Hkv, T), DEV)
            pa.pot_decode_attention(fmt, q, se_d, cm_d, sc_d, v, t_cap, d["kv_head_of_q"],
                                    B, Hq, Hkv, T, out, ws, dbg=dbg)
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
        maxima.append(m_final.cpu().numpy())
        plans.append(dbg.n_splits)
    return outs, maxima, plans, r


def test_noalloc_matches_the_workspace_call_twice():
    cases = [(dict(seed=71, B=4, Hq=32, Hkv=4, T=5000), 1, False),
             (dict(seed=72, B=1, Hq=8, Hkv=2, T=777), 0, True)]   # second: smaller
    for shape, k, had in cases:
        print(f"noalloc case {shape} k={k} had={had}", flush=True)
        seed = shape.pop("seed")
        d = make_decode_inputs(seed, **shape)
        outs, maxima, plans, r = _run_both(d, k, had)
        assert plans[0] == plans[1] and plans[0] > 1, plans
        assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))
        assert np.array_equal(maxima[0], maxima[1])
        assert np.array_equal(maxima[1], r["m_final"])
        err = float(np.abs(outs[1] - r["out"]).max())
        assert err <= O_TOL, err
        print(f"  splits={plans[1]} bit-identical to the workspace call, O err {err:.2e}",
              flush=True)
