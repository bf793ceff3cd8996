"""Irregular sizes through every chunked entry point against the oracle: a fixed, seeded
list of (m, n, T, C, dtype) combinations -- m and n down to 1 and not multiples of 4 or 16,
T of 1 and just past a chunk boundary, n above 64 -- for sfda_chunk_fwd, sfda_chunk_bwd
(every gradient) and sfda_chunk_fwd_decoupled (C <= 32).  Bars as in the per-entry-point
tests: 1e-4 (float32), 2e-2 (bfloat16), max |x - ref| / max |ref| per tensor, for every
tensor of every case.  (At m = 1 the erase is the scalar 1 - beta |k|^2, whose cancellation
would magnify bf16 operand rounding past the bar; bfloat16 inputs with at most four key
channels therefore take float32 matrix-core operands, and the m = 1 cases here check that.)
"""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import I, ensure_built, rel_err, run_oracle, to_complex, to_device, upload

pytestmark = pytest.mark.gpu


def _cases():
    rng = np.random.default_rng(2024)
    ms, ns, Ts, Cs = (1, 3, 7, 32, 41, 64), (1, 2, 5, 13, 16, 24, 72), (1, 2, 15, 17, 33, 64, 65, 130), (16, 32, 64)
    out = []
    for _ in range(24):
        out.append((int(rng.choice(ms)), int(rng.choice(ns)), int(rng.choice(Ts)), int(rng.choice(Cs)),
                    "f32" if rng.random() < 0.6 else "bf16"))
    return out


# bfloat16 either side of the operand switch (at most four key channels: float32 operands)
CASES = _cases() + [(4, 24, 65, 64, "bf16"), (5, 24, 65, 64, "bf16"), (4, 13, 33, 16, "bf16"), (5, 13, 33, 16, "bf16")]


@pytest.fixture(scope="module", autouse=True)
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return ensure_built()


def say(*a):
    print("[case]", *a, flush=True)


def make(m, n, T, dtype, seed):
    w = I.Workload("shape", 1, 2, T, m, n, 16, dtype, I.LAWS_MAIN, seed, 1e-4)
    return I.make_chunk_inputs(w)


@pytest.mark.parametrize("m,n,T,C,dtype", CASES)
def test_forward_and_backward_irregular(m, n, T, C, dtype):
    import torch
    from oracle import backward as BW
    from paper_2607_11897_amd import sfda
    tol = 1e-4 if dtype == "f32" else 2e-2
    x = make(m, n, T, dtype, seed=7000 + 97 * m + 13 * n + T)
    say("shape", (m, n, T), "C", C, dtype)
    d = upload(x)
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=C)
    torch.cuda.synchronize()
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(to_complex(o), o_ref), rel_err(to_complex(S), S_ref)
    dO, dS = I.make_cotangents(1, 2, T, m, n, dtype, seed=8000 + T)
    g = sfda.chunk_bwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"],
                       to_device(I.to_storage(dO, dtype), dtype), to_device(I.to_storage(dS, "f32"), "f32"), C=C)
    torch.cuda.synchronize()
    ref = BW.recurrence_backward(x.q, x.k, x.v, x.alpha, x.theta, x.beta, x.S0, dO, dS)
    eb, over = {}, {}
    for name in ("dq", "dk", "dv", "dS0", "dalpha", "dtheta", "dbeta"):
        got = to_complex(g[name]) if name in ("dq", "dk", "dv", "dS0") else g[name].double().cpu().numpy()
        err = float(np.max(np.abs(got - ref[name])))
        bound = tol * float(np.max(np.abs(ref[name])))
        eb[name] = rel_err(got, ref[name])
        if err > bound:
            over[name] = (err, bound)
    say("err(o)", eo, "err(S_T)", es, {k: f"{v:.1e}" for k, v in eb.items()}, "over", over)
    assert eo <= tol and es <= tol
    assert not over, over


@pytest.mark.parametrize("m,n,T,C,dtype", [c for c in CASES if c[3] <= 32][:10])
def test_decoupled_irregular(m, n, T, C, dtype):
    import torch
    from oracle import decoupled as D
    from paper_2607_11897_amd import sfda
    tol = 1e-4 if dtype == "f32" else 2e-2
    x = I.make_decoupled_inputs(1, 2, T, m, n, dtype, seed=9000 + 31 * m + n + T)
    st = x.storage()
    d = {k: to_device(st[k], dtype) for k in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")}
    o, S = sfda.chunk_fwd_decoupled(d["q"], d["k"], d["r"], d["v"], d["alpha"], d["theta"], d["eta"], d["beta"],
                                    to_device(st["S0"], "f32"), C=C)
    torch.cuda.synchronize()
    o_ref, S_ref = D.decoupled_recurrence(x.q, x.k, x.r, x.v, x.alpha, x.theta, x.eta, x.beta, x.S0)
    eo, es = rel_err(to_complex(o), o_ref), rel_err(to_complex(S), S_ref)
    say("decoupled", (m, n, T), "C", C, dtype, "err(o)", eo, "err(S_T)", es)
    assert eo <= tol and es <= tol
