"""GPU parity of sfda_chunk_fwd_decoupled (the write-decoupled variant of Sec. 3) against
the oracle's complex128 recurrence (oracle.decoupled), on the same stored inputs.

Bars as for sfda_chunk_fwd: max |x - ref| / max |ref| <= 1e-4 (float32 inputs), <= 2e-2
(bfloat16 inputs), on o and on S_T.  Cases cover ragged sequences, m < 64, n = 3, 24, 80
(several column slices), both chunk lengths, the zero state, the tied special case (r = k,
eta = beta must give sfda_chunk_fwd's result) and the benchmarked batch, heads and length
at full size with C = 32 on sampled heads.
"""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import I, ensure_built, rel_err, to_complex, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return ensure_built()


def say(*a):
    print("[case]", *a, flush=True)


def run_dec(x, C, S0=True):
    import torch
    from paper_2607_11897_amd import sfda
    st = x.storage()
    d = {k: to_device(st[k], x.dtype) for k in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")}
    s0 = to_device(st["S0"], "f32") if (S0 and st["S0"] is not None) else None
    o, S = sfda.chunk_fwd_decoupled(d["q"], d["k"], d["r"], d["v"], d["alpha"], d["theta"], d["eta"],
                                    d["beta"], s0, C=C)
    torch.cuda.synchronize()
    return to_complex(o), to_complex(S)


def oracle_dec(x, S0=True):
    from oracle import decoupled as D
    return D.decoupled_recurrence(x.q, x.k, x.r, x.v, x.alpha, x.theta, x.eta, x.beta,
                                  x.S0 if S0 else None)


@pytest.mark.parametrize("dtype,B,H,T,m,n,C", [
    ("f32", 1, 2, 100, 64, 64, 16),
    ("f32", 2, 1, 70, 33, 24, 32),
    ("f32", 1, 2, 130, 64, 80, 32),
    ("f32", 1, 1, 50, 5, 3, 16),
    ("bf16", 1, 2, 300, 64, 64, 32),
    ("bf16", 2, 1, 97, 33, 24, 16),
])
def test_decoupled_matches_oracle(dtype, B, H, T, m, n, C):
    x = I.make_decoupled_inputs(B, H, T, m, n, dtype, seed=600 + T)
    say(dtype, (B, H, T, m, n), "C", C)
    o, S = run_dec(x, C)
    o_ref, S_ref = oracle_dec(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say("err(o)", eo, "err(S_T)", es)
    tol = 1e-4 if dtype == "f32" else 2e-2
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))
    assert eo <= tol and es <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decoupled_strong_decay(dtype):
    """alpha ~ U(0.02, 0.1): a 64-token chunk decays to 1e-109, each 16-token chunk stays
    inside the float range."""
    laws = I.Laws(alpha=("uniform", 0.02, 0.1), theta=("uniform", -3.14159, 3.14159),
                  beta=("uniform", 0.0, 1.0), s0_scale=0.1)
    x = I.make_decoupled_inputs(1, 2, 3 * 64 + 37, 64, 64, dtype, seed=41, laws=laws)
    say(dtype, "decoupled strong decay")
    o, S = run_dec(x, 64)
    o_ref, S_ref = oracle_dec(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say("err(o)", eo, "err(S_T)", es)
    tol = 1e-4 if dtype == "f32" else 2e-2
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))
    assert eo <= tol and es <= tol


def test_decoupled_zero_state():
    x = I.make_decoupled_inputs(1, 2, 96, 64, 64, "f32", seed=7)
    o, S = run_dec(x, 32, S0=False)
    o_ref, S_ref = oracle_dec(x, S0=False)
    assert rel_err(o, o_ref) <= 1e-4 and rel_err(S, S_ref) <= 1e-4


def test_decoupled_tied_case_equals_chunk_fwd():
    import torch
    from paper_2607_11897_amd import sfda
    x = I.make_decoupled_inputs(1, 2, 96, 64, 64, "f32", seed=8)
    st = x.storage()
    d = {k: to_device(st[k], "f32") for k in ("q", "k", "v", "alpha", "theta", "beta")}
    s0 = to_device(st["S0"], "f32")
    o1, S1 = sfda.chunk_fwd_decoupled(d["q"], d["k"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"],
                                      d["beta"], s0, C=32)
    o2, S2 = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], s0, C=32)
    torch.cuda.synchronize()
    eo, es = rel_err(to_complex(o1), to_complex(o2)), rel_err(to_complex(S1), to_complex(S2))
    say("tied vs sfda_chunk_fwd", eo, es)
    assert eo <= 1e-5 and es <= 1e-5


def test_decoupled_chunk_lengths():
    """Every C runs 16-token chunks (same bits as C = 16); other lengths are refused."""
    import torch
    from paper_2607_11897_amd import sfda
    x = I.make_decoupled_inputs(1, 2, 100, 16, 8, "f32", seed=1)
    say("decoupled chunk lengths")
    o16, S16 = run_dec(x, 16)
    for C in (32, 64, 128):
        o, S = run_dec(x, C)
        assert np.array_equal(o, o16) and np.array_equal(S, S16), C
    st = x.storage()
    d = {k: to_device(st[k], "f32") for k in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")}
    with pytest.raises(sfda.SfdaError):
        sfda.chunk_fwd_decoupled(d["q"], d["k"], d["r"], d["v"], d["alpha"], d["theta"], d["eta"], d["beta"],
                                 None, C=48)
    torch.cuda.synchronize()


def test_decoupled_bf16_b8h16_t4k_full_sampled_heads():
    """The benchmarked batch, heads and length (bf16) with C = 64, as bench.py --mode dec runs
    it, in one call; four heads against the oracle."""
    x = I.make_decoupled_inputs(8, 16, 4096, 64, 64, "bf16", seed=3003)
    say("decoupled bf16 b8h16 t4k: running")
    o, S = run_dec(x, 64)
    for (b, h) in [(0, 0), (2, 7), (5, 11), (7, 15)]:
        o_ref, S_ref = oracle_dec(x.head(b, h))
        eo, es = rel_err(o[b, h], o_ref[0, 0]), rel_err(S[b, h], S_ref[0, 0])
        say((b, h), "err(o)", eo, "err(S_T)", es)
        assert eo <= 2e-2 and es <= 2e-2
