"""GPU parity of sfda_chunk_fwd_segmented (each head's sequence scanned as G parallel
segments, joined by the affine law of a segment, Thm 4.4, composed along the segments,
Lemma A.2) against the complex128 oracle recurrence, and against sfda_chunk_fwd.

Bars as for sfda_chunk_fwd: max-norm relative error <= 1e-4 for float32 inputs, <= 2e-2
for bfloat16 inputs, on o and on S_T.  The long-context workload runs at full size with
the segments the benchmark uses and is checked on sampled heads over prefix windows.
"""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import I, ensure_built, rel_err, run_oracle, to_complex, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return ensure_built()


def say(*a):
    print("[case]", *a, flush=True)


def run(x, C, G, in_place=False):
    import torch
    from paper_2607_11897_amd import sfda
    d = upload(x)
    S0 = d["S0"]
    S_T = S0 if (in_place and S0 is not None) else None
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], S0, C=C,
                          segments=G, S_T=S_T)
    torch.cuda.synchronize()
    return to_complex(o), to_complex(S)


def run_plain(x, C):
    import torch
    from paper_2607_11897_amd import sfda
    d = upload(x)
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=C,
                          segments=None)
    torch.cuda.synchronize()
    return to_complex(o), to_complex(S)


def make(B, H, T, m, n, C, dtype="f32", zero_state=False, seed=21):
    w = I.Workload("seg", B, H, T, m, n, C, dtype, I.LAWS_MAIN, seed, 1e-4)
    x = I.make_chunk_inputs(w)
    if zero_state:
        x = x.__class__(x.q, x.k, x.v, x.alpha, x.theta, x.beta, None, x.dtype)
    return x


@pytest.mark.parametrize("B,H,T,m,n,C,G", [
    (1, 2, 128, 64, 64, 16, 4),
    (2, 1, 96, 33, 24, 16, 3),
    (1, 3, 256, 64, 80, 32, 2),
    (1, 1, 64, 16, 8, 16, 1),
    (1, 2, 512, 64, 64, 64, 8),
    (3, 1, 192, 5, 3, 64, 3),
])
def test_segmented_f32(B, H, T, m, n, C, G):
    x = make(B, H, T, m, n, C)
    say("f32", (B, H, T, m, n), "C", C, "G", G)
    o, S = run(x, C, G)
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    op, Sp = run_plain(x, C)
    say("err(o)", eo, "err(S_T)", es, "vs plain", rel_err(o, op), rel_err(S, Sp))
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))
    assert eo <= 1e-4 and es <= 1e-4


@pytest.mark.parametrize("m,n,G", [(64, 40, 4), (21, 64, 2)])
def test_segmented_f32_in_bf16_out(m, n, G):
    """float32 inputs, bfloat16 output: the segment scans store o0 in bfloat16 and the join
    adds S_in^* X in float32 before rounding once more; o within the bf16 bar, S_T (float32)
    within 1e-4."""
    import torch
    from paper_2607_11897_amd import sfda
    x = make(2, 1, 256, m, n, 16, seed=17)
    say("f32 -> bf16", (2, 1, 256, m, n), "G", G)
    d = upload(x)
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=16,
                          segments=G, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    o, S = to_complex(o), to_complex(S)
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say("err(o)", eo, "err(S_T)", es)
    assert eo <= 2e-2 and es <= 1e-4


@pytest.mark.parametrize("dtype,G", [("f32", 4), ("bf16", 8)])
def test_segmented_strong_decay(dtype, G):
    """alpha ~ U(0.02, 0.1): a segment's transfer decays to far below the float range (its
    product P_g and the readouts X_t underflow to zero after a few chunks) and each 16-token
    block stays inside it; o and S_T within the bars (float32: the segment forward and the
    join; bfloat16: three passes)."""
    import math
    laws = I.Laws(alpha=("uniform", 0.02, 0.1), theta=("uniform", -math.pi, math.pi),
                  beta=("uniform", 0.0, 1.0), s0_scale=0.1)
    w = I.Workload("seg_strong", 1, 2, 512, 64, 48, 16, dtype, laws, 23, 1e-4)
    x = I.make_chunk_inputs(w)
    say(dtype, "strong decay, G", G)
    o, S = run(x, 16, G)
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say("err(o)", eo, "err(S_T)", es)
    tol = 1e-4 if dtype == "f32" else 2e-2
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))
    assert eo <= tol and es <= tol


def test_segmented_zero_state_and_in_place():
    x = make(1, 2, 128, 64, 64, 16, zero_state=True)
    o, S = run(x, 16, 4)
    o_ref, S_ref = run_oracle(x)
    assert rel_err(o, o_ref) <= 1e-4 and rel_err(S, S_ref) <= 1e-4
    x = make(1, 2, 128, 64, 64, 16, seed=5)
    o, S = run(x, 16, 4, in_place=True)          # S_T written over S0
    o_ref, S_ref = run_oracle(x)
    say("in place: err(o)", rel_err(o, o_ref), "err(S_T)", rel_err(S, S_ref))
    assert rel_err(o, o_ref) <= 1e-4 and rel_err(S, S_ref) <= 1e-4


@pytest.mark.parametrize("C,G", [(64, 4), (32, 8), (16, 2)])
def test_segmented_bf16(C, G):
    x = make(1, 2, 512, 64, 64, C, dtype="bf16")
    say("bf16 C", C, "G", G)
    o, S = run(x, C, G)
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say("err(o)", eo, "err(S_T)", es)
    assert eo <= 2e-2 and es <= 2e-2


def test_segmented_shape_error_launches_nothing():
    import torch
    from paper_2607_11897_amd import sfda
    x = make(1, 1, 96, 16, 8, 16)
    d = upload(x)
    with pytest.raises(sfda.SfdaError):
        sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=16,
                       segments=4)          # 96 is not a multiple of 4 * 16
    torch.cuda.synchronize()


def test_long_f32_h16_t64k_segmented_sampled_heads():
    """The long-context workload with 16 segments per head (the benchmarked setting): error
    of o over prefix windows and of S_T for two heads."""
    w = I.WORKLOADS["long_f32_h16_t64k"]
    say(w.name, "generating")
    x = I.make_chunk_inputs(w)
    say(w.name, "running, 16 segments")
    o, S = run(x, w.C, 16)
    for h in (0, 9):
        o_ref, S_ref = run_oracle(x.head(0, h))
        errs = {2 ** lg: rel_err(o[0, h, :2 ** lg], o_ref[0, 0, :2 ** lg]) for lg in range(10, 17)}
        es = rel_err(S[0, h], S_ref[0, 0])
        say(w.name, "head", h, "err(o) by prefix", errs, "err(S_T)", es)
        assert max(errs.values()) <= w.tol and es <= w.tol


def _policy(B, H, T, m, n, C, cus, dtype):
    """The segment count rule of sfda_chunk_fwd_auto_segments, restated."""
    per = B * H * ((n + 63) // 64)
    G = 1
    while G < 1024 and per * 2 * G <= cus and T % (2 * G * C) == 0 and T // (2 * G) >= 256:
        G *= 2
    return G if G >= (4 if dtype == "f32" else 8) else 1


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,H,T,m,n,C", [
    (4, 8, 2048, 64, 64, 64),       # the float32 workload: 32 heads
    (8, 16, 4096, 64, 64, 64),      # the benchmarked bf16 workload: enough heads, no segments
    (1, 16, 65536, 64, 64, 64),     # long context
    (4, 16, 4096, 64, 64, 64),      # 64 heads: G = 4, segments for float32 only
    (1, 2, 4096, 64, 64, 64),
    (1, 2, 4000, 64, 64, 64),       # T not a multiple of 8 C: no segments
    (1, 1, 1024, 64, 130, 16),
])
def test_auto_segments_policy(B, H, T, m, n, C, dtype):
    import torch
    from paper_2607_11897_amd import sfda
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    G = sfda.auto_segments(B, H, T, m, n, C, dtype)
    say("auto segments", (B, H, T, m, n, C), dtype, "CUs", cus, "G", G)
    assert G == _policy(B, H, T, m, n, C, cus, dtype)
    if cus >= 256 and (B, H, T) == (4, 8, 2048):
        assert G == 8
    if (B, H, T) == (8, 16, 4096):
        assert G == 1


def test_default_picks_segments_for_few_heads():
    """chunk_fwd's default on 2 heads x 4096 tokens runs the segmented scan the policy picks:
    the same bits as asking for that G, and the oracle's result within the float32 bar."""
    import torch
    from paper_2607_11897_amd import sfda
    x = make(1, 2, 4096, 64, 64, 64)
    G = sfda.auto_segments(1, 2, 4096, 64, 64, 64)
    say("default segments", G)
    assert G > 1
    d = upload(x)
    o1, S1 = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=64)
    o2, S2 = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=64,
                            segments=G)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(S1, S2)
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(to_complex(o1), o_ref), rel_err(to_complex(S1), S_ref)
    say("default segments err(o)", eo, "err(S_T)", es)
    assert eo <= 1e-4 and es <= 1e-4
