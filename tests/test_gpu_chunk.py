"""GPU parity of sfda_chunk_fwd against the complex128 oracle (token-by-token recurrence).

Bars: max-norm relative error <= 1e-4 for float32 inputs, <= 2e-2 for bfloat16 inputs with
float32 accumulation and state; checked on o and on S_T.  Full-size workloads run in the
same launch configuration as bench.py and are checked on a sampled set of heads (heads are
independent, so a sampled head's oracle result is exact for that head).
"""
from __future__ import annotations

import math

import numpy as np
import pytest

from gpu_util import I, ensure_built, rel_err, run_chunk, run_oracle, upload, to_complex

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return ensure_built()


def say(*a):
    print("[case]", *a, flush=True)


def check(x, C, tol, out_dtype=None, slice=None, label="", segments="auto"):
    say(label, x.shape, "C", C, x.dtype, "slice", slice, "segments", segments)
    o, S = run_chunk(x, C, out_dtype=out_dtype, slice=slice, segments=segments)
    o_ref, S_ref = run_oracle(x)
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say(label, "err(o)", eo, "err(S_T)", es)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))
    assert eo <= tol and es <= tol, (label, eo, es)
    return eo, es


def small(T=100, B=1, H=2, m=64, n=64, dtype="f32", laws=I.LAWS_MAIN, seed=7):
    w = I.Workload("case", B, H, T, m, n, 16, dtype, laws, seed, 1e-4)
    return I.make_chunk_inputs(w)


# --------------------------------------------------------------------------- workloads

@pytest.mark.parametrize("name", ["tiny_f32", "tiny_f32_n16"])
def test_tiny(name):
    w = I.WORKLOADS[name]
    check(I.make_chunk_inputs(w), w.C, w.tol, label=name)


@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_chunk_sizes_ragged(C):
    check(small(T=3 * C + 5), C, 1e-4, label=f"C{C}")


@pytest.mark.parametrize("m,n", [(5, 3), (16, 8), (33, 24), (64, 80), (48, 130)])
def test_odd_shapes(m, n):
    check(small(T=40, m=m, n=n, B=2, H=1), 16, 1e-4, label=f"m{m}n{n}")


@pytest.mark.parametrize("slice", [8, 16, 32, 64])
def test_slices_agree(slice):
    check(small(T=130, n=64), 64, 1e-4, slice=slice, label=f"slice{slice}")


def test_bf16_small():
    check(small(T=300, dtype="bf16"), 64, 2e-2, label="bf16")


def test_f32_in_bf16_out():
    x = small(T=70)
    say("f32 in, bf16 out")
    o, S = run_chunk(x, 64, out_dtype="bf16")
    o_ref, S_ref = run_oracle(x)
    assert rel_err(o, o_ref) <= 1e-2 and rel_err(S, S_ref) <= 1e-4


STRONG = I.Laws(alpha=("uniform", 0.02, 0.1), theta=("uniform", -math.pi, math.pi),
                beta=("uniform", 0.0, 1.0), s0_scale=0.1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_strong_decay(C, dtype):
    """alpha ~ U(0.02, 0.1): the decay over one 64-token chunk reaches 1e-109, far below the
    float range, while every decay ratio inside a 16-token block stays above 2^-126 (the
    local renormalisation of App. C.4)."""
    check(small(T=3 * 64 + 37, laws=STRONG, dtype=dtype), C, 1e-4 if dtype == "f32" else 2e-2,
          label=f"strong {dtype} C{C}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("s0", [0.1, None])
def test_unit_and_tiny_decay_across_channels(dtype, s0):
    """alpha exactly 1 on the even channels (no decay at all) and alpha ~ U(0.005, 0.01) on the
    odd ones (a 16-token block decays to 1e-32 .. 1e-37 there), with and without an initial
    state."""
    laws = I.Laws(alpha=("mixed", 0.005, 0.01), theta=("uniform", -math.pi, math.pi),
                  beta=("uniform", 0.0, 1.0), s0_scale=s0)
    check(small(T=200, laws=laws, dtype=dtype), 64, 1e-4 if dtype == "f32" else 2e-2,
          label=f"mixed {dtype} S0 {s0}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_large_theta(dtype):
    """theta ~ U(-50, 50) per token and channel: the phase sums reach hundreds of
    revolutions within a chunk; the kernels reduce them to [0, 1) revolutions token by
    token, so the rotations stay exact to rounding."""
    laws = I.Laws(alpha=("uniform", 0.9, 1.0), theta=("uniform", -50.0, 50.0),
                  beta=("uniform", 0.0, 1.0), s0_scale=0.1)
    check(small(T=3 * 64 + 37, laws=laws, dtype=dtype), 64, 1e-4 if dtype == "f32" else 2e-2,
          label=f"large theta {dtype}")


@pytest.mark.parametrize("dtype,ok_until,nan_from", [("bf16", 128, 128), ("f32", 144, 156)])
def test_decay_outside_range_returns_nan(dtype, ok_until, nan_from):
    """One channel decaying by 1e-48 over a whole 16-token block (alpha = 0.001, tokens
    144..159) is outside the decay range.  bf16 evaluates 64-token steps of 16-token blocks:
    the steps before the one holding that block (tokens < 128) are unaffected and match the
    oracle, from that step on the outputs and S_T are NaN.  float32 evaluates 16-token
    chunks and poisons the operand of a token once the chunk's decay so far drops below
    2^-126 (0.001^13 = 1e-39, token 156): the chunks before (tokens < 144) match the oracle,
    every output from that token on and S_T are NaN (the chunk's triangular solve may carry
    the NaN to its earlier rows too)."""
    x = small(T=200, dtype=dtype)
    x.alpha[..., 144:160, 7] = I.round_to_storage(np.full(16, 0.001), dtype)
    say(dtype, "out of range")
    o, S = run_chunk(x, 64)
    o_ref, _ = run_oracle(x)
    tol = 2e-2 if dtype == "bf16" else 1e-4
    assert rel_err(o[:, :, :ok_until], o_ref[:, :, :ok_until]) <= tol
    assert np.all(np.isnan(o[:, :, nan_from:])) and np.all(np.isnan(S))


def test_bf16_every_chunk_length_bitwise_equal():
    """The bf16 path evaluates 16-token blocks whatever C is (Thm 6.1: the result does not
    depend on the chunk length), so every accepted C gives the same bits."""
    x = small(T=3 * 64 + 37, dtype="bf16")
    say("bf16 C invariance")
    o64, S64 = run_chunk(x, 64)
    for C in (16, 32, 128):
        o, S = run_chunk(x, C)
        assert np.array_equal(o, o64) and np.array_equal(S, S64), C


@pytest.mark.parametrize("segments", [None, "auto"])
def test_fwd_f32_b4h8_t2k_full(segments):
    """The float32 workload at full size, with one scan per head and with the binding's
    default (32 heads: segment-parallel on a 256-CU device)."""
    w = I.WORKLOADS["fwd_f32_b4h8_t2k"]
    check(I.make_chunk_inputs(w), w.C, w.tol, label=w.name, segments=segments)


def test_fwd_bf16_b8h16_t4k_full_sampled_heads():
    """The benchmarked workload, run at full size; six heads are checked against the oracle."""
    w = I.WORKLOADS["fwd_bf16_b8h16_t4k"]
    say(w.name, "generating")
    x = I.make_chunk_inputs(w)
    say(w.name, "running")
    o, S = run_chunk(x, w.C)
    heads = [(0, 0), (1, 5), (3, 15), (4, 7), (6, 2), (7, 15)]
    for (b, h) in heads:
        xo = x.head(b, h)
        o_ref, S_ref = run_oracle(xo)
        eo, es = rel_err(o[b, h], o_ref[0, 0]), rel_err(S[b, h], S_ref[0, 0])
        say(w.name, (b, h), "err(o)", eo, "err(S_T)", es)
        assert eo <= w.tol and es <= w.tol
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))


def test_long_f32_h16_t64k_sampled_heads():
    """Long context: error of o over prefix windows and of S_T, for two heads."""
    w = I.WORKLOADS["long_f32_h16_t64k"]
    say(w.name, "generating")
    x = I.make_chunk_inputs(w)
    say(w.name, "running")
    o, S = run_chunk(x, w.C)
    for h in (0, 9):
        xo = x.head(0, h)
        o_ref, S_ref = run_oracle(xo)
        errs = {}
        for lg in range(10, 17):
            Tp = 2 ** lg
            errs[Tp] = rel_err(o[0, h, :Tp], o_ref[0, 0, :Tp])
        es = rel_err(S[0, h], S_ref[0, 0])
        say(w.name, "head", h, "err(o) by prefix", errs, "err(S_T)", es)
        assert max(errs.values()) <= w.tol and es <= w.tol


# --------------------------------------------------------------------------- edge cases

def test_T0_copies_state_and_in_place():
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=0)
    d = upload(x)
    say("T=0")
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=64)
    torch.cuda.synchronize()
    assert np.array_equal(to_complex(S), x.S0)
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], None, C=64)
    torch.cuda.synchronize()
    assert np.all(to_complex(S) == 0)


def test_state_in_place_and_resume():
    """S_T == S0 in place; running T1 then T2 tokens from S_T(T1) equals one run over T1+T2
    (the affine chunk parenthesisation, Cor. A.3), within the fp32 bar."""
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=150)
    d = upload(x)
    say("resume")
    o_all, S_all = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=64)
    S = d["S0"].clone()
    outs = []
    for (a, b) in ((0, 37), (37, 101), (101, 150)):
        sl = lambda t: t[:, :, a:b].contiguous()
        o, _ = sfda.chunk_fwd(sl(d["q"]), sl(d["k"]), sl(d["v"]), sl(d["alpha"]), sl(d["theta"]),
                              sl(d["beta"]), S, C=64, S_T=S)
        outs.append(o)
    torch.cuda.synchronize()
    o_ref, S_ref = run_oracle(x)
    assert rel_err(to_complex(torch.cat(outs, dim=2)), o_ref) <= 1e-4
    assert rel_err(to_complex(S), S_ref) <= 1e-4
    assert rel_err(to_complex(S), to_complex(S_all)) <= 1e-5


def test_one_token_matches_step():
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=1, B=2, H=3)
    d = upload(x)
    say("T=1 vs step")
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=16)
    S2 = d["S0"].clone()
    o2 = sfda.step(d["q"][:, :, 0].contiguous(), d["k"][:, :, 0].contiguous(), d["v"][:, :, 0].contiguous(),
                   d["alpha"][:, :, 0].contiguous(), d["theta"][:, :, 0].contiguous(),
                   d["beta"][:, :, 0].contiguous(), S2)
    torch.cuda.synchronize()
    assert rel_err(to_complex(o)[:, :, 0], to_complex(o2)) <= 1e-5
    assert rel_err(to_complex(S), to_complex(S2)) <= 1e-5


def test_deterministic_bitwise():
    x = small(T=200, dtype="bf16")
    say("determinism")
    o1, S1 = run_chunk(x, 64)
    o2, S2 = run_chunk(x, 64)
    assert np.array_equal(o1, o2) and np.array_equal(S1, S2)


def test_guard_bands_untouched():
    """Canary words around o and S_T stay intact (no out-of-range writes)."""
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=77, m=40, n=24, B=2, H=2)
    d = upload(x)
    B, H, T, m, n = x.shape
    pad = 256
    canary = -12345.0
    ob = torch.full((2 * pad + B * H * T * n * 2,), canary, device="cuda")
    sb = torch.full((2 * pad + B * H * m * n * 2,), canary, device="cuda")
    o = ob[pad:pad + B * H * T * n * 2].view(B, H, T, n, 2)
    S = sb[pad:pad + B * H * m * n * 2].view(B, H, m, n, 2)
    say("guard bands")
    sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=32, o=o, S_T=S)
    torch.cuda.synchronize()
    for buf in (ob, sb):
        assert torch.all(buf[:pad] == canary) and torch.all(buf[-pad:] == canary)
    o_ref, S_ref = run_oracle(x)
    assert rel_err(to_complex(o), o_ref) <= 1e-4 and rel_err(to_complex(S), S_ref) <= 1e-4


def test_zero_heads_is_noop():
    import torch
    from paper_2607_11897_amd import sfda
    e = torch.empty((0, 3, 10, 64, 2), device="cuda")
    say("B=0")
    o, S = sfda.chunk_fwd(e, e, e, e[..., 0], e[..., 0], e[..., 0, 0], None, C=64)
    assert o.numel() == 0 and S.numel() == 0


# --------------------------------------------------------------------------- bf16 pipeline kernel
# bf16 inputs run a different kernel (producer/consumer pipeline with range-checked buffer
# loads and stores); its ragged tails, narrow shapes and slices are covered here.

@pytest.mark.parametrize("C", [16, 32, 64, 128])
def test_bf16_chunk_sizes_ragged(C):
    check(small(T=3 * C + 5, dtype="bf16"), C, 2e-2, label=f"bf16 C{C}")


@pytest.mark.parametrize("T", [1, 15, 64, 65])
def test_bf16_short_sequences(T):
    check(small(T=T, dtype="bf16"), 64, 2e-2, label=f"bf16 T{T}")


@pytest.mark.parametrize("m,n", [(5, 3), (16, 8), (33, 24), (60, 40), (64, 80), (48, 130)])
def test_bf16_odd_shapes(m, n):
    # m % 4 != 0 loads one channel per instruction; m < 64 leaves channel groups past m;
    # n that is not a multiple of 16 leaves a partial consumer wave
    check(small(T=70, m=m, n=n, B=2, H=1, dtype="bf16"), 16, 2e-2, label=f"bf16 m{m}n{n}")


@pytest.mark.parametrize("slice", [8, 16, 24, 32, 40, 64])
def test_bf16_slices(slice):
    check(small(T=130, n=64, dtype="bf16"), 64, 2e-2, slice=slice, label=f"bf16 slice{slice}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_slices_bitwise_equal(dtype):
    """Every value column's arithmetic is the same whatever the column slice, so the slice
    sfda_chunk_fwd picks by itself (32 columns when heads are few) changes no bit."""
    x = small(T=150, B=1, H=2, n=64, dtype=dtype)
    say("slices bitwise", dtype)
    o0, S0 = run_chunk(x, 64)
    for sl in (64, 32, 16):
        o, S = run_chunk(x, 64, slice=sl)
        assert np.array_equal(o, o0) and np.array_equal(S, S0), sl


def test_bf16_in_f32_out():
    check(small(T=150, dtype="bf16"), 64, 2e-2, out_dtype="f32", label="bf16 in, f32 out")


def test_bf16_zero_state_and_strong_decay():
    laws = I.Laws(alpha=("uniform", 0.01, 0.02), theta=("uniform", -math.pi, math.pi),
                  beta=("uniform", 0.0, 1.0), s0_scale=None)
    check(small(T=200, laws=laws, dtype="bf16"), 64, 2e-2, label="bf16 S0=0 alpha0.01")


def test_bf16_resume_in_place():
    """bf16 inputs: three calls carrying S_T in place equal one call over the whole sequence."""
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=150, dtype="bf16")
    d = upload(x)
    say("bf16 resume")
    S = d["S0"].clone()
    outs = []
    for (a, b) in ((0, 37), (37, 101), (101, 150)):
        sl = lambda t: t[:, :, a:b].contiguous()
        o, _ = sfda.chunk_fwd(sl(d["q"]), sl(d["k"]), sl(d["v"]), sl(d["alpha"]), sl(d["theta"]),
                              sl(d["beta"]), S, C=64, S_T=S)
        outs.append(o)
    torch.cuda.synchronize()
    o_ref, S_ref = run_oracle(x)
    assert rel_err(to_complex(torch.cat(outs, dim=2)), o_ref) <= 2e-2
    assert rel_err(to_complex(S), S_ref) <= 2e-2


def test_bf16_T0_copies_state():
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=0, dtype="bf16")
    d = upload(x)
    say("bf16 T=0")
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=64)
    torch.cuda.synchronize()
    assert np.array_equal(to_complex(S), x.S0)


def test_bf16_guard_bands_untouched():
    """Canary words around o (bf16) and S_T stay intact: the dropped out-of-range stores of the
    ragged tail and of the columns past n never reach neighbouring memory."""
    import torch
    from paper_2607_11897_amd import sfda
    x = small(T=77, m=40, n=24, B=2, H=2, dtype="bf16")
    d = upload(x)
    B, H, T, m, n = x.shape
    pad = 256
    canary = -12288.0
    ob = torch.full((2 * pad + B * H * T * n * 2,), canary, device="cuda", dtype=torch.bfloat16)
    sb = torch.full((2 * pad + B * H * m * n * 2,), canary, device="cuda")
    o = ob[pad:pad + B * H * T * n * 2].view(B, H, T, n, 2)
    S = sb[pad:pad + B * H * m * n * 2].view(B, H, m, n, 2)
    say("bf16 guard bands")
    sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"], C=32, o=o, S_T=S)
    torch.cuda.synchronize()
    for buf in (ob, sb):
        assert torch.all(buf[:pad] == canary) and torch.all(buf[-pad:] == canary)
    o_ref, S_ref = run_oracle(x)
    assert rel_err(to_complex(o), o_ref) <= 2e-2 and rel_err(to_complex(S), S_ref) <= 2e-2


def test_bf16_largest_head():
    """One head of the longest sequence the bf16 path accepts with m = n = 64 and bf16 o
    (each head's q, k, v and o below 2 GiB: T = (2^31 - 1) // 256 = 8388607 tokens, a ragged
    last chunk).  Identity tokens (k = q = v = 0, beta = 0, alpha = 1, theta = 0) up to the
    last 1000 tokens, which follow the benchmark laws: the bulk's outputs are exactly zero,
    the state reaches the tail unchanged (S0), and the tail's outputs and S_T match the
    oracle run on the tail from S0.  Exercises the buffer ranges and offsets at the top of
    the allowed sizes."""
    import torch
    from paper_2607_11897_amd import sfda
    m = n = 64
    T = (2 ** 31 - 1) // (n * 2 * 2)
    tail = 1000
    w = I.Workload("largest", 1, 1, tail, m, n, 64, "bf16", I.LAWS_MAIN, 77, 2e-2)
    xt = I.make_chunk_inputs(w)
    st = xt.storage()
    say("bf16 largest head: T", T, "building inputs")
    dev = torch.device("cuda")

    def full(name, fill_bits, shape_tail):
        a = torch.full((T,) + shape_tail, fill_bits, dtype=torch.int16)
        a[T - tail:] = torch.from_numpy(np.ascontiguousarray(st[name][0, 0]).view(np.int16))
        return a.to(dev).view(torch.bfloat16).view((1, 1, T) + shape_tail)

    one = int(np.array([1.0], dtype=np.float32).view(np.uint32)[0] >> 16)   # bf16 bits of 1.0
    q = full("q", 0, (m, 2))
    k = full("k", 0, (m, 2))
    v = full("v", 0, (n, 2))
    alpha = full("alpha", one, (m,))
    theta = full("theta", 0, (m,))
    beta = full("beta", 0, ())
    S0 = torch.from_numpy(np.ascontiguousarray(st["S0"], dtype=np.float32)).to(dev)
    say("bf16 largest head: running")
    o, S = sfda.chunk_fwd(q, k, v, alpha, theta, beta, S0, C=64)
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(o[0, 0, :T - tail])) == 0     # value test: -0.0 counts as zero
    o_ref, S_ref = run_oracle(xt)
    eo = rel_err(to_complex(o[:, :, T - tail:]), o_ref)
    es = rel_err(to_complex(S), S_ref)
    say("bf16 largest head: err(o tail)", eo, "err(S_T)", es)
    assert eo <= 2e-2 and es <= 2e-2
