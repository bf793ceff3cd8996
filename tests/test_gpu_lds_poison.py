"""The LDS-poison debug build (libsfda_poison.so, built with SFDA_LDS_POISON): before each
chunk (fp32 path, backward scans) or pipeline step (bf16 path) rewrites its LDS operand
area, the kernels fill that area with NaN words, and the gradient pass fills its whole LDS
at entry; a stage that read an operand the current chunk or step had not written yet would
turn the outputs into NaN.  Every kernel family runs here against the oracle with the bars
of its own tests: the fp32 role-split forward and the bf16 pipeline (with and without the
32-column slice), the gated variants, the segment-parallel forward (fp32 join, bf16 third
pass), the write-decoupled forward and the backward."""
from __future__ import annotations

import os

import numpy as np
import pytest

from gpu_util import I, ensure_built, rel_err, run_chunk, run_oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def poison_lib():
    import torch
    from paper_2607_11897_amd import build, sfda
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    ensure_built()
    if not os.path.exists(build.POISON_LIB):
        build.build(verbose=False, poison=True, out=build.POISON_LIB)
    with sfda.library(build.POISON_LIB) as lib:
        yield lib
    torch.cuda.synchronize()


def say(*a):
    print("[case]", *a, flush=True)


def small(T, dtype, B=1, H=2, m=64, n=64, seed=71):
    w = I.Workload("poison", B, H, T, m, n, 16, dtype, I.LAWS_MAIN, seed, 1e-4)
    return I.make_chunk_inputs(w)


@pytest.mark.parametrize("dtype,slice_,segments", [
    ("f32", None, None), ("f32", 16, None), ("bf16", None, None), ("bf16", 32, None),
    ("bf16", 64, None), ("f32", None, 4), ("bf16", None, 4),
])
def test_forward_under_poison(dtype, slice_, segments):
    x = small(T=256 if segments else 150, dtype=dtype)
    say("poison forward", dtype, "slice", slice_, "segments", segments)
    o, S = run_chunk(x, 64, slice=slice_, segments=segments)
    o_ref, S_ref = run_oracle(x)
    tol = 1e-4 if dtype == "f32" else 2e-2
    eo, es = rel_err(o, o_ref), rel_err(S, S_ref)
    say("err(o)", eo, "err(S_T)", es)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))
    assert eo <= tol and es <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gated_under_poison(dtype):
    from test_gpu_gated import oracle_gated, run_gated
    g = I.make_gated_inputs(1, 2, 130, 64, 64, dtype, seed=77)
    o, S = run_gated(g, 64, 1e-6)
    o_ref, S_ref = oracle_gated(g, 1e-6)
    tol = 1e-4 if dtype == "f32" else 2e-2
    say("poison gated", dtype, rel_err(o, o_ref), rel_err(S, S_ref))
    assert np.all(np.isfinite(o)) and rel_err(o, o_ref) <= tol and rel_err(S, S_ref) <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decoupled_under_poison(dtype):
    from test_gpu_decoupled import oracle_dec, run_dec
    x = I.make_decoupled_inputs(1, 2, 100, 64, 64, dtype, seed=79)
    o, S = run_dec(x, 16)
    o_ref, S_ref = oracle_dec(x)
    tol = 1e-4 if dtype == "f32" else 2e-2
    say("poison decoupled", dtype, rel_err(o, o_ref), rel_err(S, S_ref))
    assert np.all(np.isfinite(o)) and rel_err(o, o_ref) <= tol and rel_err(S, S_ref) <= tol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_under_poison(dtype):
    from test_gpu_backward import check, make, oracle_bwd, run_bwd
    x = make(1, 2, 100, 64, 64, dtype, seed=83)
    dO, dS = I.make_cotangents(1, 2, 100, 64, 64, dtype, seed=84)
    got = run_bwd(x, dO, dS, 16, dtype)
    ref = oracle_bwd(x, dO, dS)
    check(got, ref, 1e-4 if dtype == "f32" else 2e-2, f"poison backward {dtype}")
