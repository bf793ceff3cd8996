"""GPU checks of sfda_chunk_solve_monitor, the conditioning watch of Prop. 6.4: for every
16-token block, ||D_beta L'||_F and the residual max |(I + D_beta L') N - I| of the
substitution that forms N = (I + D_beta L')^{-1} in the chunk kernels.

||D_beta L'||_F is compared with the oracle's L' of the same block (the closed forms of the
chunk relations, oracle.chunk_wy.ut_chunk) on the stored inputs: within 1e-4 relative for
float32 inputs, 2e-2 for bfloat16 ones (the kernels' Gram products then take bfloat16
operands).  The residual has no reference value (it measures the kernel's own rounding);
it is checked against the classical bound for a triangular solve and the evaluation of
the residual in float32, |R| <= (gamma_16 + gamma_17)(|I + X| |N| + 1) entrywise
(gamma_n = n u / (1 - n u), u = 2^-24; X = D_beta L' and N from the oracle), with a factor
4 for complex arithmetic; beta = 0 gives exactly zero, and a block outside the decay range
gives NaN."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_util import I, ensure_built, upload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def lib():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return ensure_built()


def say(*a):
    print("[case]", *a, flush=True)


def small(T, dtype, B=1, H=2, m=64, seed=31):
    w = I.Workload("monitor", B, H, T, m, 8, 16, dtype, I.LAWS_MAIN, seed, 1e-4)
    return I.make_chunk_inputs(w)


def run(x):
    import torch
    from paper_2607_11897_amd import sfda
    d = upload(x)
    res, ln = sfda.chunk_solve_monitor(d["k"], d["alpha"], d["theta"], d["beta"])
    torch.cuda.synchronize()
    return res.cpu().numpy().astype(np.float64), ln.cpu().numpy().astype(np.float64)


def oracle_blocks(x, b, h):
    """Per 16-token block of head (b, h): (||D_beta L'||_F, the residual bound)."""
    from oracle.chunk_wy import ut_chunk
    T, m = x.k.shape[2], x.k.shape[3]
    u = 2.0 ** -24
    gam = lambda n: n * u / (1 - n * u)
    out = []
    for t0 in range(0, T, 16):
        sl = slice(t0, min(T, t0 + 16))
        k = x.k[b, h, sl]
        C = k.shape[0]
        _, _, parts = ut_chunk(np.zeros_like(k), k, np.zeros((C, 1), complex), x.alpha[b, h, sl],
                               x.theta[b, h, sl], x.beta[b, h, sl], np.zeros((m, 1), complex))
        X = np.diag(x.beta[b, h, sl].astype(complex)) @ parts["L"]
        N = np.linalg.inv(np.eye(C) + X)
        bound = 4 * (gam(16) + gam(17)) * (np.max(np.abs(np.eye(C) + X) @ np.abs(N)) + 1)
        out.append((np.linalg.norm(X), bound))
    return np.array(out)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_monitor_against_definition(dtype):
    x = small(T=16 * 6 + 7, dtype=dtype)
    say("monitor", dtype)
    res, ln = run(x)
    tol = 1e-4 if dtype == "f32" else 2e-2
    for h in range(2):
        ref = oracle_blocks(x, 0, h)
        assert res.shape == (1, 2, 7) and ln.shape == (1, 2, 7)
        err = np.max(np.abs(ln[0, h] - ref[:, 0]) / np.maximum(ref[:, 0], 1e-30))
        say(dtype, "head", h, "lnorm", ln[0, h], "rel err", err, "residual", res[0, h], "bound", ref[:, 1])
        assert err <= tol
        assert np.all(np.isfinite(res[0, h])) and np.all(res[0, h] <= ref[:, 1])


def test_monitor_beta_zero_is_exact():
    """beta = 0: D_beta L' = 0, N = I, both figures exactly zero."""
    x = small(T=64, dtype="f32")
    x.beta[...] = 0.0
    res, ln = run(x)
    assert np.all(res == 0.0) and np.all(ln == 0.0)


def test_monitor_outside_decay_range_is_nan():
    """A block whose decay falls below 2^-126 (alpha = 0.001 on one channel, tokens 32..47)
    gives NaN there; the other blocks are unaffected."""
    x = small(T=80, dtype="f32")
    x.alpha[..., 32:48, 5] = I.round_to_storage(np.full(16, 0.001), "f32")
    res, ln = run(x)
    assert np.all(np.isnan(res[..., 2])) and np.all(np.isnan(ln[..., 2]))
    keep = [0, 1, 3, 4]
    assert np.all(np.isfinite(res[..., keep])) and np.all(np.isfinite(ln[..., keep]))


def test_monitor_benchmarked_workload():
    """The benchmarked bf16 workload at full size: every block well inside Prop. 6.4's
    condition, residuals at float32 rounding."""
    w = I.WORKLOADS["fwd_bf16_b8h16_t4k"]
    x = I.make_chunk_inputs(w)
    say(w.name, "monitor")
    res, ln = run(x)
    say(w.name, "max residual", res.max(), "max ||D_beta L'||_F", ln.max(), "median", np.median(ln))
    assert np.all(np.isfinite(res)) and np.all(np.isfinite(ln))
    assert res.max() <= 1e-5
