"""The allocation-free entry point sfda_chunk_fwd_segmented_noalloc (workspace in the
library's static device scratch) against sfda_chunk_fwd_segmented with a caller-owned
workspace: two calls in a row, the second smaller, each bitwise equal to the existing entry
point (same kernels on the same workspace layout) and within the float32 / bfloat16 bars of
the oracle; a request beyond the scratch is refused without a launch."""
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


def both(x, C, G):
    import torch
    from paper_2607_11897_amd import sfda
    d = upload(x)
    args = (d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"])
    o_ref, S_ref = sfda.chunk_fwd(*args, C=C, segments=G)
    o, S = sfda.chunk_fwd_segmented_noalloc(*args, C=C, segments=G)
    torch.cuda.synchronize()
    return to_complex(o), to_complex(S), to_complex(o_ref), to_complex(S_ref)


def test_noalloc_two_calls_match_segmented():
    cases = [  # (B, H, T, m, n, C, G, dtype): the second is smaller and changes every size
        (2, 3, 256, 64, 64, 32, 4, "f32"),
        (1, 2, 96, 16, 8, 16, 3, "bf16"),
    ]
    for (B, H, T, m, n, C, G, dt) in cases:
        w = I.Workload("noalloc", B, H, T, m, n, C, dt, I.LAWS_MAIN, 11 + T, 1e-4)
        x = I.make_chunk_inputs(w)
        say("noalloc", (B, H, T, m, n), "C", C, "G", G, dt)
        o, S, o_ref, S_ref = both(x, C, G)
        assert np.array_equal(o, o_ref) and np.array_equal(S, S_ref)
        o_or, S_or = run_oracle(x)
        tol = 1e-4 if dt == "f32" else 2e-2
        eo, es = rel_err(o, o_or), rel_err(S, S_or)
        say("err(o)", eo, "err(S_T)", es)
        assert eo <= tol and es <= tol


def test_noalloc_refuses_beyond_scratch():
    import torch
    from paper_2607_11897_amd import sfda
    w = I.Workload("big", 1, 64, 128, 64, 64, 16, "f32", I.LAWS_MAIN, 5, 1e-4)
    x = I.make_chunk_inputs(w)
    d = upload(x)
    say("noalloc beyond scratch")
    with pytest.raises(sfda.SfdaError, match="SFDA_ERR_SCRATCH"):
        sfda.chunk_fwd_segmented_noalloc(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"],
                                         C=16, segments=8)
    torch.cuda.synchronize()
