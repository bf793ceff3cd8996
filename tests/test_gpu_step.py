"""GPU parity of sfda_step (recurrent decode) against the complex128 oracle."""
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


def _head_list(B, H):
    return [(b, h) for b in range(B) for h in range(H)]


@pytest.mark.parametrize("B,H,m,n,dtype", [(2, 3, 64, 64, "f32"), (1, 2, 5, 3, "f32"),
                                           (2, 2, 64, 100, "f32"), (1, 1, 16, 8, "f32"),
                                           (2, 3, 64, 64, "bf16"), (3, 1, 33, 17, "f32"),
                                           (2, 2, 60, 40, "f32"), (1, 3, 50, 130, "bf16"),
                                           (2, 1, 7, 2, "f32"), (1, 2, 64, 4, "bf16")])
def test_step_small(B, H, m, n, dtype):
    import torch
    import oracle
    from paper_2607_11897_amd import sfda
    heads = _head_list(B, H)
    S = np.stack([I.decode_state_head(b, h, m, n) for (b, h) in heads]).reshape(B, H, m, n)
    Sd = to_device(I.to_storage(S, "f32"), "f32")
    say("step", B, H, m, n, dtype)
    tol = 1e-4 if dtype == "f32" else 2e-2
    for step in range(5):
        x = I.decode_step_heads(step, heads, m, n, dtype=dtype)
        st = x.storage()
        d = {k: to_device(st[k], dtype).reshape((B, H) + st[k].shape[2:]) for k in st}
        o = sfda.step(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], Sd)
        torch.cuda.synchronize()
        rs = lambda a: a.reshape((B, H) + a.shape[2:])
        o_ref, S = oracle.step(rs(x.q), rs(x.k), rs(x.v), rs(x.alpha), rs(x.theta), rs(x.beta), S)
        eo, es = rel_err(to_complex(o), o_ref), rel_err(to_complex(Sd), S)
        assert eo <= tol and es <= tol, (step, eo, es)
        if dtype == "f32":
            S = to_complex(Sd)   # keep both sides on the same state (checks one step at a time)


@pytest.mark.parametrize("m,n", [(64, 64), (60, 40), (50, 130), (7, 2)])
def test_step_guard_bands_untouched(m, n):
    """Canary words around S and o stay intact: rows past m, columns past n in a ragged last
    slice and the last head's state never write outside their buffers."""
    import torch
    import oracle
    from paper_2607_11897_amd import sfda
    B, H = 2, 2
    heads = _head_list(B, H)
    pad = 256
    canary = -12288.0
    S = np.stack([I.decode_state_head(b, h, m, n) for (b, h) in heads]).reshape(B, H, m, n)
    sb = torch.full((2 * pad + B * H * m * n * 2,), canary, device="cuda")
    ob = torch.full((2 * pad + B * H * n * 2,), canary, device="cuda")
    Sd = sb[pad:pad + B * H * m * n * 2].view(B, H, m, n, 2)
    Sd.copy_(to_device(I.to_storage(S, "f32"), "f32"))
    o = ob[pad:pad + B * H * n * 2].view(B, H, n, 2)
    x = I.decode_step_heads(0, heads, m, n)
    st = x.storage()
    d = {k: to_device(st[k], "f32").reshape((B, H) + st[k].shape[2:]) for k in st}
    say("step guard bands", m, n)
    sfda.step(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], Sd, o=o)
    torch.cuda.synchronize()
    for buf in (sb, ob):
        assert torch.all(buf[:pad] == canary) and torch.all(buf[-pad:] == canary)
    rs = lambda a: a.reshape((B, H) + a.shape[2:])
    o_ref, S_ref = oracle.step(rs(x.q), rs(x.k), rs(x.v), rs(x.alpha), rs(x.theta), rs(x.beta), S)
    assert rel_err(to_complex(o), o_ref) <= 1e-4 and rel_err(to_complex(Sd), S_ref) <= 1e-4


def test_decode_f32_b512h32_1024_steps_sampled_heads():
    """The decode workload: state [512, 32, 64, 64] complex fp32, 1024 steps with fresh
    inputs.  Eight heads take their inputs from the seeded numpy generator and are followed
    by the oracle across all 1024 steps; the other heads get torch-generated inputs with
    the same laws."""
    import torch
    import oracle
    from paper_2607_11897_amd import sfda
    D = I.DECODE
    B, H, m, n, steps = D["B"], D["H"], D["m"], D["n"], D["steps"]
    sample = [(0, 0), (17, 3), (100, 31), (255, 16), (256, 0), (333, 7), (480, 29), (511, 31)]
    say("decode full size, allocating state")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(D["seed"])
    Sd = (torch.randn(B, H, m, n, 2, generator=gen, device="cuda") * (0.1 / np.sqrt(2.0)))
    S_ref = np.stack([I.decode_state_head(b, h, m, n) for (b, h) in sample])[None]
    for i, (b, h) in enumerate(sample):
        Sd[b, h] = to_device(I.to_storage(S_ref[0, i], "f32"), "f32")
    idx_b = torch.tensor([b for b, _ in sample], device="cuda")
    idx_h = torch.tensor([h for _, h in sample], device="cuda")
    worst_o = 0.0
    for step in range(steps):
        q, k, v, a, th, bt = I.fill_decode_bulk_torch(gen, B, H, m, n, "cuda")
        x = I.decode_step_heads(step, sample, m, n)
        st = x.storage()
        for t, key in ((q, "q"), (k, "k"), (v, "v"), (a, "alpha"), (th, "theta"), (bt, "beta")):
            t[idx_b, idx_h] = to_device(st[key][0], "f32")
        o = sfda.step(q, k, v, a, th, bt, Sd)
        o_s = to_complex(o[idx_b, idx_h])[None]
        o_ref, S_ref = oracle.step(x.q, x.k, x.v, x.alpha, x.theta, x.beta, S_ref)
        worst_o = max(worst_o, rel_err(o_s, o_ref))
        if step % 128 == 0 or step == steps - 1:
            say("decode step", step, "worst err(o) so far", worst_o)
        assert worst_o <= D["tol"], (step, worst_o)
    torch.cuda.synchronize()
    es = rel_err(to_complex(Sd[idx_b, idx_h])[None], S_ref)
    say("decode final err(S)", es)
    assert es <= D["tol"]
