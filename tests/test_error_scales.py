"""Pins of the componentwise error scales used in the bfloat16 gradient bars (CPU only):
each scale bounds the magnitude of the exact gradient element by element (triangle
inequality), is exact where no term cancels (beta = 0: dS0 = conj(lambda) G exactly; n = 1
also makes |g| a single term), and at m = 1 the cancellation it measures is the scalar
erase factor 1 - beta |k|^2."""
from __future__ import annotations

import numpy as np

from error_scales import bf16_gradient_bound, erase_term_scales
from oracle import backward as BW


def cn(rng, shape):
    return (rng.normal(size=shape) + 1j * rng.normal(size=shape)) / np.sqrt(2.0)


def sample(seed, B=1, H=2, T=9, m=5, n=4):
    rng = np.random.default_rng(seed)
    k = cn(rng, (B, H, T, m))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    return dict(q=cn(rng, (B, H, T, m)), k=k, v=cn(rng, (B, H, T, n)),
                alpha=rng.uniform(0.7, 1.0, (B, H, T, m)), theta=rng.uniform(-np.pi, np.pi, (B, H, T, m)),
                beta=rng.uniform(0, 1, (B, H, T)), S0=cn(rng, (B, H, m, n)),
                dO=cn(rng, (B, H, T, n)), dS_T=cn(rng, (B, H, m, n)))


def both(x):
    ref = BW.recurrence_backward(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], x["S0"],
                                 x["dO"], x["dS_T"])
    sc = erase_term_scales(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], x["S0"],
                           x["dO"], x["dS_T"])
    return ref, sc


def test_scales_bound_the_exact_gradients():
    for seed in range(4):
        ref, sc = both(sample(seed))
        for name in ("dS0", "dalpha", "dtheta"):
            assert np.all(np.abs(ref[name]) <= sc[name] * (1 + 1e-12) + 1e-300), (seed, name)


def test_scales_are_exact_without_the_erase():
    x = sample(7, n=1)
    x["beta"] = np.zeros_like(x["beta"])
    ref, sc = both(x)
    assert np.allclose(sc["dS0"], np.abs(ref["dS0"]), rtol=1e-12, atol=0)
    # with one value column and no erase, g is a single product: |dalpha|^2 + |dtheta / alpha|^2 = |g|^2
    g = np.hypot(ref["dalpha"], ref["dtheta"] / x["alpha"])
    assert np.allclose(g, sc["dalpha"], rtol=1e-12, atol=0)


def test_single_channel_cancellation_is_the_erase_factor():
    x = sample(3, T=1, m=1, n=6)
    x["k"] = np.ones_like(x["k"])                       # |k|^2 = 1
    ref, sc = both(x)
    beta = x["beta"][:, :, 0]
    # exact dS0 = conj(lambda) (1 - beta) G; the scale is alpha (1 + beta) |G|
    ratio = np.abs(ref["dS0"]) / sc["dS0"]
    assert np.allclose(ratio, ((1 - beta) / (1 + beta))[..., None, None], rtol=1e-12)


def test_bound_widens_only_the_erase_gradients():
    ref, sc = both(sample(1))
    assert bf16_gradient_bound("dq", ref["dq"], sc) == 2e-2 * np.max(np.abs(ref["dq"]))
    assert bf16_gradient_bound("dS0", ref["dS0"], sc) >= 2e-2 * np.max(np.abs(ref["dS0"]))
