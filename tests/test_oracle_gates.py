"""Pins of the oracle's gate and key parameterization (Sec. 3, stable parameterization:
equations param-alpha, param-theta, param-beta, param-key), CPU only.

Each check rests on something other than the oracle's own formulas: a library routine
(scipy's logistic function), an inverse function (arctanh), an exact special value, a
symmetry, or a bound the paper states for the parameterized recurrence (||Lambda|| <= 1,
0 <= beta ||k||^2 <= 1, hence ||A_t||_2 <= 1 as in Prop. 6.3).  Copies of the map with a
planted mistake must each fail one of them.
"""
from __future__ import annotations

import numpy as np
import pytest
from scipy.special import expit

from oracle import gates as G

AMIN, AMAX, TMAX = 0.35, 0.999, 1.2


def sample(seed, T=64, m=16, scale=3.0):
    rng = np.random.default_rng(seed)
    a = rng.normal(0.0, scale, (T, m))
    b = rng.normal(0.0, scale, (T, m))
    c = rng.normal(0.0, scale, (T,))
    k_raw = rng.normal(0.0, 1.0, (T, m)) + 1j * rng.normal(0.0, 1.0, (T, m))
    return a, b, c, k_raw


def check_map(fn, eps=1e-3):
    """All pins for a gate map fn(a, b, c, k_raw, amin, amax, tmax, eps); returns the names
    of the pins that fail."""
    failed = []
    a, b, c, k_raw = sample(1)
    alpha, theta, beta, k = fn(a, b, c, k_raw, AMIN, AMAX, TMAX, eps)
    # sigmoid: scipy's logistic function, and beta is exactly it
    if not np.allclose(beta, expit(c), rtol=0, atol=1e-15):
        failed.append("beta = logistic(c)")
    # alpha: affine image of the logistic function onto [amin, amax]
    if not np.allclose((alpha - AMIN) / (AMAX - AMIN), expit(a), rtol=0, atol=1e-12):
        failed.append("alpha = amin + (amax - amin) logistic(a)")
    # special values: a = 0 gives the midpoint, b = 0 gives no phase, c = 0 gives 1/2
    z = np.zeros((1, 4))
    al0, th0, be0, _ = fn(z, z, np.zeros(1), np.ones((1, 4)), AMIN, AMAX, TMAX, eps)
    if not (np.all(al0 == 0.5 * (AMIN + AMAX)) and np.all(th0 == 0.0) and np.all(be0 == 0.5)):
        failed.append("special values at zero")
    # theta: inverse function and bounds
    inner = theta / TMAX
    if not (np.all(np.abs(theta) <= TMAX) and
            np.allclose(np.arctanh(np.clip(inner, -1 + 1e-15, 1 - 1e-15))[np.abs(b) < 5], b[np.abs(b) < 5],
                        rtol=1e-9, atol=1e-9)):
        failed.append("theta = tmax tanh(b)")
    # keys: parallel to the raw keys; unit norm at eps = 0; norm ||k~|| / (||k~|| + eps)
    nr = np.linalg.norm(k_raw, axis=-1)
    _, _, _, k0 = fn(a, b, c, k_raw, AMIN, AMAX, TMAX, 0.0)
    if not np.allclose(np.linalg.norm(k0, axis=-1), 1.0, rtol=0, atol=1e-14):
        failed.append("unit keys at eps = 0")
    if not np.allclose(k0 * nr[:, None], k_raw, rtol=1e-13, atol=1e-13):
        failed.append("keys parallel to the raw keys")
    if not np.allclose(np.linalg.norm(k, axis=-1), nr / (nr + eps), rtol=1e-13, atol=0):
        failed.append("key norm ||k~|| / (||k~|| + eps)")
    # Sec. 3: ||Lambda|| <= 1, 0 <= beta ||k||^2 <= 1, so every transition is a contraction
    bk = beta * np.linalg.norm(k, axis=-1) ** 2
    if not (np.all(alpha <= 1.0) and np.all(alpha >= 0.0) and np.all((bk >= 0) & (bk <= 1))):
        failed.append("bounds of Sec. 3")
    worst = 0.0
    for t in range(a.shape[0]):
        lam = alpha[t] * np.exp(1j * theta[t])
        A = (np.eye(a.shape[1]) - beta[t] * np.outer(k[t], k[t].conj())) @ np.diag(lam)
        worst = max(worst, np.linalg.norm(A, 2))
    if worst > 1.0 + 1e-12:
        failed.append("||A_t||_2 <= 1")
    return failed


def test_gate_map_passes_every_pin():
    assert check_map(G.gates) == []
    assert check_map(G.gates, eps=0.0) == []


def test_sigmoid_has_no_overflow():
    x = np.array([-1000.0, -60.0, -1e-300, 0.0, 1e-300, 60.0, 1000.0])
    s = G.sigmoid(x)
    assert np.all(np.isfinite(s)) and np.allclose(s, expit(x), rtol=0, atol=1e-300)
    assert np.allclose(G.sigmoid(-x), 1.0 - G.sigmoid(x), rtol=0, atol=1e-16)


def test_zero_raw_key_gives_zero_key():
    z = np.zeros((2, 8))
    k_raw = np.zeros((2, 8), dtype=np.complex128)
    for eps in (0.0, 1e-6):
        _, _, _, k = G.gates(z, z, np.zeros(2), k_raw, AMIN, AMAX, TMAX, eps)
        assert np.all(k == 0)


def _mutant(kind):
    def fn(a, b, c, k_raw, amin, amax, tmax, eps):
        alpha, theta, beta, k = G.gates(a, b, c, k_raw, amin, amax, tmax, eps)
        if kind == "span":             # amax instead of (amax - amin)
            alpha = amin + amax * G.sigmoid(a)
        elif kind == "theta_sigmoid":  # sigmoid in place of tanh
            theta = tmax * G.sigmoid(b)
        elif kind == "norm_squared":   # ||k~||^2 in the denominator
            nr2 = np.sum(np.abs(k_raw) ** 2, axis=-1, keepdims=True)
            k = k_raw / (nr2 + eps)
        elif kind == "beta_tanh":      # tanh in place of the logistic function
            beta = np.tanh(c)
        elif kind == "eps_inside":     # eps added under the square root
            nr = np.sqrt(np.sum(np.abs(k_raw) ** 2, axis=-1, keepdims=True) + eps)
            k = k_raw / nr
        return alpha, theta, beta, k
    return fn


@pytest.mark.parametrize("kind", ["span", "theta_sigmoid", "norm_squared", "beta_tanh", "eps_inside"])
def test_planted_mistake_in_gate_map_is_caught(kind):
    assert check_map(_mutant(kind)) != [], f"mutant {kind} passed every pin"
