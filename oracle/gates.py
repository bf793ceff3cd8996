"""The paper's stable parameterization of the gates and keys -- TEST INFRASTRUCTURE ONLY.

Sec. 3 ("Stable parameterization", equations param-alpha, param-theta, param-beta and
param-key) maps unconstrained per-token projections to the recurrence's parameters:

    alpha_t = alpha_min + (alpha_max - alpha_min) * sigmoid(a_t)   (per channel)
    theta_t = theta_max * tanh(b_t)                                  (per channel)
    beta_t  = sigmoid(c_t)                                           (per token)
    k_t     = k~_t / (||k~_t||_2 + eps)                              (norm over the m
                                                                      complex channels)

so that ||Lambda_t||_2 <= 1, 0 <= beta_t <= 1 and ||k_t||_2 <= 1.  Plain float64 numpy;
the gated forward is this map followed by the oracle recurrence.
"""
from __future__ import annotations

import numpy as np


def sigmoid(x):
    """1 / (1 + e^-x), written so neither branch overflows."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def gates(a, b, c, k_raw, alpha_min: float, alpha_max: float, theta_max: float, eps: float):
    """(alpha, theta, beta, k) from the pre-activations a, b [..., m], c [...] and the raw
    complex keys k_raw [..., m] (Sec. 3, stable parameterization)."""
    alpha = alpha_min + (alpha_max - alpha_min) * sigmoid(a)
    theta = theta_max * np.tanh(np.asarray(b, dtype=np.float64))
    beta = sigmoid(c)
    k_raw = np.asarray(k_raw, dtype=np.complex128)
    norm = np.sqrt(np.sum(np.abs(k_raw) ** 2, axis=-1, keepdims=True))
    den = norm + eps
    k = np.divide(k_raw, den, out=np.zeros_like(k_raw), where=den > 0)
    return alpha, theta, beta, k
