"""The write-decoupled SFDA recurrence -- TEST INFRASTRUCTURE ONLY.

Sec. 3 (write-decoupled variant, eq. sfda-decoupled-main) separates the erase direction
from the write direction:

    S_t = (I - eta_t k_t k_t^*) Lambda_t S_{t-1} + beta_t r_t v_t^*,   o_t = S_t^* q_t

with Lambda_t = diag(alpha_t e^{i theta_t}) as in the tied model, an erase strength eta_t
and a write strength beta_t (scalars per token) and a write direction r_t in C^m.  Setting
r_t = k_t and eta_t = beta_t recovers tied SFDA.  Plain complex128 numpy, one token at a
time, vectorised over the (b, h) heads; the update is applied in the order the definition
reads (phase-decay, erase, write), the readout after it.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def decoupled_recurrence(q, k, r, v, alpha, theta, eta, beta, S0: Optional[np.ndarray] = None):
    """q, k, r: [B,H,T,m] complex; v: [B,H,T,n] complex; alpha, theta: [B,H,T,m] real;
    eta, beta: [B,H,T] real; S0: [B,H,m,n] complex or None (zero state).
    Returns (o [B,H,T,n], S_T [B,H,m,n]), complex128."""
    q = np.asarray(q, dtype=np.complex128)
    k = np.asarray(k, dtype=np.complex128)
    r = np.asarray(r, dtype=np.complex128)
    v = np.asarray(v, dtype=np.complex128)
    alpha = np.asarray(alpha, dtype=np.float64)
    theta = np.asarray(theta, dtype=np.float64)
    eta = np.asarray(eta, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    B, H, T, m = q.shape
    n = v.shape[-1]
    S = np.zeros((B, H, m, n), np.complex128) if S0 is None else np.array(S0, dtype=np.complex128)
    o = np.empty((B, H, T, n), np.complex128)
    for t in range(T):
        lam = alpha[:, :, t] * (np.cos(theta[:, :, t]) + 1j * np.sin(theta[:, :, t]))
        S = lam[..., None] * S                                                  # Lambda_t S
        kt = k[:, :, t]
        x = np.einsum("bhi,bhic->bhc", np.conj(kt), S)                          # k^* Lambda S
        S = S - eta[:, :, t, None, None] * kt[..., None] * x[:, :, None, :]      # erase along k
        S = S + beta[:, :, t, None, None] * r[:, :, t][..., None] * np.conj(v[:, :, t])[:, :, None, :]
        o[:, :, t] = np.einsum("bhic,bhi->bhc", np.conj(S), q[:, :, t])        # S_t^* q_t
    return o, S
