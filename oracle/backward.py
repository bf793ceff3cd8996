"""Reverse-mode gradients of the SFDA forward -- TEST INFRASTRUCTURE ONLY.

The forward is the token recurrence of Sec. 3, Eq. (sfda), with the readout after the
update:

    lambda_t = alpha_t * exp(i theta_t)                  (per channel)
    S'_t     = diag(lambda_t) S_{t-1}
    D_t      = conj(v_t)^T - k_t^* S'_t                  (row of n values)
    S_t      = S'_t + beta_t k_t D_t                     (= (I - beta k k^*) Lambda S + beta k v^*)
    o_t      = S_t^* q_t

For a real scalar loss L with upstream gradients dO = dL/do and dS_T = dL/dS_T, this
module returns dL/dq, dL/dk, dL/dv, dL/dalpha, dL/dtheta, dL/dbeta and dL/dS0.  The
gradient of a complex variable z = x + i y is dL/dx + i dL/dy (so that a first-order
change of L is Re(sum conj(dz) * delta z)); real variables get the ordinary derivative.

Derivation (the adjoint of each line above, taken in reverse; Gs is dL/dS_t):
  from o_t:   Gs += q_t dO_t^*,            dq_t = S_t dO_t
  from S_t:   u = Gs^* k_t  (n values),    dv_t = beta_t u,
              dbeta_t = Re(sum_c u_c D_c), dk_t = beta_t (Gs conj(D_t) - S'_t u),
              G' = Gs - beta_t k_t (k_t^* Gs)   (the adjoint of I - beta k k^*)
  from S'_t:  g_i = sum_c G'_ic conj(S_{t-1,ic}),
              dalpha_t = Re(conj(g) e^{i theta_t}), dtheta_t = Re(conj(g) i lambda_t),
              Gs <- diag(conj(lambda_t)) G'
and dS0 is Gs after the first token.  Plain float64 / complex128 numpy, one token at a
time, vectorised over the (b, h) heads only; every state S_{t-1} is kept from a forward
sweep, so memory grows as T m n per head (call per head for long sequences).

Pinned in tests/test_oracle_backward.py by central finite differences of the C oracle's
forward, by Euler's identity for the parts of the forward that are homogeneous of degree
one, and by planted mistakes that those checks must catch.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def forward_states(q, k, v, alpha, theta, beta, S0: Optional[np.ndarray] = None):
    """The recurrence with every state kept.  Shapes as in oracle.recurrence.
    Returns (o [B,H,T,n], states [T+1, B,H,m,n] with states[t] = S_t, states[0] = S0)."""
    q = np.asarray(q, dtype=np.complex128)
    k = np.asarray(k, dtype=np.complex128)
    v = np.asarray(v, dtype=np.complex128)
    alpha = np.asarray(alpha, dtype=np.float64)
    theta = np.asarray(theta, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    B, H, T, m = q.shape
    n = v.shape[-1]
    S = np.zeros((B, H, m, n), np.complex128) if S0 is None else np.array(S0, dtype=np.complex128)
    states = np.empty((T + 1, B, H, m, n), np.complex128)
    states[0] = S
    o = np.empty((B, H, T, n), np.complex128)
    for t in range(T):
        lam = alpha[:, :, t] * np.exp(1j * theta[:, :, t])          # [B,H,m]
        Sp = lam[..., None] * S
        kt = k[:, :, t]
        D = np.conj(v[:, :, t]) - np.einsum("bhi,bhic->bhc", np.conj(kt), Sp)
        S = Sp + beta[:, :, t, None, None] * kt[..., None] * D[:, :, None, :]
        states[t + 1] = S
        o[:, :, t] = np.einsum("bhic,bhi->bhc", np.conj(S), q[:, :, t])
    return o, states


def recurrence_backward(q, k, v, alpha, theta, beta, S0, dO, dS_T=None):
    """Gradients of L with dL/do = dO [B,H,T,n] and dL/dS_T = dS_T [B,H,m,n] (None = 0).

    Returns a dict with dq, dk [B,H,T,m] complex; dv [B,H,T,n] complex; dalpha, dtheta
    [B,H,T,m] real; dbeta [B,H,T] real; dS0 [B,H,m,n] complex (the gradient with respect
    to the initial state, also when S0 is None = the zero state)."""
    q = np.asarray(q, dtype=np.complex128)
    k = np.asarray(k, dtype=np.complex128)
    v = np.asarray(v, dtype=np.complex128)
    alpha = np.asarray(alpha, dtype=np.float64)
    theta = np.asarray(theta, dtype=np.float64)
    beta = np.asarray(beta, dtype=np.float64)
    dO = np.asarray(dO, dtype=np.complex128)
    B, H, T, m = q.shape
    n = v.shape[-1]
    _, states = forward_states(q, k, v, alpha, theta, beta, S0)

    dq = np.zeros((B, H, T, m), np.complex128)
    dk = np.zeros((B, H, T, m), np.complex128)
    dv = np.zeros((B, H, T, n), np.complex128)
    dalpha = np.zeros((B, H, T, m))
    dtheta = np.zeros((B, H, T, m))
    dbeta = np.zeros((B, H, T))
    Gs = np.zeros((B, H, m, n), np.complex128) if dS_T is None else np.array(dS_T, dtype=np.complex128)

    for t in range(T - 1, -1, -1):
        S_prev, S_t = states[t], states[t + 1]
        qt, kt = q[:, :, t], k[:, :, t]
        bt = beta[:, :, t]
        lam = alpha[:, :, t] * np.exp(1j * theta[:, :, t])
        Sp = lam[..., None] * S_prev
        D = np.conj(v[:, :, t]) - np.einsum("bhi,bhic->bhc", np.conj(kt), Sp)
        # readout o_t = S_t^* q_t
        dq[:, :, t] = np.einsum("bhic,bhc->bhi", S_t, dO[:, :, t])
        Gs = Gs + qt[..., None] * np.conj(dO[:, :, t])[:, :, None, :]
        # erase and write S_t = S' + beta k D
        u = np.einsum("bhic,bhi->bhc", np.conj(Gs), kt)
        dv[:, :, t] = bt[..., None] * u
        dbeta[:, :, t] = np.real(np.sum(u * D, axis=-1))
        dk[:, :, t] = bt[..., None] * (np.einsum("bhic,bhc->bhi", Gs, np.conj(D)) -
                                       np.einsum("bhic,bhc->bhi", Sp, u))
        Gp = Gs - bt[..., None, None] * kt[..., None] * np.conj(u)[:, :, None, :]
        # phase-decay S' = diag(lambda) S_{t-1}
        g = np.sum(Gp * np.conj(S_prev), axis=-1)
        dalpha[:, :, t] = np.real(np.conj(g) * np.exp(1j * theta[:, :, t]))
        dtheta[:, :, t] = np.real(np.conj(g) * 1j * lam)
        Gs = np.conj(lam)[..., None] * Gp
    return dict(dq=dq, dk=dk, dv=dv, dalpha=dalpha, dtheta=dtheta, dbeta=dbeta, dS0=Gs)


def loss(o, S_T, dO, dS_T=None) -> float:
    """The real scalar L = Re sum conj(dO) o + Re sum conj(dS_T) S_T whose gradients
    recurrence_backward returns (dL/do = dO, dL/dS_T = dS_T)."""
    val = float(np.real(np.sum(np.conj(dO) * o)))
    if dS_T is not None:
        val += float(np.real(np.sum(np.conj(dS_T) * S_T)))
    return val
