"""Componentwise error scales for the bfloat16 backward (tolerances only, no expected values).

A matrix product that rounds its operands to bfloat16 (unit roundoff u = 2^-9) and
accumulates in float32 returns each entry of a sum of products with an error bounded by a
small multiple of u times the sum of the ABSOLUTE values of the products, not of the sum
itself.  Where the sum cancels, the result can be much smaller than its terms.  Three of the
gradients pass through the adjoint of the erase I - beta k k^*:

    G' = G - beta k (k^* G)            (G = dL/dS_t after the readout term)
    dS0 = conj(lambda_1) G'             (at the first token)
    dalpha_t, dtheta_t from g_i = sum_c G'_ic conj(S_{t-1, ic})

and with beta |k|^2 near 1 (exact when m = 1: the erase is the scalar 1 - beta |k|^2) they
are much smaller than the terms they are formed from.  erase_term_scales returns, element
by element, the sum of the absolute values of those terms, computed from the exact
intermediates of the oracle's own forward states:

    |G'| <= |G| + beta |k| (|k|^T |G|)           elementwise
    scale(dS0)_ic        = alpha_1i |G'|_ic       (first token)
    scale(dalpha)_t,i    = sum_c |G'|_ic |S_{t-1}|_ic
    scale(dtheta)_t,i    = alpha_t,i * scale(dalpha)_t,i

Each is an upper bound of |the exact gradient| (the triangle inequality), with equality for
dS0 when beta = 0 and for |g| when n = 1 and beta = 0.
"""
from __future__ import annotations

import numpy as np

from oracle import backward as BW

U_BF16 = 2.0 ** -9


def erase_term_scales(q, k, v, alpha, theta, beta, S0, dO, dS_T):
    """Shapes as in oracle.backward.recurrence_backward.  Returns a dict with the
    componentwise scales of dS0 [B,H,m,n], dalpha and dtheta [B,H,T,m] (real, >= 0)."""
    q = np.asarray(q, np.complex128)
    k = np.asarray(k, np.complex128)
    alpha = np.asarray(alpha, np.float64)
    theta = np.asarray(theta, np.float64)
    beta = np.asarray(beta, np.float64)
    dO = np.asarray(dO, np.complex128)
    B, H, T, m = q.shape
    _, states = BW.forward_states(q, k, v, alpha, theta, beta, S0)
    n = states.shape[-1]
    G = np.zeros((B, H, m, n), np.complex128) if dS_T is None else np.array(dS_T, np.complex128)
    s_alpha = np.zeros((B, H, T, m))
    s_S0 = np.zeros((B, H, m, n))
    for t in range(T - 1, -1, -1):
        kt, bt = k[:, :, t], beta[:, :, t]
        G = G + q[:, :, t][..., None] * np.conj(dO[:, :, t])[:, :, None, :]
        akG = np.einsum("bhi,bhic->bhc", np.abs(kt), np.abs(G))
        Gp_abs = np.abs(G) + bt[..., None, None] * np.abs(kt)[..., None] * akG[:, :, None, :]
        s_alpha[:, :, t] = np.sum(Gp_abs * np.abs(states[t]), axis=-1)
        s_S0 = alpha[:, :, t][..., None] * Gp_abs
        u = np.einsum("bhic,bhi->bhc", np.conj(G), kt)
        Gp = G - bt[..., None, None] * kt[..., None] * np.conj(u)[:, :, None, :]
        G = np.conj(alpha[:, :, t] * np.exp(1j * theta[:, :, t]))[..., None] * Gp
    return dict(dS0=s_S0, dalpha=s_alpha, dtheta=alpha * s_alpha)


def bf16_gradient_bound(name: str, ref: np.ndarray, scales: dict, tol: float = 2e-2) -> float:
    """Largest admissible max |x - ref| for a bfloat16 gradient: tol * max |ref|, widened for
    dS0, dalpha and dtheta to 8 u * max(scale) -- each term reaches them through at most
    four bfloat16 matrix products (conj(Y') G, N^* G_Delta, (conj(K) G)^* G_E and the
    state-times-adjoint product), each rounding two operands."""
    bound = tol * float(np.max(np.abs(ref))) if ref.size else 0.0
    if name in scales:
        bound = max(bound, 8 * U_BF16 * float(np.max(scales[name])))
    return bound
