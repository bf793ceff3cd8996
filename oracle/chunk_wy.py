"""The paper's chunk method on the CPU, float64 -- TEST INFRASTRUCTURE ONLY.

Everything here is plain numpy on one (batch, head) at a time, written from the
paper's statements in their order and notation; it shares nothing with the GPU
library.  Complex conjugate transpose is written ``^*`` as in the paper (App. A:
the identities hold over C with conjugate transpose).

Contents
  phase_decay          Lambda_t = diag(alpha_t * e^{i theta_t})            (Sec. 3, Eq. (sfda))
  transition, write    A_t = (I - beta_t k_t k_t^*) Lambda_t, B_t = beta_t k_t v_t^*   (Def. 3.1)
  wy_vectors           u_t = beta_t k_t, r_t = Lambda_t^* k_t               (Cor. 4.3)
  constructive_wy      left-to-right recursion for (Gamma, Y, W, M)         (Thm 4.2; Alg. 1)
  wy_matrix            Gamma - Y M W^*                                     (Thm 4.2 invariant)
  compose_wy           block-WY closure of two factor tuples                (Thm 4.1)
  zero_state_write     B^chunk via the zero-initial-state recurrence       (Thm 4.4; Alg. 1)
  chunk_summary        the transfer object (Gamma, Y, W, M, B)              (Alg. 1)
  apply_transfer       Gamma S - Y (M (W^* S)) + B                          (eq. (apply-transfer))
  forward_chunked      boundary-state scan with prefix outputs             (Thm 6.1, Thm 4.5)
  ut_chunk / forward_ut  closed forms of the same factors (derived below)
  dense_recurrence     brute force with explicit m x m transition matrices

Closed forms used by ``ut_chunk`` (derived from the Thm 4.2 recursion by induction;
indices are local to a chunk, t, j = 1..C, g_t = lambda_1 * ... * lambda_t elementwise):
  Gamma_t = diag(g_t)
  Y_t[:, j] = diag(g_t / g_j) u_j                  (Lambda_t Y_{t-1} scales old columns)
  W_t[:, j] = Gamma_j^* k_j = diag(conj(g_j)) k_j  (Gamma_{j-1}^* Lambda_j^* k_j)
  M = (I + L' D_beta)^{-1},  L'[t, j] = k_t^* diag(g_t / g_j) k_j for j < t, else 0
      (row t of the M recursion is -r_t^* Y_{t-1} M_{t-1} = -(L' D_beta)[t, :t] M_{t-1})
and, writing delta_t for the row beta_t (v_t^* - k_t^* Lambda_t S_{t-1}) so that
S_t = Lambda_t S_{t-1} + k_t delta_t, with T = D_beta M = (I + D_beta L')^{-1} D_beta:
  Delta = T (conj(V) - (conj(K) * G) S_in)
  O^*   = (conj(Q) * G) S_in + tril(A) Delta,   A[r, j] = q_r^* diag(g_r / g_j) k_j (j <= r)
  S_out = diag(g_C) S_in + (K * (g_C / G))^T Delta
Rows of conj(V), conj(K) * G, ... are tokens; ``*`` between arrays is elementwise.
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import numpy as np


def H(x: np.ndarray) -> np.ndarray:
    """Conjugate transpose (the paper's ^*)."""
    return np.conj(np.swapaxes(x, -1, -2))


# --------------------------------------------------------------------------- Sec. 3

def phase_decay(alpha: np.ndarray, theta: np.ndarray) -> np.ndarray:
    """Diagonal of Lambda_t = diag(alpha_t * e^{i theta_t}) (Eq. (sfda))."""
    return alpha * (np.cos(theta) + 1j * np.sin(theta))


def transition(k: np.ndarray, alpha: np.ndarray, theta: np.ndarray, beta: float) -> np.ndarray:
    """Dense A_t = (I - beta_t k_t k_t^*) Lambda_t (Def. 3.1), m x m."""
    m = k.shape[0]
    kk = np.outer(k, np.conj(k))
    return (np.eye(m) - beta * kk) @ np.diag(phase_decay(alpha, theta))


def write(k: np.ndarray, v: np.ndarray, beta: float) -> np.ndarray:
    """B_t = beta_t k_t v_t^* (Def. 3.1), m x n."""
    return beta * np.outer(k, np.conj(v))


def dense_recurrence(q, k, v, alpha, theta, beta, S0=None):
    """Brute force for one head: S_t = A_t S_{t-1} + B_t, o_t = S_t^* q_t with explicit
    m x m matrices.  q,k: [T,m]; v: [T,n]; returns (o [T,n], S_T [m,n])."""
    T, m = q.shape
    n = v.shape[1]
    S = np.zeros((m, n), complex) if S0 is None else np.array(S0, complex)
    o = np.zeros((T, n), complex)
    for t in range(T):
        S = transition(k[t], alpha[t], theta[t], beta[t]) @ S + write(k[t], v[t], beta[t])
        o[t] = H(S) @ q[t]
    return o, S


# --------------------------------------------------------------------------- Sec. 4

def wy_vectors(k, alpha, theta, beta):
    """u_t = beta_t k_t, r_t = Lambda_t^* k_t, so that A_t = Lambda_t - u_t r_t^* (Cor. 4.3)."""
    lam = phase_decay(alpha, theta)
    return beta * k, np.conj(lam) * k


def constructive_wy(lams: np.ndarray, us: np.ndarray, rs: np.ndarray, prefixes: bool = False):
    """Left-to-right chunk-WY recursion (Thm 4.2), lambdas as diagonals.

    lams, us, rs: [C, m].  Starts from Gamma_0 = I and empty Y, W, M and applies
      Gamma_t = Lambda_t Gamma_{t-1}
      Y_t     = [Lambda_t Y_{t-1}, u_t]
      W_t     = [W_{t-1}, Gamma_{t-1}^* r_t]
      M_t     = [[M_{t-1}, 0], [-r_t^* Y_{t-1} M_{t-1}, 1]]
    Returns (gamma_diag [m], Y [m,C], W [m,C], M [C,C]); with ``prefixes`` a list of the
    tuple after every token.
    """
    C, m = us.shape
    gamma = np.ones(m, complex)
    Y = np.zeros((m, 0), complex)
    W = np.zeros((m, 0), complex)
    M = np.zeros((0, 0), complex)
    out = []
    for t in range(C):
        lam, u, r = lams[t], us[t], rs[t]
        gamma_old, Y_old, W_old, M_old = gamma, Y, W, M
        gamma = lam * gamma_old
        Y = np.concatenate([lam[:, None] * Y_old, u[:, None]], axis=1)
        W = np.concatenate([W_old, (np.conj(gamma_old) * r)[:, None]], axis=1)
        row = -(np.conj(r) @ Y_old) @ M_old
        M = np.zeros((t + 1, t + 1), complex)
        M[:t, :t] = M_old
        M[t, :t] = row
        M[t, t] = 1.0
        if prefixes:
            out.append((gamma, Y, W, M))
    return out if prefixes else (gamma, Y, W, M)


def wy_matrix(gamma: np.ndarray, Y: np.ndarray, W: np.ndarray, M: np.ndarray) -> np.ndarray:
    """P = Gamma - Y M W^* (Thm 4.2 invariant / Cor. 4.3)."""
    return np.diag(gamma) - Y @ M @ H(W)


def compose_wy(t1, t2):
    """Block-WY closure (Thm 4.1): tuple of A_2 A_1 from tuples of A_1 then A_2.
    Each tuple is (Gamma [m,m] dense, Y, W, M)."""
    G1, Y1, W1, M1 = t1
    G2, Y2, W2, M2 = t2
    G21 = G2 @ G1
    Y21 = np.concatenate([G2 @ Y1, Y2], axis=1)
    W21 = np.concatenate([W1, H(G1) @ W2], axis=1)
    r1, r2 = M1.shape[0], M2.shape[0]
    M21 = np.zeros((r1 + r2, r1 + r2), complex)
    M21[:r1, :r1] = M1
    M21[r1:, :r1] = -M2 @ H(W2) @ Y1 @ M1
    M21[r1:, r1:] = M2
    return G21, Y21, W21, M21


def zero_state_write(k, v, alpha, theta, beta, prefixes: bool = False):
    """B^chunk = sum_i A_{C:i+1} B_i computed by the zero-initial-state recurrence
    bar S_0 = 0, bar S_t = A_t bar S_{t-1} + B_t (Thm 4.4; last step of Alg. 1).
    The recurrence is applied in its diagonal-plus-rank-one form A_t = Lambda_t - u_t r_t^*."""
    C, m = k.shape
    n = v.shape[1]
    S = np.zeros((m, n), complex)
    out = []
    for t in range(C):
        lam = phase_decay(alpha[t], theta[t])
        u, r = wy_vectors(k[t], alpha[t], theta[t], beta[t])
        S = lam[:, None] * S - np.outer(u, np.conj(r) @ S) + write(k[t], v[t], beta[t])
        if prefixes:
            out.append(S.copy())
    return out if prefixes else S


def chunk_summary(k, v, alpha, theta, beta):
    """Transfer object (Gamma, Y, W, M, B) of one chunk (Alg. 1)."""
    lams = phase_decay(alpha, theta)
    us, rs = wy_vectors(k, alpha, theta, beta[:, None])
    gamma, Y, W, M = constructive_wy(lams, us, rs)
    return gamma, Y, W, M, zero_state_write(k, v, alpha, theta, beta)


def apply_transfer(tr, S: np.ndarray) -> np.ndarray:
    """S_out = Gamma S - Y (M (W^* S)) + B (eq. (apply-transfer))."""
    gamma, Y, W, M, B = tr
    return gamma[:, None] * S - Y @ (M @ (H(W) @ S)) + B


def forward_chunked(q, k, v, alpha, theta, beta, S0=None, C: int = 16):
    """Boundary-state scan over chunks of C tokens (Thm 6.1), one head.

    Inside a chunk the outputs use the prefix factors (Thm 4.5):
      o_r = S_0^* P_r^* q_r + (B_r)^* q_r,  P_r = Gamma_r - Y_r M_r W_r^*,
    with B_r the zero-state recurrence after r tokens; the boundary state is carried by
    the apply-transfer equation.  A ragged last chunk is simply shorter.
    q,k: [T,m]; v: [T,n]; returns (o [T,n], S_T [m,n])."""
    T, m = q.shape
    n = v.shape[1]
    S = np.zeros((m, n), complex) if S0 is None else np.array(S0, complex)
    o = np.zeros((T, n), complex)
    for c0 in range(0, T, C):
        sl = slice(c0, min(T, c0 + C))
        kc, vc, ac, tc, bc, qc = k[sl], v[sl], alpha[sl], theta[sl], beta[sl], q[sl]
        lams = phase_decay(ac, tc)
        us, rs = wy_vectors(kc, ac, tc, bc[:, None])
        pref = constructive_wy(lams, us, rs, prefixes=True)
        Bpref = zero_state_write(kc, vc, ac, tc, bc, prefixes=True)
        for r, ((gamma, Y, W, M), Br) in enumerate(zip(pref, Bpref)):
            P = wy_matrix(gamma, Y, W, M)
            o[c0 + r] = H(S) @ (H(P) @ qc[r]) + H(Br) @ qc[r]
        gamma, Y, W, M = pref[-1]
        S = apply_transfer((gamma, Y, W, M, Bpref[-1]), S)
    return o, S


# --------------------------------------------------------------------------- closed forms

def ut_chunk(q, k, v, alpha, theta, beta, S):
    """One chunk through the closed forms in the module docstring.
    Returns (o [C,n], S_out [m,n], parts) where parts holds G, L', A, T, Delta."""
    C = k.shape[0]
    lam = phase_decay(alpha, theta)                 # [C, m]
    G = np.cumprod(lam, axis=0)                     # g_t
    ratio = G[:, None, :] / G[None, :, :]           # g_t / g_j   [t, j, m]
    Kst = np.einsum("ti,tji,ji->tj", np.conj(k), ratio, k)
    Lp = np.tril(Kst, -1)
    A = np.tril(np.einsum("ri,rji,ji->rj", np.conj(q), ratio, k))
    Db = np.diag(beta.astype(complex))
    Tm = np.linalg.solve(np.eye(C) + Db @ Lp, Db)
    Delta = Tm @ (np.conj(v) - (np.conj(k) * G) @ S)
    OH = (np.conj(q) * G) @ S + A @ Delta
    S_out = G[-1][:, None] * S + (k * (G[-1][None, :] / G)).T @ Delta
    return np.conj(OH), S_out, dict(G=G, L=Lp, A=A, T=Tm, Delta=Delta)


def forward_ut(q, k, v, alpha, theta, beta, S0=None, C: int = 16):
    """Chunked forward through ``ut_chunk`` (one head); ragged last chunk allowed."""
    T, m = q.shape
    n = v.shape[1]
    S = np.zeros((m, n), complex) if S0 is None else np.array(S0, complex)
    o = np.zeros((T, n), complex)
    for c0 in range(0, T, C):
        sl = slice(c0, min(T, c0 + C))
        oc, S, _ = ut_chunk(q[sl], k[sl], v[sl], alpha[sl], theta[sl], beta[sl], S)
        o[sl] = oc
    return o, S
