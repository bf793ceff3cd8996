"""Checks that pin a one-head SFDA recurrence to what the paper and the mathematics fix.

Each ``pin_*`` takes ``rec(q, k, v, alpha, theta, beta, S0) -> (o [T,n], S_T [m,n])`` for a
single head (q,k: [T,m] complex; v: [T,n] complex; alpha,theta: [T,m]; beta: [T]) and
raises AssertionError when the recurrence violates the fixed property.  They run on the
oracle (where they must pass) and on deliberately broken recurrences (where at least one
must fail), which shows the set is sharp enough to catch a plausible slip.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

from oracle import chunk_wy as cw

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def cn(rng, shape):
    return (rng.standard_normal(shape) + 1j * rng.standard_normal(shape)) / math.sqrt(2)


def unit_keys(rng, T, m):
    k = cn(rng, (T, m))
    return k / np.linalg.norm(k, axis=1, keepdims=True)


def random_head(seed, T, m, n, alpha=(0.8, 1.0), s0=True):
    rng = _rng(seed)
    q = cn(rng, (T, m))
    k = unit_keys(rng, T, m)
    v = cn(rng, (T, n))
    a = rng.uniform(alpha[0], alpha[1], (T, m))
    th = rng.uniform(-math.pi, math.pi, (T, m))
    b = rng.uniform(0, 1, T)
    S0 = cn(rng, (m, n)) if s0 else None
    return q, k, v, a, th, b, S0


def rel(x, ref):
    return float(np.max(np.abs(x - ref)) / max(np.max(np.abs(ref)), 1e-300))


# --------------------------------------------------------------------------- golden

def pin_hand_examples(rec):
    """Hand-derived tiny cases (tests/golden/hand_examples.json; Sec. 3 Eq. (sfda))."""
    with open(os.path.join(GOLDEN, "hand_examples.json")) as f:
        g = json.load(f)

    def cx(a):
        a = np.asarray(a, float)
        return a[..., 0] + 1j * a[..., 1]

    for ex in g["examples"]:
        toks = ex["tokens"]
        q = np.stack([cx(t["q"]) for t in toks])
        k = np.stack([cx(t["k"]) for t in toks])
        v = np.stack([cx(t["v"]) for t in toks])
        a = np.array([t["alpha"] for t in toks], float)
        th = np.array([t["theta"] for t in toks], float)
        b = np.array([t["beta"] for t in toks], float)
        S0 = cx(ex["S0"])
        o, S = rec(q, k, v, a, th, b, S0)
        assert np.max(np.abs(o - cx(ex["o"]))) < 1e-14, (ex["name"], o)
        assert np.max(np.abs(S - cx(ex["S_T"]))) < 1e-14, (ex["name"], S)


# --------------------------------------------------------------------------- definition

def pin_definition_dense(rec, seeds=(1, 2, 3)):
    """P-def: per-token dense transition A_t S + B_t and readout S^* q (Def. 3.1)."""
    for s in seeds:
        q, k, v, a, th, b, S0 = random_head(s, 24, 6, 4)
        o, S = rec(q, k, v, a, th, b, S0)
        o2, S2 = cw.dense_recurrence(q, k, v, a, th, b, S0)
        assert rel(o, o2) < 1e-13 and rel(S, S2) < 1e-13


def pin_delta_retrieval(rec):
    """With beta = 1 and |k| = 1 the erase clears the k direction and the write stores v, so
    k^* S_t = v_t^* and querying with the same key returns the value: o_t = S_t^* k_t = v_t
    (Sec. 3: the delta rule inside Eq. (sfda))."""
    q, k, v, a, th, b, S0 = random_head(11, 32, 8, 5)
    b = np.ones_like(b)
    o, S = rec(k.copy(), k, v, a, th, b, S0)
    assert np.max(np.abs(o - v)) < 1e-13
    assert np.max(np.abs(np.conj(k[-1]) @ S - np.conj(v[-1]))) < 1e-13


def pin_beta_zero_closed_form(rec, T=4096):
    """P-beta0: beta = 0 gives S_t = Lambda_t S_{t-1} (Prop. 2.1), so
    S_T = diag(prod_t alpha_t e^{i theta_t}) S_0 = diag(exp(sum log alpha + i sum theta)) S_0
    and o_t = S_t^* q_t (App. C.6, stage 1)."""
    q, k, v, a, th, b, S0 = random_head(5, T, 6, 3, alpha=(0.999, 1.0))
    th = th * 0.3
    b = np.zeros(T)
    o, S = rec(q, k, v, a, th, b, S0)
    la = np.cumsum(np.log(a), axis=0)
    ph = np.cumsum(th, axis=0)
    G = np.exp(la + 1j * ph)                                   # [T, m]
    S_ref = G[-1][:, None] * S0
    o_ref = np.einsum("tij,ti->tj", np.conj(G[:, :, None] * S0[None]), q)
    assert rel(S, S_ref) < 1e-12, rel(S, S_ref)
    assert rel(o, o_ref) < 1e-12, rel(o, o_ref)


def kda_real(q, k, v, alpha, beta, S0):
    """Kimi Delta Attention over the reals (Eq. (1) of the introduction):
    S_t = (I - beta_t k_t k_t^T) diag(alpha_t) S_{t-1} + beta_t k_t v_t^T,  o_t = S_t^T q_t.
    Written independently with explicit real matrices."""
    T, m = q.shape
    S = np.array(S0, float)
    o = np.zeros((T, v.shape[1]))
    for t in range(T):
        E = np.eye(m) - beta[t] * np.outer(k[t], k[t])
        S = E @ (np.diag(alpha[t]) @ S) + beta[t] * np.outer(k[t], v[t])
        o[t] = S.T @ q[t]
    return o, S


def pin_kda(rec, golden=None):
    """P-KDA: theta = 0 with real q, k, v, S0 reduces exactly to KDA (Prop. 3.2;
    Table 8 prints error 0)."""
    rng = _rng(7)
    T, m, n = 40, 6, 4
    q = rng.standard_normal((T, m))
    k = rng.standard_normal((T, m))
    k /= np.linalg.norm(k, axis=1, keepdims=True)
    v = rng.standard_normal((T, n))
    a = rng.uniform(0.7, 1.0, (T, m))
    b = rng.uniform(0, 1, T)
    S0 = rng.standard_normal((m, n))
    o, S = rec(q + 0j, k + 0j, v + 0j, a, np.zeros((T, m)), b, S0 + 0j)
    o2, S2 = kda_real(q, k, v, a, b, S0)
    assert np.max(np.abs(o.imag)) == 0.0 and np.max(np.abs(S.imag)) == 0.0
    assert rel(o.real, o2) < 1e-13 and rel(S.real, S2) < 1e-13


def pin_cyclic(rec, golden):
    """P-cyc: beta = 0, alpha = 1, theta_t = 2 pi a_t / 5 is an exact mod-5 counter with
    |z_T| = |z_0| (Prop. 3.4); the paper prints norm drift 3.0e-14 and modular error
    3.0e-12 at T = 16384 (Table 8)."""
    T, mod = golden["cyclic_T"], golden["cyclic_modulus"]
    rng = _rng(9)
    m, n = 4, 2
    steps = rng.integers(0, mod, (T, m))
    th = 2 * math.pi * steps / mod
    q, k, v = cn(rng, (T, m)), unit_keys(rng, T, m), cn(rng, (T, n))
    S0 = cn(rng, (m, n))
    o, S = rec(q, k, v, np.ones((T, m)), th, np.zeros(T), S0)
    drift = np.max(np.abs(np.abs(S) - np.abs(S0)))
    assert drift <= 10 * golden["cyclic_norm_drift_T16384"], drift
    count = np.sum(steps, axis=0) % mod
    z_ref = np.exp(2j * math.pi * count / mod)[:, None] * S0
    assert np.max(np.abs(S - z_ref)) <= 10 * golden["cyclic_modular_error_T16384"]


def pin_register(rec):
    """P-reg: alpha = 1, theta = 0, beta = 1, k = e_i overwrites row i of S with v^* and
    leaves the other rows untouched (Thm 5.9, register memory).  The untouched rows are
    compared bitwise; row i is S_i + (v^* - S_i) in floating point, so it is checked to
    within a few units in the last place."""
    rng = _rng(13)
    m, n, T = 5, 3, 12
    S0 = cn(rng, (m, n))
    S = S0.copy()
    for t in range(T):
        i = int(rng.integers(0, m))
        k = np.zeros((1, m), complex)
        k[0, i] = 1.0
        v = cn(rng, (1, n))
        q = cn(rng, (1, m))
        _, S_new = rec(q, k, v, np.ones((1, m)), np.zeros((1, m)), np.ones(1), S)
        others = [r for r in range(m) if r != i]
        assert np.array_equal(S_new[others], S[others]), (t, i)
        assert np.max(np.abs(S_new[i] - np.conj(v[0]))) <= 4e-16 * max(1.0, np.max(np.abs(S))), (t, i)
        S = S_new


def pin_projector():
    """P-proj: k_i = e_i, beta = 1, Lambda = I for i = 1..r gives the product
    I - sum_i e_i e_i^T (Prop. 5.4 example), through the dense transition."""
    m, r = 7, 4
    P = np.eye(m, dtype=complex)
    for i in range(r):
        k = np.zeros(m, complex)
        k[i] = 1.0
        P = cw.transition(k, np.ones(m), np.zeros(m), 1.0) @ P
    ref = np.eye(m)
    ref[:r, :r] = 0
    assert np.array_equal(P, ref)


def pin_associativity(rec):
    """P-assoc: running T1 tokens, then T2 tokens from the resulting state, equals running
    T1 + T2 tokens (Cor. A.3, chunk parenthesisation) -- bitwise for a recurrence."""
    q, k, v, a, th, b, S0 = random_head(17, 50, 5, 3)
    o, S = rec(q, k, v, a, th, b, S0)
    o1, S1 = rec(q[:21], k[:21], v[:21], a[:21], th[:21], b[:21], S0)
    o2, S2 = rec(q[21:], k[21:], v[21:], a[21:], th[21:], b[21:], S1)
    assert np.array_equal(np.concatenate([o1, o2]), o) and np.array_equal(S2, S)


def pin_linearity(rec):
    """P-lin: for fixed (q, k, alpha, theta, beta), S_T is linear in S0 and conjugate-linear
    in v; o is conjugate-linear in S0 and linear in v (Eq. (sfda) with v^* the conjugate
    transpose and o = S^* q)."""
    q, k, v, a, th, b, S0 = random_head(19, 30, 5, 3)
    rng = _rng(20)
    c = complex(0.3, -1.7)
    v2, S02 = cn(rng, v.shape), cn(rng, S0.shape)
    zero_v, zero_S = np.zeros_like(v), np.zeros_like(S0)
    # state part: S_T(S0, v=0) linear in S0
    _, Sa = rec(q, k, zero_v, a, th, b, S0)
    _, Sb = rec(q, k, zero_v, a, th, b, S02)
    oc, Sc = rec(q, k, zero_v, a, th, b, c * S0 + S02)
    assert rel(Sc, c * Sa + Sb) < 1e-13
    # value part: S_T(S0=0, v) conjugate-linear in v, o linear in v
    oa, Sva = rec(q, k, v, a, th, b, zero_S)
    ob, Svb = rec(q, k, v2, a, th, b, zero_S)
    od, Svd = rec(q, k, c * v + v2, a, th, b, zero_S)
    assert rel(Svd, np.conj(c) * Sva + Svb) < 1e-13
    assert rel(od, c * oa + ob) < 1e-13
    # o conjugate-linear in S0 (v = 0)
    o1, _ = rec(q, k, zero_v, a, th, b, S0)
    o2, _ = rec(q, k, zero_v, a, th, b, S02)
    assert rel(oc, np.conj(c) * o1 + o2) < 1e-13


def pin_padding(rec):
    """P-pad: identity tokens (k = 0, beta = 0, alpha = 1, theta = 0) leave S unchanged,
    since then A_t = I and B_t = 0 (Def. 3.1) -- bitwise."""
    q, k, v, a, th, b, S0 = random_head(23, 6, 4, 3)
    T = 6
    _, S = rec(q, np.zeros_like(k), v, np.ones((T, 4)), np.zeros((T, 4)), np.zeros(T), S0)
    assert np.array_equal(S, S0)


def pin_stability(rec):
    """P-stab: ||A_t||_2 <= 1 when |lambda| <= 1 and 0 <= beta ||k||^2 <= 2 (Prop. 6.3;
    Table 8: max 0.9977 over samples), and ||S_t||_F <= ||S_0||_F + sum_i ||B_i||_F
    along a trajectory."""
    rng = _rng(29)
    m = 8
    worst = 0.0
    for _ in range(2000):
        k = cn(rng, (m,))
        k *= rng.uniform(0, 1) / np.linalg.norm(k)
        A = cw.transition(k, rng.uniform(0, 1, m), rng.uniform(-math.pi, math.pi, m),
                          rng.uniform(0, 1))
        worst = max(worst, np.linalg.norm(A, 2))
    assert worst <= 1.0 + 1e-12, worst
    q, k, v, a, th, b, S0 = random_head(31, 64, 6, 4, alpha=(0.5, 1.0))
    S = S0
    bound = np.linalg.norm(S0)
    for t in range(64):
        _, S = rec(q[t:t + 1], k[t:t + 1], v[t:t + 1], a[t:t + 1], th[t:t + 1], b[t:t + 1], S)
        bound += np.linalg.norm(cw.write(k[t], v[t], b[t]))
        assert np.linalg.norm(S) <= bound * (1 + 1e-12)


def pin_chunk_invariance(rec, Cs=(1, 2, 3, 5, 8, 16, 32, 64), tol=1e-10):
    """P-C: the boundary-state scan with any chunk size reproduces the recurrent states
    and outputs (Thm 6.1 with Thm 4.5), including a ragged last chunk."""
    for C in Cs:
        for T in (2 * C, 2 * C + max(1, C // 3)):
            q, k, v, a, th, b, S0 = random_head(100 + C + T, T, 8, 4)
            o, S = rec(q, k, v, a, th, b, S0)
            o2, S2 = cw.forward_chunked(q, k, v, a, th, b, S0, C)
            assert rel(o2, o) < tol and rel(S2, S) < tol, (C, T, rel(o2, o), rel(S2, S))


def all_recurrence_pins(golden):
    return [
        ("hand", pin_hand_examples),
        ("def", pin_definition_dense),
        ("retrieval", pin_delta_retrieval),
        ("beta0", pin_beta_zero_closed_form),
        ("kda", pin_kda),
        ("cyclic", lambda r: pin_cyclic(r, golden)),
        ("register", pin_register),
        ("assoc", pin_associativity),
        ("linearity", pin_linearity),
        ("padding", pin_padding),
        ("stability", pin_stability),
        ("chunkC", lambda r: pin_chunk_invariance(r, Cs=(1, 3, 8, 16))),
    ]
