"""The oracle against what the paper and the mathematics fix (CPU only).

Pins for the token recurrence (C oracle) and for the chunk method (numpy, float64):
constructive chunk-WY identity (Thm 4.2), block-WY closure (Thm 4.1), affine transfer
(Thm 4.4), closed-form factors, rank budget (Thm 5.3), chunk-size invariance (Thm 6.1).
Planted mistakes in a CPU copy of the recurrence must each fail at least one pin.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import chunk_wy as cw
import oracle_pins as P

GOLD = json.load(open(os.path.join(P.GOLDEN, "paper_residuals.json")))


def rec_c(q, k, v, a, th, b, S0):
    o, S = oracle.recurrence(q[None, None], k[None, None], v[None, None], a[None, None],
                             th[None, None], b[None, None],
                             None if S0 is None else np.asarray(S0)[None, None])
    return o[0, 0], S[0, 0]


@pytest.mark.parametrize("name,pin", P.all_recurrence_pins(GOLD), ids=lambda x: x if isinstance(x, str) else "")
def test_oracle_recurrence_pins(name, pin):
    pin(rec_c)


def test_projector_example():
    P.pin_projector()


def test_batched_heads_match_single_heads():
    """Heads are independent: the batched call equals per-head calls (bitwise)."""
    rng = np.random.default_rng(3)
    B, Hh, T, m, n = 2, 3, 20, 5, 4
    q, k, v = P.cn(rng, (B, Hh, T, m)), P.cn(rng, (B, Hh, T, m)), P.cn(rng, (B, Hh, T, n))
    a, th, b = rng.uniform(.8, 1, (B, Hh, T, m)), rng.uniform(-3, 3, (B, Hh, T, m)), rng.uniform(0, 1, (B, Hh, T))
    S0 = P.cn(rng, (B, Hh, m, n))
    o, S = oracle.recurrence(q, k, v, a, th, b, S0)
    for bb in range(B):
        for hh in range(Hh):
            o1, S1 = rec_c(q[bb, hh], k[bb, hh], v[bb, hh], a[bb, hh], th[bb, hh], b[bb, hh], S0[bb, hh])
            assert np.array_equal(o1, o[bb, hh]) and np.array_equal(S1, S[bb, hh])


def test_step_equals_one_token_recurrence():
    rng = np.random.default_rng(4)
    B, Hh, m, n = 2, 2, 6, 5
    q, k, v = P.cn(rng, (B, Hh, m)), P.cn(rng, (B, Hh, m)), P.cn(rng, (B, Hh, n))
    a, th, b = rng.uniform(.8, 1, (B, Hh, m)), rng.uniform(-3, 3, (B, Hh, m)), rng.uniform(0, 1, (B, Hh))
    S = P.cn(rng, (B, Hh, m, n))
    o, S1 = oracle.step(q, k, v, a, th, b, S)
    o2, S2 = oracle.recurrence(q[:, :, None], k[:, :, None], v[:, :, None], a[:, :, None],
                               th[:, :, None], b[:, :, None], S)
    assert np.array_equal(o, o2[:, :, 0]) and np.array_equal(S1, S2)


# --------------------------------------------------------------------------- planted mistakes

def rec_mutant(kind):
    """A plain numpy recurrence with one deliberate slip (CPU only)."""
    def rec(q, k, v, a, th, b, S0):
        T, m = q.shape
        n = v.shape[1]
        S = np.zeros((m, n), complex) if S0 is None else np.array(S0, complex)
        o = np.zeros((T, n), complex)
        for t in range(T):
            lam = a[t] * np.exp(1j * th[t])
            if kind == "conj_lambda":
                lam = np.conj(lam)
            vv = v[t] if kind == "no_conj_v" else np.conj(v[t])
            kh = k[t] if kind == "k_transpose" else np.conj(k[t])
            S_prev = S
            if kind == "erase_before_decay":
                S = S - b[t] * np.outer(k[t], kh @ S)
                S = lam[:, None] * S + b[t] * np.outer(k[t], vv)
            else:
                S = lam[:, None] * S
                beta_e = 1.0 if kind == "no_beta_erase" else b[t]
                S = S - beta_e * np.outer(k[t], kh @ S) + b[t] * np.outer(k[t], vv)
            if kind == "readout_before_update":
                o[t] = np.conj(S_prev).T @ q[t]
            elif kind == "readout_no_conj":
                o[t] = S.T @ q[t]
            elif kind == "readout_swapped":
                o[t] = np.conj(S.T @ np.conj(q[t]))
            else:
                o[t] = np.conj(S).T @ q[t]
        return o, S
    return rec


MUTANTS = ["conj_lambda", "no_conj_v", "k_transpose", "erase_before_decay",
           "no_beta_erase", "readout_before_update", "readout_no_conj"]


def test_unmutated_numpy_recurrence_passes():
    rec = rec_mutant("none")
    for name, pin in P.all_recurrence_pins(GOLD):
        pin(rec)


@pytest.mark.parametrize("kind", MUTANTS)
def test_planted_mistake_is_caught(kind):
    rec = rec_mutant(kind)
    failed = []
    for name, pin in P.all_recurrence_pins(GOLD):
        try:
            pin(rec)
        except AssertionError:
            failed.append(name)
    assert failed, f"mutant {kind} passed every pin"


# --------------------------------------------------------------------------- chunk method

def _chunk(seed, C, m, n=3):
    q, k, v, a, th, b, S0 = P.random_head(seed, C, m, n, alpha=(0.6, 1.0))
    return q, k, v, a, th, b, S0


@pytest.mark.parametrize("C,m", [(1, 4), (2, 3), (5, 8), (8, 8), (16, 16), (16, 6)])
def test_constructive_wy_all_prefixes(C, m):
    """P6: P_t = Gamma_t - Y_t M_t W_t^* equals the dense product A_t...A_1 for every prefix
    (Thm 4.2, Cor. 4.3); the paper prints worst case 1.9e-15 (Table 8)."""
    q, k, v, a, th, b, S0 = _chunk(40 + C + m, C, m)
    lams = cw.phase_decay(a, th)
    us, rs = cw.wy_vectors(k, a, th, b[:, None])
    pref = cw.constructive_wy(lams, us, rs, prefixes=True)
    Pd = np.eye(m, dtype=complex)
    for t in range(C):
        Pd = cw.transition(k[t], a[t], th[t], b[t]) @ Pd
        gamma, Y, W, M = pref[t]
        assert Y.shape == (m, t + 1) and M.shape == (t + 1, t + 1)
        err = np.max(np.abs(cw.wy_matrix(gamma, Y, W, M) - Pd)) / np.max(np.abs(Pd))
        assert err <= 10 * GOLD["constructive_chunk_wy_product"], (t, err)
        assert np.allclose(np.triu(M, 1), 0) and np.allclose(np.diag(M), 1)


def test_single_step_dplr_form():
    """A_t = Lambda_t - u_t r_t^* with u = beta k, r = Lambda^* k (eq. (single-step-wy))."""
    q, k, v, a, th, b, S0 = _chunk(5, 6, 7)
    for t in range(6):
        u, r = cw.wy_vectors(k[t], a[t], th[t], b[t])
        A = np.diag(cw.phase_decay(a[t], th[t])) - np.outer(u, np.conj(r))
        assert np.max(np.abs(A - cw.transition(k[t], a[t], th[t], b[t]))) < 1e-15


@pytest.mark.parametrize("r1,r2,m", [(1, 1, 3), (3, 5, 8), (6, 4, 6)])
def test_block_wy_closure(r1, r2, m):
    """P-clo: tuples compose into the tuple of A_2 A_1 with rank r1 + r2 (Thm 4.1);
    the paper prints worst case 6.7e-16 (Table 8)."""
    rng = np.random.default_rng(r1 * 10 + r2)

    def tup(r):
        return (np.diag(P.cn(rng, (m,))), P.cn(rng, (m, r)), P.cn(rng, (m, r)), P.cn(rng, (r, r)))

    t1, t2 = tup(r1), tup(r2)
    dense = lambda t: t[0] - t[1] @ t[3] @ cw.H(t[2])
    c = cw.compose_wy(t1, t2)
    assert c[1].shape == (m, r1 + r2) and c[3].shape == (r1 + r2, r1 + r2)
    ref = dense(t2) @ dense(t1)
    err = np.max(np.abs(dense(c) - ref)) / np.max(np.abs(ref))
    assert err <= 10 * GOLD["block_wy_closure"], err


def test_block_wy_closure_of_chunk_summaries():
    """Composing the constructive summaries of two chunks equals the summary of the joined
    chunk's dense product (Thm 4.1 applied to Thm 4.2 outputs)."""
    q, k, v, a, th, b, S0 = _chunk(77, 10, 6)
    lams = cw.phase_decay(a, th)
    us, rs = cw.wy_vectors(k, a, th, b[:, None])
    g1, Y1, W1, M1 = cw.constructive_wy(lams[:4], us[:4], rs[:4])
    g2, Y2, W2, M2 = cw.constructive_wy(lams[4:], us[4:], rs[4:])
    c = cw.compose_wy((np.diag(g1), Y1, W1, M1), (np.diag(g2), Y2, W2, M2))
    Pd = np.eye(6, dtype=complex)
    for t in range(10):
        Pd = cw.transition(k[t], a[t], th[t], b[t]) @ Pd
    assert np.max(np.abs(c[0] - c[1] @ c[3] @ cw.H(c[2]) - Pd)) < 1e-14


@pytest.mark.parametrize("C,m,n", [(4, 4, 3), (16, 8, 5), (32, 16, 8)])
def test_affine_chunk_transfer(C, m, n):
    """P-aff: S_C = (Gamma - Y M W^*) S_0 + B^chunk with B^chunk from the zero-state
    recurrence (Thm 4.4; apply-transfer equation); the paper prints 2.4e-16 (Table 8)."""
    q, k, v, a, th, b, S0 = _chunk(60 + C, C, m, n)
    o, S = rec_c(q, k, v, a, th, b, S0)
    tr = cw.chunk_summary(k, v, a, th, b)
    S2 = cw.apply_transfer(tr, S0)
    err = np.max(np.abs(S2 - S)) / np.max(np.abs(S))
    assert err <= 100 * GOLD["affine_chunk_transfer"], err
    # B^chunk is the sum of A_{C:i+1} B_i written out with dense matrices
    Bsum = np.zeros((m, n), complex)
    for i in range(C):
        term = cw.write(k[i], v[i], b[i])
        for j in range(i + 1, C):
            term = cw.transition(k[j], a[j], th[j], b[j]) @ term
        Bsum += term
    assert np.max(np.abs(Bsum - tr[4])) < 1e-13


@pytest.mark.parametrize("C,m", [(4, 16), (8, 16), (16, 16), (16, 32), (32, 16)])
def test_rank_budget(C, m):
    """P-rank: rank(P_C - Gamma_C) = min(C, m) for generic inputs (Thm 5.3; chunk sanity
    check after Table 8)."""
    q, k, v, a, th, b, S0 = _chunk(90 + C + m, C, m)
    lams = cw.phase_decay(a, th)
    us, rs = cw.wy_vectors(k, a, th, b[:, None])
    gamma, Y, W, M = cw.constructive_wy(lams, us, rs)
    corr = Y @ M @ cw.H(W)
    sv = np.linalg.svd(corr, compute_uv=False)
    assert int(np.sum(sv > 1e-10 * sv[0])) == min(C, m)


@pytest.mark.parametrize("C", [1, 2, 3, 5, 8, 16, 32, 64])
def test_chunk_invariance_vs_oracle(C):
    """P-C: chunk-WY scan (Alg. 1 + apply-transfer + prefix outputs) matches the oracle to
    1e-10 in float64 for every C, including a ragged last chunk (Thm 6.1)."""
    P.pin_chunk_invariance(rec_c, Cs=(C,), tol=1e-10)


@pytest.mark.parametrize("C", [1, 2, 5, 16, 64])
def test_closed_forms_match_recursion_and_oracle(C):
    """P7: closed-form Y, W, M of the module docstring equal the Thm 4.2 recursion, and
    the chunked closed-form forward matches the oracle."""
    m = 8
    q, k, v, a, th, b, S0 = P.random_head(200 + C, C, m, 4, alpha=(0.6, 1.0))
    lams = cw.phase_decay(a, th)
    us, rs = cw.wy_vectors(k, a, th, b[:, None])
    gamma, Y, W, M = cw.constructive_wy(lams, us, rs)
    G = np.cumprod(lams, axis=0)
    Yc = ((G[-1][None, :] / G) * (b[:, None] * k)).T
    Wc = (np.conj(G) * k).T
    Lp = np.tril(np.einsum("ti,tji,ji->tj", np.conj(k), G[:, None, :] / G[None, :, :], k), -1)
    Mc = np.linalg.inv(np.eye(C) + Lp @ np.diag(b))
    assert np.max(np.abs(Yc - Y)) < 1e-13 and np.max(np.abs(Wc - W)) < 1e-13
    assert np.max(np.abs(Mc - M)) < 1e-11
    assert np.max(np.abs(gamma - G[-1])) < 1e-14
    T = 3 * C + 1
    q, k, v, a, th, b, S0 = P.random_head(300 + C, T, m, 4, alpha=(0.6, 1.0))
    o, S = rec_c(q, k, v, a, th, b, S0)
    o2, S2 = cw.forward_ut(q, k, v, a, th, b, S0, C)
    assert P.rel(o2, o) < 1e-10 and P.rel(S2, S) < 1e-10


def test_oracle_errors_on_bad_arguments():
    with pytest.raises(RuntimeError):
        z = np.zeros((1, 1, 2, 0))
        oracle.recurrence(z, z, np.zeros((1, 1, 2, 1)), z.real, z.real, np.zeros((1, 1, 2)))


def test_inputs_module_is_reproducible_and_stored():
    """The generator draws each head from its own stream and rounds to the storage dtype."""
    from paper_2607_11897_amd import inputs as I
    w = I.WORKLOADS["tiny_f32"]
    x = I.make_chunk_inputs(w)
    y = I.make_chunk_inputs(w, heads=[(0, 0)])
    assert np.array_equal(x.q, y.q) and np.array_equal(x.beta, y.beta)
    assert np.allclose(np.linalg.norm(x.k, axis=-1), 1, atol=1e-6)
    assert np.array_equal(x.q.real.astype(np.float32).astype(np.float64), x.q.real)
    wb = I.WORKLOADS["fwd_bf16_b8h16_t4k"]
    z = I.make_chunk_inputs(wb, T=8, B=1, H=1)
    bits = I.f32_to_bf16_bits(z.alpha.astype(np.float32))
    assert np.array_equal(I.bf16_bits_to_f32(bits).astype(np.float64), z.alpha)
    # bf16 rounding is nearest-even: 1 + 2^-8 (a tie) rounds down to 1, 1 + 3*2^-8 rounds up
    t = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8], np.float32)
    assert list(I.bf16_bits_to_f32(I.f32_to_bf16_bits(t))) == [1.0, 1 + 2 ** -6]
