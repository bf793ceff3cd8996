"""Pins of the write-decoupled recurrence (oracle.decoupled; Sec. 3, write-decoupled
variant), CPU only.

Each check rests on something other than the oracle's own loop: the tied C oracle (the
variant with r = k, eta = beta is tied SFDA), a closed form (eta = 0 leaves a decayed sum of
writes), an exact projector property (eta = 1 with unit keys, no decay, removes the key's
component before the write), real linearity in S0 and conjugate linearity in v, and the
dense transition matrices built explicitly.  Copies with a planted mistake must each fail
one of them.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle import decoupled as D


def cn(rng, shape):
    return (rng.normal(size=shape) + 1j * rng.normal(size=shape)) / np.sqrt(2.0)


def sample(seed, B=1, H=2, T=24, m=6, n=4, unit=True):
    rng = np.random.default_rng(seed)
    k = cn(rng, (B, H, T, m))
    r = cn(rng, (B, H, T, m))
    if unit:
        k /= np.linalg.norm(k, axis=-1, keepdims=True)
        r /= np.linalg.norm(r, axis=-1, keepdims=True)
    return dict(q=cn(rng, (B, H, T, m)), k=k, r=r, v=cn(rng, (B, H, T, n)),
                alpha=rng.uniform(0.7, 1.0, (B, H, T, m)), theta=rng.uniform(-np.pi, np.pi, (B, H, T, m)),
                eta=rng.uniform(0, 1, (B, H, T)), beta=rng.uniform(0, 1, (B, H, T)), S0=cn(rng, (B, H, m, n)))


def run(fn, x, **over):
    y = dict(x, **over)
    return fn(y["q"], y["k"], y["r"], y["v"], y["alpha"], y["theta"], y["eta"], y["beta"], y["S0"])


def rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def pins(fn):
    """Names of the pins a decoupled recurrence fn fails."""
    failed = []
    x = sample(1)
    # tied SFDA: r = k, eta = beta, against the C oracle
    o, S = run(fn, x, r=x["k"], eta=x["beta"])
    o_c, S_c = oracle.recurrence(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], x["S0"])
    if not (rel(o, o_c) <= 1e-13 and rel(S, S_c) <= 1e-13):
        failed.append("tied reduction")
    # eta = 0: S_T = diag(prod lambda) S0 + sum_t diag(prod_{s>t} lambda_s) beta_t r_t v_t^*
    x0 = dict(x, eta=np.zeros_like(x["eta"]))
    _, S = run(fn, x0)
    lam = x["alpha"] * np.exp(1j * x["theta"])                            # [B,H,T,m]
    T = lam.shape[2]
    expect = np.prod(lam, axis=2)[..., None] * x["S0"]
    for t in range(T):
        decay = np.prod(lam[:, :, t + 1:], axis=2)                        # empty product = 1
        expect = expect + (decay * x["beta"][:, :, t, None] * x["r"][:, :, t])[..., None] * \
            np.conj(x["v"][:, :, t])[:, :, None, :]
    if not rel(S, expect) <= 1e-12:
        failed.append("eta = 0 closed form")
    # eta = 1, unit keys, no decay: k_t^* S_t = beta_t (k_t^* r_t) v_t^* after every token
    xe = dict(x, eta=np.ones_like(x["eta"]), alpha=np.ones_like(x["alpha"]), theta=np.zeros_like(x["theta"]))
    ok = True
    for t in (1, 7, 23):
        sl = {kk: (vv[:, :, :t] if kk not in ("S0",) else vv) for kk, vv in xe.items()}
        _, S = run(fn, sl)
        kt, rt, vt, bt = xe["k"][:, :, t - 1], xe["r"][:, :, t - 1], xe["v"][:, :, t - 1], xe["beta"][:, :, t - 1]
        lhs = np.einsum("bhi,bhic->bhc", np.conj(kt), S)
        rhs = (bt * np.einsum("bhi,bhi->bh", np.conj(kt), rt))[..., None] * np.conj(vt)
        ok = ok and np.max(np.abs(lhs - rhs)) <= 1e-13
    if not ok:
        failed.append("exact erase along unit keys")
    # S_T real-linear in S0 with v = 0; conjugate-linear in v from the zero state; o linear in q
    xv = dict(x, v=np.zeros_like(x["v"]))
    _, S1 = run(fn, xv)
    _, S2 = run(fn, xv, S0=(2 - 3j) * x["S0"])
    xz = dict(x, S0=np.zeros_like(x["S0"]))
    _, S3 = run(fn, xz)
    _, S4 = run(fn, xz, v=(2 - 3j) * x["v"])
    o5, _ = run(fn, xz)
    o6, _ = run(fn, xz, q=(2 - 3j) * x["q"])
    if not (rel(S2, (2 - 3j) * S1) <= 1e-13 and rel(S4, np.conj(2 - 3j) * S3) <= 1e-13 and
            rel(o6, (2 - 3j) * o5) <= 1e-13):
        failed.append("linearity")
    # dense transitions on one tiny head
    xs = sample(4, B=1, H=1, T=6, m=3, n=2)
    o, S = run(fn, xs)
    Sd = xs["S0"][0, 0].copy()
    od = []
    for t in range(6):
        kt, rt, vt = xs["k"][0, 0, t], xs["r"][0, 0, t], xs["v"][0, 0, t]
        A = (np.eye(3) - xs["eta"][0, 0, t] * np.outer(kt, np.conj(kt))) @ np.diag(
            xs["alpha"][0, 0, t] * np.exp(1j * xs["theta"][0, 0, t]))
        Sd = A @ Sd + xs["beta"][0, 0, t] * np.outer(rt, np.conj(vt))
        od.append(np.conj(Sd).T @ xs["q"][0, 0, t])
    if not (rel(o[0, 0], np.array(od)) <= 1e-13 and rel(S[0, 0], Sd) <= 1e-13):
        failed.append("dense transitions")
    return failed


def test_decoupled_oracle_passes_every_pin():
    assert pins(D.decoupled_recurrence) == []


def test_non_unit_keys_and_zero_state_run():
    x = sample(9, unit=False)
    o, S = run(D.decoupled_recurrence, x, S0=None)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(S))


def _mutant(kind):
    def fn(q, k, r, v, alpha, theta, eta, beta, S0):
        B, H, T, m = q.shape
        S = np.array(S0, dtype=np.complex128)
        o = np.empty((B, H, T, v.shape[-1]), np.complex128)
        for t in range(T):
            lam = alpha[:, :, t] * np.exp(1j * theta[:, :, t])
            S = lam[..., None] * S
            kt, rt = k[:, :, t], r[:, :, t]
            ed = rt if kind == "erase_along_r" else kt
            vv = v[:, :, t] if kind == "v_not_conj" else np.conj(v[:, :, t])
            wstr = eta[:, :, t] if kind == "write_with_eta" else beta[:, :, t]
            w = wstr[..., None, None] * rt[..., None] * vv[:, :, None, :]
            if kind == "write_before_erase":
                S = S + w
            xr = np.einsum("bhi,bhic->bhc", ed if kind == "erase_k_transposed" else np.conj(ed), S)
            S = S - eta[:, :, t, None, None] * ed[..., None] * xr[:, :, None, :]
            if kind != "write_before_erase":
                S = S + w
            o[:, :, t] = np.einsum("bhic,bhi->bhc", np.conj(S), q[:, :, t])
        return o, S
    return fn


@pytest.mark.parametrize("kind", ["erase_along_r", "v_not_conj", "write_with_eta", "write_before_erase",
                                  "erase_k_transposed"])
def test_planted_mistake_in_decoupled_recurrence_is_caught(kind):
    assert pins(_mutant(kind)) != [], kind


def test_unmutated_copy_passes():
    assert pins(_mutant("none")) == []
