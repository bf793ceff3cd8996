"""Pins of the oracle's reverse-mode gradients (oracle.backward), CPU only.

What fixes the gradients independently of their derivation:
* central finite differences of the forward -- the C oracle's token recurrence, itself
  pinned in test_oracle_pins.py -- for every real coordinate of every input (q, k, v
  real and imaginary parts, alpha, theta, beta, S0), on tiny heads;
* Euler's identity for parts of the forward that are homogeneous of degree one: o is
  real-linear in q and, from the zero state, in v; from v = 0, o and S_T are real-linear
  in S0 -- so there L equals Re <grad, input> exactly;
* special values: beta = 0 leaves dk, dv and dbeta's write part at zero, alpha = 1 and
  theta = 0 with beta = 0 make every state S0, so dS0 = sum_t q_t dO_t^* + dS_T.
Copies of the adjoint with a planted mistake must each fail one of these.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle import backward as BW

FIELDS_C = ("q", "k", "v", "S0")
FIELDS_R = ("alpha", "theta", "beta")


def cn(rng, shape):
    return (rng.normal(size=shape) + 1j * rng.normal(size=shape)) / np.sqrt(2.0)


def head(seed, B=1, H=1, T=6, m=3, n=2, beta=(0.0, 1.0), alpha=(0.6, 1.0), s0=True):
    rng = np.random.default_rng(seed)
    k = cn(rng, (B, H, T, m))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    x = dict(q=cn(rng, (B, H, T, m)), k=k, v=cn(rng, (B, H, T, n)),
             alpha=rng.uniform(*alpha, (B, H, T, m)), theta=rng.uniform(-np.pi, np.pi, (B, H, T, m)),
             beta=rng.uniform(*beta, (B, H, T)),
             S0=cn(rng, (B, H, m, n)) if s0 else np.zeros((B, H, m, n), np.complex128))
    up = dict(dO=cn(rng, (B, H, T, n)), dS_T=cn(rng, (B, H, m, n)))
    return x, up


def forward(x):
    return oracle.recurrence(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], x["S0"])


def L_of(x, up):
    o, S = forward(x)
    return BW.loss(o, S, up["dO"], up["dS_T"])


def fd_grads(x, up, h=1e-6):
    """dL/d(every real coordinate) by central differences of the C oracle."""
    out = {}
    for f in FIELDS_C + FIELDS_R:
        base = x[f]
        parts = (1.0, 1j) if f in FIELDS_C else (1.0,)
        g = np.zeros(base.shape, np.complex128 if f in FIELDS_C else np.float64)
        for idx in np.ndindex(base.shape):
            for p in parts:
                xp = dict(x); xm = dict(x)
                xp[f] = base.copy(); xm[f] = base.copy()
                xp[f][idx] += h * p
                xm[f][idx] -= h * p
                d = (L_of(xp, up) - L_of(xm, up)) / (2 * h)
                g[idx] += d * (1.0 if p == 1.0 else 1j)
        out[f] = g
    return out


def analytic(x, up, fn=BW.recurrence_backward):
    g = fn(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], x["S0"], up["dO"], up["dS_T"])
    return dict(q=g["dq"], k=g["dk"], v=g["dv"], S0=g["dS0"], alpha=g["dalpha"], theta=g["dtheta"],
                beta=g["dbeta"])


def fd_mismatch(x, up, fn=BW.recurrence_backward, tol=2e-7):
    """Names of the gradients that disagree with finite differences."""
    fd = fd_grads(x, up)
    an = analytic(x, up, fn)
    bad = []
    for f in fd:
        scale = max(np.max(np.abs(fd[f])), 1e-3)
        if not np.max(np.abs(fd[f] - an[f])) <= tol * scale:
            bad.append(f)
    return bad


def test_forward_states_match_c_oracle():
    x, _ = head(5, B=2, H=2, T=40, m=6, n=5)
    o, states = BW.forward_states(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], x["S0"])
    o_c, S_c = forward(x)
    assert np.max(np.abs(o - o_c)) <= 1e-13 * np.max(np.abs(o_c))
    assert np.max(np.abs(states[-1] - S_c)) <= 1e-13 * np.max(np.abs(S_c))


@pytest.mark.parametrize("seed,kw", [
    (1, dict()),
    (2, dict(B=2, H=1, T=5, m=2, n=3)),
    (3, dict(beta=(1.0, 1.0))),               # full erase with unit keys (singular transitions)
    (4, dict(alpha=(0.05, 0.3), T=4)),          # strong decay
    (5, dict(s0=False, m=4, n=1)),               # zero state, one value column
])
def test_gradients_match_finite_differences(seed, kw):
    x, up = head(seed, **kw)
    assert fd_mismatch(x, up) == []


def test_gradients_with_non_unit_keys():
    x, up = head(7, T=5)
    x["k"] = x["k"] * np.array([0.3, 1.7, 0.9, 2.2, 0.5])[None, None, :, None]
    assert fd_mismatch(x, up) == []


def test_euler_identities():
    x, up = head(11, B=2, H=2, T=30, m=5, n=4, s0=False)
    zero_dS = np.zeros_like(up["dS_T"])
    # o is real-linear in v from the zero state: L = Re <dv, v> (S_T as well)
    g = analytic(x, up)
    assert np.isclose(L_of(x, up), np.real(np.vdot(g["v"], x["v"])), rtol=1e-12, atol=0)
    # o is real-linear in q (S_T does not depend on q): with dS_T = 0, L = Re <dq, q>
    x2, up2 = head(12, B=1, H=2, T=30, m=5, n=4)
    up2 = dict(dO=up2["dO"], dS_T=zero_dS[:1])
    g2 = analytic(x2, up2)
    assert np.isclose(L_of(x2, up2), np.real(np.vdot(g2["q"], x2["q"])), rtol=1e-12, atol=0)
    # from v = 0, o and S_T are real-linear in S0: L = Re <dS0, S0>
    x3, up3 = head(13, B=1, H=2, T=30, m=5, n=4)
    x3["v"] = np.zeros_like(x3["v"])
    g3 = analytic(x3, up3)
    assert np.isclose(L_of(x3, up3), np.real(np.vdot(g3["S0"], x3["S0"])), rtol=1e-12, atol=0)


def test_special_values():
    x, up = head(17, B=1, H=1, T=12, m=4, n=3)
    x["beta"] = np.zeros_like(x["beta"])
    g = analytic(x, up)
    # no write and no erase: v and the keys do not enter
    assert np.all(g["v"] == 0) and np.all(g["k"] == 0)
    # alpha = 1, theta = 0, beta = 0: S_t = S0 for every t
    x["alpha"] = np.ones_like(x["alpha"])
    x["theta"] = np.zeros_like(x["theta"])
    g = analytic(x, up)
    expect = up["dS_T"] + np.einsum("bhti,bhtc->bhic", x["q"], np.conj(up["dO"]))
    assert np.max(np.abs(g["S0"] - expect)) <= 1e-13


def test_zero_state_none_equals_zeros():
    x, up = head(19, s0=False)
    a = BW.recurrence_backward(x["q"], x["k"], x["v"], x["alpha"], x["theta"], x["beta"], None,
                               up["dO"], up["dS_T"])
    b = analytic(x, up)
    assert np.array_equal(a["dq"], b["q"]) and np.array_equal(a["dS0"], b["S0"])


# --------------------------------------------------------------------------- planted mistakes

def _mutant(kind):
    """A copy of the adjoint sweep with one planted mistake."""
    def fn(q, k, v, alpha, theta, beta, S0, dO, dS_T):
        B, H, T, m = q.shape
        n = v.shape[-1]
        _, states = BW.forward_states(q, k, v, alpha, theta, beta, S0)
        out = dict(dq=np.zeros_like(q), dk=np.zeros_like(k), dv=np.zeros_like(v),
                   dalpha=np.zeros(alpha.shape), dtheta=np.zeros(theta.shape), dbeta=np.zeros(beta.shape))
        Gs = np.array(dS_T, dtype=np.complex128)
        for t in range(T - 1, -1, -1):
            S_prev, S_t = states[t], states[t + 1]
            qt, kt, bt = q[:, :, t], k[:, :, t], beta[:, :, t]
            lam = alpha[:, :, t] * np.exp(1j * theta[:, :, t])
            Sp = lam[..., None] * S_prev
            D = np.conj(v[:, :, t]) - np.einsum("bhi,bhic->bhc", np.conj(kt), Sp)
            out["dq"][:, :, t] = np.einsum("bhic,bhc->bhi", S_prev if kind == "dq_prev_state" else S_t,
                                           dO[:, :, t])
            if kind != "readout_after_write":
                Gs = Gs + qt[..., None] * np.conj(dO[:, :, t])[:, :, None, :]
            u = np.einsum("bhic,bhi->bhc", np.conj(Gs), kt)
            if kind == "readout_after_write":
                Gs = Gs + qt[..., None] * np.conj(dO[:, :, t])[:, :, None, :]
            out["dv"][:, :, t] = bt[..., None] * (np.conj(u) if kind == "dv_conj" else u)
            out["dbeta"][:, :, t] = np.real(np.sum(u * D, axis=-1))
            lin = np.einsum("bhic,bhc->bhi", Gs, np.conj(D))
            anti = np.einsum("bhic,bhc->bhi", Sp, u)
            out["dk"][:, :, t] = bt[..., None] * (lin if kind == "dk_no_erase_term" else lin - anti)
            sgn = 1.0 if kind == "erase_sign" else -1.0
            Gp = Gs + sgn * bt[..., None, None] * kt[..., None] * np.conj(u)[:, :, None, :]
            g = np.sum(Gp * np.conj(S_prev), axis=-1)
            out["dalpha"][:, :, t] = np.real(np.conj(g) * np.exp(1j * theta[:, :, t]))
            dth = np.conj(g) * 1j * (np.exp(1j * theta[:, :, t]) if kind == "dtheta_no_alpha" else lam)
            out["dtheta"][:, :, t] = np.real(dth)
            Gs = (lam if kind == "lambda_not_conj" else np.conj(lam))[..., None] * Gp
        out["dS0"] = Gs
        return out
    return fn


MUTANTS = ["dq_prev_state", "readout_after_write", "dv_conj", "dk_no_erase_term", "erase_sign",
           "dtheta_no_alpha", "lambda_not_conj"]


def test_unmutated_copy_passes():
    x, up = head(23, T=5)
    assert fd_mismatch(x, up, fn=_mutant("none")) == []


@pytest.mark.parametrize("kind", MUTANTS)
def test_planted_mistake_in_adjoint_is_caught(kind):
    x, up = head(23, T=5)
    assert fd_mismatch(x, up, fn=_mutant(kind)) != [], f"mutant {kind} passed"
