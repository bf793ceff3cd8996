"""Seeded synthetic inputs for the SFDA hot path.

This module draws and stores inputs only; it contains none of the
recurrence's arithmetic, so the CPU oracle and the GPU library can both
consume exactly the same stored values.

Shapes follow the paper's problem statement (Sec. 3, Eq. (sfda) and the
output rule that follows it): per (batch, head) a complex key/query of
``m`` coordinates, a complex value of ``n`` coordinates, channel-wise real
decay ``alpha`` and phase ``theta`` (``m`` each) and a scalar step ``beta``.
The complex Gaussian law is ``CN(0,1) = (N(0,1) + i N(0,1)) / sqrt(2)`` and
keys are L2-normalised over their ``m`` complex coordinates (the key rule of
the stable parameterisation in Sec. 3, with epsilon = 0).

Every (batch, head) pair draws from its own ``numpy`` PCG64 stream seeded by
``(seed, b, h)``, in the fixed order q, k, v, alpha-source, theta, beta, S0,
each drawn in float64 (complex: real plane, then imaginary plane).  Heads
are therefore reproducible one at a time, which lets a test check a sampled
subset of heads of a full-size run against the oracle.

Storage rounding is round-to-nearest-even to float32, and for bfloat16 a
second round-to-nearest-even from float32.  The oracle is given the stored
(rounded) values upcast exactly to float64.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np

# ---------------------------------------------------------------------------
# workload table
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Laws:
    """Distribution laws of one workload (all drawn per token, per head)."""
    alpha: tuple          # ("uniform", lo, hi) | ("softplus", scale) | ("mixed", lo, hi)
    theta: tuple          # ("uniform", lo, hi) | ("normal", std)
    beta: tuple           # ("uniform", lo, hi)
    s0_scale: Optional[float]  # None => zero initial state


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    T: int
    m: int
    n: int
    C: int
    dtype: str            # "f32" | "bf16"  (storage of q,k,v,alpha,theta,beta and o)
    laws: Laws
    seed: int
    tol: float            # max-norm relative error bound against the oracle


LAWS_TINY = Laws(alpha=("uniform", 0.90, 0.999), theta=("uniform", -math.pi, math.pi),
                 beta=("uniform", 0.0, 1.0), s0_scale=None)
LAWS_MAIN = Laws(alpha=("softplus", 16.0), theta=("normal", 0.5),
                 beta=("uniform", 0.0, 1.0), s0_scale=0.1)
LAWS_LONG = Laws(alpha=("uniform", 0.99, 0.9999), theta=("uniform", -math.pi, math.pi),
                 beta=("uniform", 0.5, 1.0), s0_scale=0.1)

WORKLOADS = {
    # tiny fp32 forward: m=16 complex key coordinates (d_k=32), d_v=16 real = 8 complex
    "tiny_f32": Workload("tiny_f32", 1, 1, 256, 16, 8, 16, "f32", LAWS_TINY, 1000, 1e-4),
    # same, with 16 complex value columns
    "tiny_f32_n16": Workload("tiny_f32_n16", 1, 1, 256, 16, 16, 16, "f32", LAWS_TINY, 1000, 1e-4),
    # fp32 chunk forward, d_k = d_v = 128 real
    "fwd_f32_b4h8_t2k": Workload("fwd_f32_b4h8_t2k", 4, 8, 2048, 64, 64, 64, "f32", LAWS_MAIN, 1001, 1e-4),
    # bf16 in/out, fp32 state and accumulation: the headline throughput workload
    "fwd_bf16_b8h16_t4k": Workload("fwd_bf16_b8h16_t4k", 8, 16, 4096, 64, 64, 64, "bf16", LAWS_MAIN, 1002, 2e-2),
    # long-context stability, near-unit decay
    "long_f32_h16_t64k": Workload("long_f32_h16_t64k", 1, 16, 65536, 64, 64, 64, "f32", LAWS_LONG, 1003, 1e-4),
}

# recurrent decode: state [512, 32, 64, 64] complex fp32, 1024 steps, main laws
DECODE = dict(name="decode_f32_b512h32", B=512, H=32, m=64, n=64, steps=1024,
              laws=LAWS_MAIN, seed=1004, tol=1e-4)


# ---------------------------------------------------------------------------
# storage rounding
# ---------------------------------------------------------------------------

def f32_to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    bias = ((b >> 16) & 1) + np.uint32(0x7FFF)
    return ((b + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def round_to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round a float64 (or complex128) array to the storage dtype; return float64/complex128
    holding exactly the stored values."""
    if np.iscomplexobj(x):
        return round_to_storage(x.real, dtype) + 1j * round_to_storage(x.imag, dtype)
    x32 = x.astype(np.float32)
    if dtype == "f32":
        return x32.astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f32(f32_to_bf16_bits(x32)).astype(np.float64)
    raise ValueError(dtype)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stored buffer for upload: complex arrays become interleaved (re, im) pairs on a
    trailing axis of 2; float32 or bf16 (as uint16 bits)."""
    if np.iscomplexobj(x):
        x = np.stack([x.real, x.imag], axis=-1)
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f32":
        return x32
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(dtype)


# ---------------------------------------------------------------------------
# draws
# ---------------------------------------------------------------------------

def _cn(rng: np.random.Generator, shape) -> np.ndarray:
    re = rng.standard_normal(shape)
    im = rng.standard_normal(shape)
    return (re + 1j * im) / math.sqrt(2.0)


def _alpha(rng, law, shape):
    if law[0] == "uniform":
        return rng.uniform(law[1], law[2], shape)
    if law[0] == "mixed":           # even channels exactly 1, odd channels U(lo, hi)
        a = rng.uniform(law[1], law[2], shape)
        a[..., 0::2] = 1.0
        return a
    if law[0] == "softplus":
        x = rng.standard_normal(shape)
        return np.exp(-np.logaddexp(0.0, x) / law[1])
    raise ValueError(law)


def _theta(rng, law, shape):
    if law[0] == "uniform":
        return rng.uniform(law[1], law[2], shape)
    if law[0] == "normal":
        return law[1] * rng.standard_normal(shape)
    raise ValueError(law)


def _normalise_keys(k: np.ndarray) -> np.ndarray:
    nrm = np.sqrt(np.sum(k.real ** 2 + k.imag ** 2, axis=-1, keepdims=True))
    return k / nrm


def draw_head(laws: Laws, seed_seq: Sequence[int], T: int, m: int, n: int):
    """One head's float64 draws (unrounded), in the fixed draw order."""
    rng = np.random.Generator(np.random.PCG64(list(seed_seq)))
    q = _cn(rng, (T, m))
    k = _normalise_keys(_cn(rng, (T, m)))
    v = _cn(rng, (T, n))
    alpha = _alpha(rng, laws.alpha, (T, m))
    theta = _theta(rng, laws.theta, (T, m))
    beta = rng.uniform(laws.beta[1], laws.beta[2], (T,))
    S0 = None if laws.s0_scale is None else laws.s0_scale * _cn(rng, (m, n))
    return q, k, v, alpha, theta, beta, S0


@dataclasses.dataclass
class ChunkInputs:
    """Stored inputs of one chunk-forward call, as exact float64/complex128 values.

    q, k: [B,H,T,m] complex; v: [B,H,T,n] complex; alpha, theta: [B,H,T,m];
    beta: [B,H,T]; S0: [B,H,m,n] complex (float32 values) or None.
    """
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    alpha: np.ndarray
    theta: np.ndarray
    beta: np.ndarray
    S0: Optional[np.ndarray]
    dtype: str

    @property
    def shape(self):
        B, H, T, m = self.q.shape
        return B, H, T, m, self.v.shape[-1]

    def storage(self) -> dict:
        """Buffers exactly as uploaded (interleaved complex; f32 or bf16 bits)."""
        d = {name: to_storage(getattr(self, name), self.dtype)
             for name in ("q", "k", "v", "alpha", "theta", "beta")}
        d["S0"] = None if self.S0 is None else to_storage(self.S0, "f32")
        return d

    def head(self, b: int, h: int) -> "ChunkInputs":
        return ChunkInputs(self.q[b:b + 1, h:h + 1], self.k[b:b + 1, h:h + 1],
                           self.v[b:b + 1, h:h + 1], self.alpha[b:b + 1, h:h + 1],
                           self.theta[b:b + 1, h:h + 1], self.beta[b:b + 1, h:h + 1],
                           None if self.S0 is None else self.S0[b:b + 1, h:h + 1],
                           self.dtype)


@dataclasses.dataclass
class GatedInputs:
    """Stored inputs of one gated chunk-forward call (pre-activations), as exact
    float64/complex128 values.  q, k_raw: [B,H,T,m] complex; v: [B,H,T,n] complex;
    a, b: [B,H,T,m]; c: [B,H,T]; S0: [B,H,m,n] complex or None."""
    q: np.ndarray
    k_raw: np.ndarray
    v: np.ndarray
    a: np.ndarray
    b: np.ndarray
    c: np.ndarray
    S0: Optional[np.ndarray]
    dtype: str

    @property
    def shape(self):
        B, H, T, m = self.q.shape
        return B, H, T, m, self.v.shape[-1]

    def storage(self) -> dict:
        d = {name: to_storage(getattr(self, name), self.dtype)
             for name in ("q", "k_raw", "v", "a", "b", "c")}
        d["S0"] = None if self.S0 is None else to_storage(self.S0, "f32")
        return d

    def head(self, b: int, h: int) -> "GatedInputs":
        sl = (slice(b, b + 1), slice(h, h + 1))
        return GatedInputs(self.q[sl], self.k_raw[sl], self.v[sl], self.a[sl], self.b[sl],
                           self.c[sl], None if self.S0 is None else self.S0[sl], self.dtype)


def make_gated_inputs(B: int, H: int, T: int, m: int, n: int, dtype: str, seed: int,
                      a_mean: float = 2.0, a_std: float = 1.5, b_std: float = 1.0,
                      c_std: float = 1.0, s0_scale: Optional[float] = 0.1,
                      zero_key_every: int = 0) -> GatedInputs:
    """Seeded pre-activations: q, k_raw, v complex Gaussian CN(0, 1) (raw keys not
    normalised), a ~ N(a_mean, a_std^2), b ~ N(0, b_std^2), c ~ N(0, c_std^2) per head from
    PCG64 streams seeded (seed, b, h), drawn in the order q, k_raw, v, a, b, c, S0; every
    zero_key_every-th token (if > 0) gets an all-zero raw key.  Rounded to the storage
    dtype, which both the oracle and the GPU read."""
    shp = lambda *t: (B, H) + t
    q = np.empty(shp(T, m), np.complex128); k_raw = np.empty_like(q)
    v = np.empty(shp(T, n), np.complex128)
    a = np.empty(shp(T, m)); bb = np.empty(shp(T, m)); c = np.empty(shp(T))
    S0 = None if s0_scale is None else np.empty(shp(m, n), np.complex128)
    for ib in range(B):
        for ih in range(H):
            rng = np.random.Generator(np.random.PCG64([seed, ib, ih]))
            q[ib, ih] = _cn(rng, (T, m))
            k_raw[ib, ih] = _cn(rng, (T, m))
            v[ib, ih] = _cn(rng, (T, n))
            a[ib, ih] = rng.normal(a_mean, a_std, (T, m))
            bb[ib, ih] = rng.normal(0.0, b_std, (T, m))
            c[ib, ih] = rng.normal(0.0, c_std, (T,))
            if S0 is not None:
                S0[ib, ih] = s0_scale * _cn(rng, (m, n))
    if zero_key_every > 0:
        k_raw[:, :, ::zero_key_every, :] = 0
    st = lambda x: round_to_storage(x, dtype)
    return GatedInputs(st(q), st(k_raw), st(v), st(a), st(bb), st(c),
                       None if S0 is None else round_to_storage(S0, "f32"), dtype)


def make_chunk_inputs(w: Workload, T: Optional[int] = None, B: Optional[int] = None,
                      H: Optional[int] = None, heads: Optional[Sequence] = None,
                      m: Optional[int] = None, n: Optional[int] = None) -> ChunkInputs:
    """Seeded inputs of a workload.  ``T``/``B``/``H``/``m``/``n`` override the sizes (for
    parity cases); ``heads`` restricts to a list of (b, h) pairs, returned as B=1, H=len."""
    B = w.B if B is None else B
    H = w.H if H is None else H
    T = w.T if T is None else T
    m = w.m if m is None else m
    n = w.n if n is None else n
    pairs = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    draws = [draw_head(w.laws, (w.seed, b, h), T, m, n) for (b, h) in pairs]
    shape_bh = (B, H) if heads is None else (1, len(pairs))

    def stack(i, dtype):
        if draws[0][i] is None:
            return None
        a = np.stack([d[i] for d in draws]).reshape(shape_bh + draws[0][i].shape)
        return round_to_storage(a, dtype)

    return ChunkInputs(stack(0, w.dtype), stack(1, w.dtype), stack(2, w.dtype),
                       stack(3, w.dtype), stack(4, w.dtype), stack(5, w.dtype),
                       stack(6, "f32"), w.dtype)


@dataclasses.dataclass
class DecoupledInputs:
    """Stored inputs of one write-decoupled forward call, as exact float64/complex128
    values.  q, k, r: [B,H,T,m] complex; v: [B,H,T,n] complex; alpha, theta: [B,H,T,m];
    eta, beta: [B,H,T]; S0: [B,H,m,n] complex or None."""
    q: np.ndarray
    k: np.ndarray
    r: np.ndarray
    v: np.ndarray
    alpha: np.ndarray
    theta: np.ndarray
    eta: np.ndarray
    beta: np.ndarray
    S0: Optional[np.ndarray]
    dtype: str

    @property
    def shape(self):
        B, H, T, m = self.q.shape
        return B, H, T, m, self.v.shape[-1]

    def storage(self) -> dict:
        d = {name: to_storage(getattr(self, name), self.dtype)
             for name in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")}
        d["S0"] = None if self.S0 is None else to_storage(self.S0, "f32")
        return d

    def head(self, b: int, h: int) -> "DecoupledInputs":
        sl = (slice(b, b + 1), slice(h, h + 1))
        return DecoupledInputs(self.q[sl], self.k[sl], self.r[sl], self.v[sl], self.alpha[sl],
                               self.theta[sl], self.eta[sl], self.beta[sl],
                               None if self.S0 is None else self.S0[sl], self.dtype)


def make_decoupled_inputs(B: int, H: int, T: int, m: int, n: int, dtype: str, seed: int,
                          laws: Laws = None, heads: Optional[Sequence] = None) -> DecoupledInputs:
    """Seeded write-decoupled inputs with the laws of the main workloads (default: those of
    the benchmarked shape): q, v ~ CN(0, 1), k and r ~ CN(0, 1) normalised, alpha and theta
    by the laws, eta ~ U(0, 1) (erase strengths), beta by the law (write strengths), S0 by
    the law; per head from PCG64 streams seeded (seed, b, h, 2), drawn in the order q, k,
    r, v, alpha, theta, eta, beta, S0; rounded to the storage dtype."""
    laws = LAWS_MAIN if laws is None else laws
    pairs = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    shape_bh = (B, H) if heads is None else (1, len(pairs))
    cols = {name: [] for name in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta", "S0")}
    for (b, h) in pairs:
        rng = np.random.Generator(np.random.PCG64([seed, b, h, 2]))
        cols["q"].append(_cn(rng, (T, m)))
        cols["k"].append(_normalise_keys(_cn(rng, (T, m))))
        cols["r"].append(_normalise_keys(_cn(rng, (T, m))))
        cols["v"].append(_cn(rng, (T, n)))
        cols["alpha"].append(_alpha(rng, laws.alpha, (T, m)))
        cols["theta"].append(_theta(rng, laws.theta, (T, m)))
        cols["eta"].append(rng.uniform(0.0, 1.0, (T,)))
        cols["beta"].append(rng.uniform(laws.beta[1], laws.beta[2], (T,)))
        cols["S0"].append(None if laws.s0_scale is None else laws.s0_scale * _cn(rng, (m, n)))

    def stack(name, dtype):
        if cols[name][0] is None:
            return None
        a = np.stack(cols[name])
        return round_to_storage(a.reshape(shape_bh + a.shape[1:]), dtype)

    return DecoupledInputs(*(stack(nm, dtype) for nm in ("q", "k", "r", "v", "alpha", "theta", "eta", "beta")),
                           stack("S0", "f32"), dtype)


def make_cotangents(B: int, H: int, T: int, m: int, n: int, out_dtype: str, seed: int,
                    dS_scale: Optional[float] = 1.0, heads: Optional[Sequence] = None):
    """Seeded upstream gradients for the backward: dO = dL/do [B,H,T,n] ~ CN(0, 1) rounded
    to o's storage dtype, and dS_T = dL/dS_T [B,H,m,n] ~ dS_scale CN(0, 1) rounded to
    float32 (None when dS_scale is None).  Per head from PCG64 streams seeded
    (seed, b, h, 1), drawn in the order dO, dS_T; ``heads`` as in make_chunk_inputs."""
    pairs = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    shape_bh = (B, H) if heads is None else (1, len(pairs))
    dO = np.empty((len(pairs), T, n), np.complex128)
    dS = None if dS_scale is None else np.empty((len(pairs), m, n), np.complex128)
    for j, (b, h) in enumerate(pairs):
        rng = np.random.Generator(np.random.PCG64([seed, b, h, 1]))
        dO[j] = _cn(rng, (T, n))
        if dS is not None:
            dS[j] = dS_scale * _cn(rng, (m, n))
    dO = round_to_storage(dO.reshape(shape_bh + (T, n)), out_dtype)
    dS = None if dS is None else round_to_storage(dS.reshape(shape_bh + (m, n)), "f32")
    return dO, dS


# ---------------------------------------------------------------------------
# decode-step inputs
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class StepInputs:
    """One decode token per head. q,k: [B,H,m]; v: [B,H,n]; alpha,theta: [B,H,m]; beta: [B,H]."""
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    alpha: np.ndarray
    theta: np.ndarray
    beta: np.ndarray
    dtype: str = "f32"

    def storage(self) -> dict:
        return {name: to_storage(getattr(self, name), self.dtype)
                for name in ("q", "k", "v", "alpha", "theta", "beta")}


def decode_state_head(b: int, h: int, m: int = 64, n: int = 64, seed: int = DECODE["seed"],
                      scale: float = 0.1) -> np.ndarray:
    """Initial decode state of one head: scale * CN(0,1), stored as float32 values."""
    rng = np.random.Generator(np.random.PCG64([seed, 1, b, h]))
    return round_to_storage(scale * _cn(rng, (m, n)), "f32")


def decode_step_heads(step: int, heads: Sequence, m: int = 64, n: int = 64,
                      laws: Laws = LAWS_MAIN, seed: int = DECODE["seed"],
                      dtype: str = "f32") -> StepInputs:
    """Per-step token inputs for a list of (b, h) heads, returned with shape [1, len(heads), ...]."""
    cols = []
    for (b, h) in heads:
        rng = np.random.Generator(np.random.PCG64([seed, 2, step, b, h]))
        q = _cn(rng, (m,))
        k = _normalise_keys(_cn(rng, (m,)))
        v = _cn(rng, (n,))
        alpha = _alpha(rng, laws.alpha, (m,))
        theta = _theta(rng, laws.theta, (m,))
        beta = rng.uniform(laws.beta[1], laws.beta[2], ())
        cols.append((q, k, v, alpha, theta, beta))
    st = [round_to_storage(np.stack([c[i] for c in cols])[None], dtype) for i in range(6)]
    return StepInputs(*st, dtype=dtype)


def fill_decode_bulk_torch(gen, B: int, H: int, m: int, n: int, device, laws: Laws = LAWS_MAIN):
    """Fill decode-step inputs for all heads with torch's seeded generator (device tensors,
    float32 interleaved layout).  Used for the heads a test does not sample; same laws."""
    import torch
    f = dict(device=device, dtype=torch.float32)

    def cn(shape):
        return torch.randn(*shape, 2, generator=gen, **f) / math.sqrt(2.0)

    q = cn((B, H, m))
    k = cn((B, H, m))
    k = k / torch.sqrt((k * k).sum(dim=(-1, -2), keepdim=True))
    v = cn((B, H, n))
    x = torch.randn(B, H, m, generator=gen, **f)
    alpha = torch.exp(-torch.nn.functional.softplus(x) / laws.alpha[1])
    theta = laws.theta[1] * torch.randn(B, H, m, generator=gen, **f)
    beta = torch.rand(B, H, generator=gen, **f) * (laws.beta[2] - laws.beta[1]) + laws.beta[1]
    return q, k, v, alpha, theta, beta
