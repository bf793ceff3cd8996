"""CPU oracle for SFDA -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  The GPU library never uses it, and it imports nothing
from the GPU library.

* ``recurrence`` / ``step``: the plain token-by-token recurrence (Sec. 3, Eq. (sfda)
  and the readout o_t = S_t^* q_t) in complex double precision, implemented in C
  (``oracle.c``) and called through ctypes.
* ``chunk_wy``: the paper's chunk method on the CPU in float64 numpy (Thm 4.1, Thm 4.2,
  Cor 4.3, Thm 4.4, Thm 4.5, Alg. 1 and the apply-transfer equation), plus dense
  brute-force helpers used by the pins.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# another build of oracle.c to load instead (the sanitizer pass points here); loaded as is
_LIB_OVERRIDE = os.environ.get("SFDA_ORACLE_LIB")
_lib = None


def build(verbose: bool = False, sanitize: bool = False, out: str = _LIB) -> str:
    """Compile oracle.c into liboracle.so (plain C, OpenMP, no fast-math).  sanitize builds
    it with clang under AddressSanitizer and UndefinedBehaviorSanitizer instead (serial: the
    OpenMP pragmas only split the loops over heads); out is the library path."""
    if sanitize:
        cmd = ["/opt/rocm/llvm/bin/clang", "-O1", "-g", "-std=c99", "-fPIC", "-shared", "-Wall",
               "-Wno-unknown-pragmas", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
               "-fno-sanitize-recover=undefined", "-o", out + ".tmp", _SRC, "-lm"]
    else:
        cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared", "-Wall",
               "-o", out + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build()
            lib = ctypes.CDLL(_LIB)
        d = ctypes.POINTER(ctypes.c_double)
        i = ctypes.c_int
        lib.oracle_recurrence.argtypes = [i, i, i, i, i, d, d, d, d, d, d, d, d, d, i]
        lib.oracle_recurrence.restype = i
        lib.oracle_step.argtypes = [i, i, i, i, d, d, d, d, d, d, d, d, i]
        lib.oracle_step.restype = i
        lib.oracle_max_threads.restype = i
        _lib = lib
    return _lib


def _c(x: np.ndarray):
    return x.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _as_pairs(x: np.ndarray) -> np.ndarray:
    """complex128 -> contiguous float64 [..., 2]."""
    x = np.asarray(x, dtype=np.complex128)
    return np.ascontiguousarray(np.stack([x.real, x.imag], axis=-1))


def _from_pairs(x: np.ndarray) -> np.ndarray:
    return x[..., 0] + 1j * x[..., 1]


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def recurrence(q, k, v, alpha, theta, beta, S0: Optional[np.ndarray] = None,
               nthreads: int = 0):
    """Token-by-token SFDA forward.

    q, k: [B,H,T,m] complex; v: [B,H,T,n] complex; alpha, theta: [B,H,T,m] real;
    beta: [B,H,T] real; S0: [B,H,m,n] complex or None (zero state).
    Returns (o [B,H,T,n] complex128, S_T [B,H,m,n] complex128).
    """
    lib = _load()
    B, H, T, m = np.shape(q)
    n = np.shape(v)[-1]
    qp, kp, vp = _as_pairs(q), _as_pairs(k), _as_pairs(v)
    a = np.ascontiguousarray(alpha, dtype=np.float64)
    th = np.ascontiguousarray(theta, dtype=np.float64)
    b = np.ascontiguousarray(beta, dtype=np.float64)
    s0 = None if S0 is None else _as_pairs(S0)
    o = np.zeros((B, H, T, n, 2))
    ST = np.zeros((B, H, m, n, 2))
    rc = lib.oracle_recurrence(B, H, T, m, n, _c(qp), _c(kp), _c(vp), _c(a), _c(th), _c(b),
                               None if s0 is None else _c(s0), _c(o), _c(ST), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"oracle_recurrence failed with code {rc}")
    return _from_pairs(o), _from_pairs(ST)


def step(q, k, v, alpha, theta, beta, S, nthreads: int = 0):
    """One decode token for every head.  q,k: [B,H,m]; v: [B,H,n]; alpha,theta: [B,H,m];
    beta: [B,H]; S: [B,H,m,n].  Returns (o [B,H,n], S_new [B,H,m,n])."""
    lib = _load()
    B, H, m = np.shape(q)
    n = np.shape(v)[-1]
    qp, kp, vp = _as_pairs(q), _as_pairs(k), _as_pairs(v)
    a = np.ascontiguousarray(alpha, dtype=np.float64)
    th = np.ascontiguousarray(theta, dtype=np.float64)
    b = np.ascontiguousarray(beta, dtype=np.float64)
    Sp = _as_pairs(S)
    o = np.zeros((B, H, n, 2))
    rc = lib.oracle_step(B, H, m, n, _c(qp), _c(kp), _c(vp), _c(a), _c(th), _c(b),
                         _c(Sp), _c(o), int(nthreads))
    if rc != 0:
        raise RuntimeError(f"oracle_step failed with code {rc}")
    return _from_pairs(o), _from_pairs(Sp)
