"""Thin Python binding of libsfda (ctypes).  Argument marshalling only: every step of the
computation runs in the HIP kernels behind the C ABI declared in include/sfda.h.

Tensors are torch tensors on the GPU, contiguous, with complex values stored as a trailing
axis of 2 (re, im) -- float32 (``torch.view_as_real`` of complex64 gives this layout) or
bfloat16.  torch is used for device memory and streams only.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; SFDA_LIBRARY names another build to load (the sanitizer pass uses it)
LIB_PATH = os.environ.get("SFDA_LIBRARY") or os.path.join(HERE, "libsfda.so")

SFDA_F32, SFDA_BF16 = 0, 1
STATUS = {0: "SFDA_OK", 1: "SFDA_ERR_NULL", 2: "SFDA_ERR_SHAPE", 3: "SFDA_ERR_CHUNK",
          4: "SFDA_ERR_DTYPE", 5: "SFDA_ERR_ALIGN", 6: "SFDA_ERR_ALIAS", 7: "SFDA_ERR_HIP",
          8: "SFDA_ERR_SCRATCH"}
NOALLOC_SCRATCH_BYTES = 32 * 1024 * 1024      # SFDA_NOALLOC_SCRATCH_BYTES
EXPORTS = ("sfda_chunk_fwd", "sfda_chunk_fwd_sliced", "sfda_chunk_fwd_gated", "sfda_chunk_fwd_decoupled",
           "sfda_chunk_fwd_segmented", "sfda_chunk_fwd_segmented_noalloc",
           "sfda_chunk_fwd_segmented_workspace_bytes", "sfda_chunk_fwd_auto_segments",
           "sfda_chunk_bwd", "sfda_chunk_bwd_workspace_bytes", "sfda_chunk_solve_monitor",
           "sfda_step", "sfda_status_string", "sfda_abi_version")

_lib = None


class SfdaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = load_library().sfda_status_string(status).decode()
        super().__init__(f"{where}: {STATUS.get(status, status)} ({msg})")


@contextlib.contextmanager
def library(path: str):
    """Run the binding against another build of the library at `path` (the LDS-poison
    debug build in its test) for the duration of a with-block, then go back to the one
    loaded before.  Nothing may be in flight on the device when the block ends."""
    global _lib
    saved = _lib
    _lib = None
    try:
        yield load_library(path)
    finally:
        _lib = saved


def load_library(path: str = LIB_PATH):
    """Load libsfda.so; raises if it has not been built (there is no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libsfda.so not found at {path}: build it with "
                           "`python -m paper_2607_11897_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(path)
    vp, i = ctypes.c_void_p, ctypes.c_int
    lib.sfda_chunk_fwd.argtypes = [vp] * 9 + [i] * 6 + [i, i, vp]
    lib.sfda_chunk_fwd.restype = i
    lib.sfda_chunk_fwd_sliced.argtypes = [vp] * 9 + [i] * 7 + [i, i, vp]
    lib.sfda_chunk_fwd_sliced.restype = i
    f = ctypes.c_float
    lib.sfda_chunk_fwd_gated.argtypes = [vp] * 9 + [i] * 6 + [f] * 4 + [i, i, vp]
    lib.sfda_chunk_fwd_gated.restype = i
    lib.sfda_chunk_fwd_decoupled.argtypes = [vp] * 11 + [i] * 6 + [i, i, vp]
    lib.sfda_chunk_fwd_decoupled.restype = i
    lib.sfda_chunk_fwd_segmented.argtypes = [vp] * 9 + [i] * 7 + [i, i, vp, ctypes.c_size_t, vp]
    lib.sfda_chunk_fwd_segmented.restype = i
    lib.sfda_chunk_fwd_segmented_noalloc.argtypes = [vp] * 9 + [i] * 7 + [i, i, vp]
    lib.sfda_chunk_fwd_segmented_noalloc.restype = i
    lib.sfda_chunk_fwd_segmented_workspace_bytes.argtypes = [i] * 7
    lib.sfda_chunk_fwd_segmented_workspace_bytes.restype = ctypes.c_size_t
    lib.sfda_chunk_fwd_auto_segments.argtypes = [i] * 7
    lib.sfda_chunk_solve_monitor.argtypes = [vp] * 6 + [i] * 5 + [vp]
    lib.sfda_chunk_solve_monitor.restype = i
    lib.sfda_chunk_fwd_auto_segments.restype = i
    lib.sfda_chunk_bwd.argtypes = [vp] * 16 + [i] * 6 + [i, i, vp, ctypes.c_size_t, vp]
    lib.sfda_chunk_bwd.restype = i
    lib.sfda_chunk_bwd_workspace_bytes.argtypes = [i] * 6
    lib.sfda_chunk_bwd_workspace_bytes.restype = ctypes.c_size_t
    lib.sfda_step.argtypes = [vp] * 8 + [i] * 4 + [i, i, vp]
    lib.sfda_step.restype = i
    lib.sfda_status_string.argtypes = [i]
    lib.sfda_status_string.restype = ctypes.c_char_p
    lib.sfda_abi_version.restype = i
    _lib = lib
    return lib


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return SFDA_F32
    if t.dtype == torch.bfloat16:
        return SFDA_BF16
    raise TypeError(f"unsupported dtype {t.dtype} (float32 or bfloat16)")


def _check(named: dict) -> None:
    """Every given tensor has its expected shape and sits on the first tensor's GPU: the
    library receives bare pointers and sizes, so a short buffer or a host pointer would
    only show up as a fault inside a kernel.  `named` maps a name to (tensor or None,
    expected shape)."""
    dev = None
    for name, (t, shape) in named.items():
        if t is None:
            continue
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    for name, (t, _) in named.items():
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"{name} is on {t.device}, the other tensors on {dev}")


def _need_f32(**named) -> None:
    """States (S0, S_T, dS_T, S) are complex float32 whatever the inputs' dtype: the library
    reads and writes m * n * 8 bytes per head there, so a half-width buffer would be
    overrun."""
    import torch
    for name, t in named.items():
        if t is not None and t.dtype != torch.float32:
            raise TypeError(f"{name} must be float32 (got {t.dtype})")


def _dims(q, v, nd):
    if q.dim() != nd or v.dim() != nd:
        raise ValueError(f"q and v must have {nd} dimensions")
    return q.shape


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def chunk_fwd(q, k, v, alpha, theta, beta, S0=None, C: int = 64, *, o=None, S_T=None,
              out_dtype=None, want_state: bool = True, slice: Optional[int] = None,
              segments="auto", workspace=None, stream=None) -> Tuple:
    """SFDA chunkwise forward.  q, k: [B,H,T,m,2]; v: [B,H,T,n,2]; alpha, theta: [B,H,T,m];
    beta: [B,H,T] (all float32 or all bfloat16); S0: [B,H,m,n,2] float32 or None.
    Returns (o [B,H,T,n,2] in out_dtype, S_T [B,H,m,n,2] float32 or None).
    slice: value columns per workgroup (sfda_chunk_fwd_sliced); segments: G parallel
    segments per head (sfda_chunk_fwd_segmented; `workspace` a uint8 device tensor of at
    least segmented_workspace_bytes(...) bytes, allocated here when not given), None for one
    scan per head (sfda_chunk_fwd), or "auto" (the default, without a slice): the count
    sfda_chunk_fwd_auto_segments suggests, segments when the heads alone would leave most
    compute units idle (the workspace then comes from torch's allocator)."""
    import torch
    lib = load_library()
    B, H, T, m, _ = _dims(q, v, 5)
    n = v.shape[3]
    in_code = _dtype_code(q)
    for t in (k, v, alpha, theta, beta):
        if t.dtype != q.dtype:
            raise TypeError("q, k, v, alpha, theta, beta must share one dtype")
    out_dtype = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, T, n, 2), dtype=out_dtype, device=q.device)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device=q.device)
    _need_f32(S0=S0, S_T=S_T)
    _dtype_code(o)
    _check(dict(q=(q, (B, H, T, m, 2)), k=(k, (B, H, T, m, 2)), v=(v, (B, H, T, n, 2)),
                alpha=(alpha, (B, H, T, m)), theta=(theta, (B, H, T, m)), beta=(beta, (B, H, T)),
                S0=(S0, (B, H, m, n, 2)), o=(o, (B, H, T, n, 2)), S_T=(S_T, (B, H, m, n, 2)),
                workspace=(workspace, tuple(workspace.shape) if workspace is not None else ())))
    args = [_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(theta), _ptr(beta), _ptr(S0),
            _ptr(o), _ptr(S_T), B, H, T, m, n, C]
    if isinstance(segments, str):
        if segments != "auto":
            raise ValueError(f"segments must be an int, None or 'auto', not {segments!r}")
        segments = None
        if slice is None and q.is_cuda:
            with torch.cuda.device(q.device):
                G = int(lib.sfda_chunk_fwd_auto_segments(B, H, T, m, n, C, in_code))
            segments = G if G > 1 else None
    if segments is not None:
        nws = lib.sfda_chunk_fwd_segmented_workspace_bytes(B, H, T, m, n, segments, in_code)
        if workspace is None:
            workspace = torch.empty(max(nws, 1), dtype=torch.uint8, device=q.device)
        st = lib.sfda_chunk_fwd_segmented(*args, segments, in_code, _dtype_code(o), _ptr(workspace),
                                          workspace.numel() * workspace.element_size(), _stream(stream))
        if st != 0:
            raise SfdaError(st, "sfda_chunk_fwd_segmented")
        return o, S_T
    if slice is None:
        st = lib.sfda_chunk_fwd(*args, in_code, _dtype_code(o), _stream(stream))
    else:
        st = lib.sfda_chunk_fwd_sliced(*args, slice, in_code, _dtype_code(o), _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_chunk_fwd")
    return o, S_T


def chunk_fwd_segmented_noalloc(q, k, v, alpha, theta, beta, S0=None, C: int = 64, *, segments: int,
                                o=None, S_T=None, out_dtype=None, want_state: bool = True,
                                stream=None) -> Tuple:
    """chunk_fwd with `segments` parallel segments per head whose workspace is the library's
    static scratch (sfda_chunk_fwd_segmented_noalloc: the call allocates no device memory;
    o and S_T are allocated here only when not given).  Shapes and results as chunk_fwd."""
    import torch
    lib = load_library()
    B, H, T, m, _ = _dims(q, v, 5)
    n = v.shape[3]
    in_code = _dtype_code(q)
    for t in (k, v, alpha, theta, beta):
        if t.dtype != q.dtype:
            raise TypeError("q, k, v, alpha, theta, beta must share one dtype")
    out_dtype = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, T, n, 2), dtype=out_dtype, device=q.device)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device=q.device)
    _need_f32(S0=S0, S_T=S_T)
    _dtype_code(o)
    _check(dict(q=(q, (B, H, T, m, 2)), k=(k, (B, H, T, m, 2)), v=(v, (B, H, T, n, 2)),
                alpha=(alpha, (B, H, T, m)), theta=(theta, (B, H, T, m)), beta=(beta, (B, H, T)),
                S0=(S0, (B, H, m, n, 2)), o=(o, (B, H, T, n, 2)), S_T=(S_T, (B, H, m, n, 2))))
    st = lib.sfda_chunk_fwd_segmented_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(theta), _ptr(beta),
                                              _ptr(S0), _ptr(o), _ptr(S_T), B, H, T, m, n, C, segments,
                                              in_code, _dtype_code(o), _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_chunk_fwd_segmented_noalloc")
    return o, S_T


def chunk_fwd_gated(q, k_raw, v, a, b, c, S0=None, C: int = 64, *, alpha_min: float,
                    alpha_max: float, theta_max: float, eps: float, o=None, S_T=None,
                    out_dtype=None, want_state: bool = True, stream=None) -> Tuple:
    """SFDA chunkwise forward on pre-activations (sfda_chunk_fwd_gated): alpha, theta, beta
    and the keys are formed inside the kernel from a, b [B,H,T,m], c [B,H,T] and the raw
    keys k_raw [B,H,T,m,2].  Shapes and results otherwise as chunk_fwd."""
    import torch
    lib = load_library()
    B, H, T, m, _ = _dims(q, v, 5)
    n = v.shape[3]
    in_code = _dtype_code(q)
    for t in (k_raw, v, a, b, c):
        if t.dtype != q.dtype:
            raise TypeError("q, k_raw, v, a, b, c must share one dtype")
    out_dtype = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, T, n, 2), dtype=out_dtype, device=q.device)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device=q.device)
    _need_f32(S0=S0, S_T=S_T)
    _dtype_code(o)
    _check(dict(q=(q, (B, H, T, m, 2)), k_raw=(k_raw, (B, H, T, m, 2)), v=(v, (B, H, T, n, 2)),
                a=(a, (B, H, T, m)), b=(b, (B, H, T, m)), c=(c, (B, H, T)),
                S0=(S0, (B, H, m, n, 2)), o=(o, (B, H, T, n, 2)), S_T=(S_T, (B, H, m, n, 2))))
    st = lib.sfda_chunk_fwd_gated(_ptr(q), _ptr(k_raw), _ptr(v), _ptr(a), _ptr(b), _ptr(c), _ptr(S0),
                                  _ptr(o), _ptr(S_T), B, H, T, m, n, C, float(alpha_min),
                                  float(alpha_max), float(theta_max), float(eps), in_code,
                                  _dtype_code(o), _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_chunk_fwd_gated")
    return o, S_T


def chunk_fwd_decoupled(q, k, r, v, alpha, theta, eta, beta, S0=None, C: int = 32, *, o=None,
                        S_T=None, out_dtype=None, want_state: bool = True, stream=None) -> Tuple:
    """Write-decoupled forward (sfda_chunk_fwd_decoupled): erase along k with strengths eta
    [B,H,T], write along r [B,H,T,m,2] with strengths beta [B,H,T]; C 16 or 32.  Shapes and
    results otherwise as chunk_fwd."""
    import torch
    lib = load_library()
    B, H, T, m, _ = _dims(q, v, 5)
    n = v.shape[3]
    in_code = _dtype_code(q)
    for t in (k, r, v, alpha, theta, eta, beta):
        if t.dtype != q.dtype:
            raise TypeError("q, k, r, v, alpha, theta, eta, beta must share one dtype")
    out_dtype = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, T, n, 2), dtype=out_dtype, device=q.device)
    if S_T is None and want_state:
        S_T = torch.empty((B, H, m, n, 2), dtype=torch.float32, device=q.device)
    _need_f32(S0=S0, S_T=S_T)
    _dtype_code(o)
    _check(dict(q=(q, (B, H, T, m, 2)), k=(k, (B, H, T, m, 2)), r=(r, (B, H, T, m, 2)),
                v=(v, (B, H, T, n, 2)), alpha=(alpha, (B, H, T, m)), theta=(theta, (B, H, T, m)),
                eta=(eta, (B, H, T)), beta=(beta, (B, H, T)), S0=(S0, (B, H, m, n, 2)),
                o=(o, (B, H, T, n, 2)), S_T=(S_T, (B, H, m, n, 2))))
    st = lib.sfda_chunk_fwd_decoupled(_ptr(q), _ptr(k), _ptr(r), _ptr(v), _ptr(alpha), _ptr(theta), _ptr(eta),
                                      _ptr(beta), _ptr(S0), _ptr(o), _ptr(S_T), B, H, T, m, n, C, in_code,
                                      _dtype_code(o), _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_chunk_fwd_decoupled")
    return o, S_T


def chunk_bwd(q, k, v, alpha, theta, beta, S0, dO, dS_T=None, C: int = 64, *,
              want_dS0: bool = True, workspace=None, stream=None) -> dict:
    """Gradients of a real loss through the chunkwise forward (sfda_chunk_bwd), given
    dO = dL/do [B,H,T,n,2] (o's dtype) and dS_T = dL/dS_T [B,H,m,n,2] float32 or None.
    Inputs as chunk_fwd.  Returns dq, dk, dv, dalpha, dtheta, dbeta in the inputs' dtype and
    dS0 (float32, or None without want_dS0); complex gradients are dL/dRe + i dL/dIm.
    `workspace`: a uint8 device tensor of at least bwd_workspace_bytes(...) bytes, allocated
    here when not given."""
    import torch
    lib = load_library()
    B, H, T, m, _ = _dims(q, v, 5)
    n = v.shape[3]
    in_code = _dtype_code(q)
    for t in (k, v, alpha, theta, beta):
        if t.dtype != q.dtype:
            raise TypeError("q, k, v, alpha, theta, beta must share one dtype")
    _need_f32(S0=S0, dS_T=dS_T)
    _dtype_code(dO)
    _check(dict(q=(q, (B, H, T, m, 2)), k=(k, (B, H, T, m, 2)), v=(v, (B, H, T, n, 2)),
                alpha=(alpha, (B, H, T, m)), theta=(theta, (B, H, T, m)), beta=(beta, (B, H, T)),
                S0=(S0, (B, H, m, n, 2)), dO=(dO, (B, H, T, n, 2)), dS_T=(dS_T, (B, H, m, n, 2))))
    g = dict(dq=torch.empty_like(q), dk=torch.empty_like(k), dv=torch.empty_like(v),
             dalpha=torch.empty_like(alpha), dtheta=torch.empty_like(theta), dbeta=torch.empty_like(beta),
             dS0=torch.empty((B, H, m, n, 2), dtype=torch.float32, device=q.device) if want_dS0 else None)
    nws = lib.sfda_chunk_bwd_workspace_bytes(B, H, T, m, n, C)
    if workspace is None:
        workspace = torch.empty(max(nws, 1), dtype=torch.uint8, device=q.device)
    _check(dict(q=(q, (B, H, T, m, 2)), workspace=(workspace, tuple(workspace.shape))))
    st = lib.sfda_chunk_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(theta), _ptr(beta), _ptr(S0),
                            _ptr(dO), _ptr(dS_T), _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]),
                            _ptr(g["dalpha"]), _ptr(g["dtheta"]), _ptr(g["dbeta"]), _ptr(g["dS0"]),
                            B, H, T, m, n, C, in_code, _dtype_code(dO), _ptr(workspace),
                            workspace.numel() * workspace.element_size(), _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_chunk_bwd")
    return g


def bwd_workspace_bytes(B: int, H: int, T: int, m: int, n: int, C: int) -> int:
    return int(load_library().sfda_chunk_bwd_workspace_bytes(B, H, T, m, n, C))


def chunk_solve_monitor(k, alpha, theta, beta, stream=None) -> Tuple:
    """The triangular solve of every 16-token block checked on its own
    (sfda_chunk_solve_monitor): returns (residual, lnorm), float32 [B, H, ceil(T / 16)],
    the max-abs entry of (I + D_beta L') N - I and ||D_beta L'||_F.  k: [B,H,T,m,2];
    alpha, theta: [B,H,T,m]; beta: [B,H,T] (float32 or bfloat16)."""
    import torch
    lib = load_library()
    if k.dim() != 5 or k.shape[-1] != 2:
        raise ValueError(f"k must be [B,H,T,m,2], not {tuple(k.shape)}")
    B, H, T, m = k.shape[0], k.shape[1], k.shape[2], k.shape[3]
    code = _dtype_code(k)
    for t in (alpha, theta, beta):
        if t.dtype != k.dtype:
            raise TypeError("k, alpha, theta, beta must share one dtype")
    _check(dict(k=(k, (B, H, T, m, 2)), alpha=(alpha, (B, H, T, m)), theta=(theta, (B, H, T, m)),
                beta=(beta, (B, H, T))))
    nb = (T + 15) // 16
    residual = torch.empty((B, H, nb), dtype=torch.float32, device=k.device)
    lnorm = torch.empty((B, H, nb), dtype=torch.float32, device=k.device)
    st = lib.sfda_chunk_solve_monitor(_ptr(k), _ptr(alpha), _ptr(theta), _ptr(beta), _ptr(residual),
                                      _ptr(lnorm), B, H, T, m, code, _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_chunk_solve_monitor")
    return residual, lnorm


def auto_segments(B: int, H: int, T: int, m: int, n: int, C: int = 64, dtype: str = "f32") -> int:
    """sfda_chunk_fwd_auto_segments on the current device (1: one scan per head); dtype: the
    inputs' ("f32" or "bf16")."""
    code = {"f32": SFDA_F32, "bf16": SFDA_BF16}[dtype]
    return int(load_library().sfda_chunk_fwd_auto_segments(B, H, T, m, n, C, code))


def segmented_workspace_bytes(B: int, H: int, T: int, m: int, n: int, G: int, dtype: str = "f32") -> int:
    """Workspace of sfda_chunk_fwd_segmented; dtype: the inputs' ("f32" or "bf16")."""
    code = {"f32": SFDA_F32, "bf16": SFDA_BF16}[dtype]
    return int(load_library().sfda_chunk_fwd_segmented_workspace_bytes(B, H, T, m, n, G, code))


def step(q, k, v, alpha, theta, beta, S, *, o=None, out_dtype=None, stream=None):
    """One decode token per head.  q, k: [B,H,m,2]; v: [B,H,n,2]; alpha, theta: [B,H,m];
    beta: [B,H]; S: [B,H,m,n,2] float32, updated in place.  Returns o [B,H,n,2]."""
    import torch
    lib = load_library()
    B, H, m, _ = _dims(q, v, 4)
    n = v.shape[2]
    in_code = _dtype_code(q)
    for t in (k, v, alpha, theta, beta):
        if t.dtype != q.dtype:
            raise TypeError("q, k, v, alpha, theta, beta must share one dtype")
    _need_f32(S=S)
    out_dtype = q.dtype if out_dtype is None else out_dtype
    if o is None:
        o = torch.empty((B, H, n, 2), dtype=out_dtype, device=q.device)
    _dtype_code(o)
    _check(dict(q=(q, (B, H, m, 2)), k=(k, (B, H, m, 2)), v=(v, (B, H, n, 2)), alpha=(alpha, (B, H, m)),
                theta=(theta, (B, H, m)), beta=(beta, (B, H)), S=(S, (B, H, m, n, 2)), o=(o, (B, H, n, 2))))
    st = lib.sfda_step(_ptr(q), _ptr(k), _ptr(v), _ptr(alpha), _ptr(theta), _ptr(beta),
                       _ptr(S), _ptr(o), B, H, m, n, in_code, _dtype_code(o), _stream(stream))
    if st != 0:
        raise SfdaError(st, "sfda_step")
    return o
