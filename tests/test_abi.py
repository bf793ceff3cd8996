"""The C-ABI library loads and exports what include/sfda.h declares, and its argument checks
return the documented status codes before anything is launched (CPU only: these calls
never reach the GPU, the pointers are never dereferenced)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

from gpu_util import ROOT, ensure_built

HEADER = os.path.join(ROOT, "include", "sfda.h")


@pytest.fixture(scope="module")
def lib():
    return ensure_built()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sfda_\w+)\s*\(", src)))


def test_header_declares_expected_api():
    names = declared_functions()
    from paper_2607_11897_amd import sfda
    assert set(names) == set(sfda.EXPORTS), names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_abi_version_and_status_strings(lib):
    assert lib.sfda_abi_version() == 3
    for s in range(9):
        assert len(lib.sfda_status_string(s)) > 0
    assert lib.sfda_status_string(99) == b"unknown status"


A = 1 << 20          # fake, 16-byte aligned device addresses, spaced far apart
P = [A * (i + 1) for i in range(9)]


def chunk(lib, q=P[0], k=P[1], v=P[2], a=P[3], th=P[4], b=P[5], s0=P[6], o=P[7], st=P[8],
          B=1, H=1, T=4, m=8, n=8, C=16, din=0, dout=0):
    return lib.sfda_chunk_fwd(q, k, v, a, th, b, s0, o, st, B, H, T, m, n, C, din, dout, None)


def step(lib, q=P[0], k=P[1], v=P[2], a=P[3], th=P[4], b=P[5], S=P[6], o=P[7],
         B=1, H=1, m=8, n=8, din=0, dout=0):
    return lib.sfda_step(q, k, v, a, th, b, S, o, B, H, m, n, din, dout, None)


def test_chunk_argument_errors(lib):
    assert chunk(lib, q=None) == 1
    assert chunk(lib, o=None) == 1
    assert chunk(lib, m=0) == 2 and chunk(lib, m=65) == 2 and chunk(lib, n=0) == 2
    assert chunk(lib, T=-1) == 2 and chunk(lib, B=-1) == 2
    assert chunk(lib, C=8) == 3 and chunk(lib, C=256) == 3 and chunk(lib, C=48) == 3
    assert chunk(lib, din=2) == 4 and chunk(lib, dout=-1) == 4
    assert chunk(lib, q=P[0] + 8) == 5
    assert chunk(lib, o=P[0]) == 6                    # o on top of q
    assert chunk(lib, st=P[3] + 64) == 6              # S_T inside alpha
    assert chunk(lib, st=P[6] + 16) == 6              # S_T partly overlapping S0
    assert lib.sfda_chunk_fwd_sliced(*P, 1, 1, 4, 8, 8, 16, 12, 0, 0, None) == 2   # slice % 8
    assert lib.sfda_chunk_fwd_sliced(*P, 1, 1, 4, 8, 8, 16, 72, 0, 0, None) == 2
    # bf16 inputs: each head's share of q, k, v and o below 2 GiB (32-bit buffer ranges);
    # with m = n = 64 and bf16 o the longest head is (2^31 - 1) // 256 = 8388607 tokens
    Pf = [1 << 44 + i for i in range(9)]      # addresses far enough apart for 2 GiB buffers
    big = dict(zip(("q", "k", "v", "a", "th", "b", "s0", "o", "st"), Pf))
    assert chunk(lib, T=8388608, m=64, n=64, din=1, dout=1, **big) == 2
    assert chunk(lib, T=4194304, m=64, n=64, din=1, dout=0, **big) == 2    # fp32 o
    # the float32 kernels address one chunk's rows of v and o (at most 32 tokens) with 32-bit
    # byte offsets: 32 * n * 8 < 2^31 (n = 2^23 is refused, though m * n * 8 < 2^31 with m = 1)
    assert chunk(lib, T=64, m=1, n=1 << 23, C=64, **big) == 2
    # B*H == 0 is a no-op and never touches the pointers
    assert chunk(lib, B=0, q=None, o=None) == 0


def seg(lib, T=64, G=2, C=16, ws=A * 20, nws=1 << 40, q=P[0], B=1, H=1, m=8, n=8, din=0):
    return lib.sfda_chunk_fwd_segmented(q, *P[1:], B, H, T, m, n, C, G, din, 0, ws, nws, None)


def test_segmented_workspace_size(lib):
    # per segment: P_g (m x m) + B_g and the incoming state (m x n); per head and token X_t
    # (m)
    # (float32 inputs), complex float32
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(2, 3, 256, 64, 48, 4, 0) == \
        (24 * (64 * 64 + 2 * 64 * 48) + 6 * 256 * 64) * 8
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(2, 3, 256, 64, 48, 4, 1) == 24 * (64 * 64 + 2 * 64 * 48) * 8
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(1, 1, 64, 65, 8, 1, 0) == 0
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(1, 1, 64, 8, 8, 0, 0) == 0
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(1, 1, -1, 8, 8, 1, 0) == 0
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(1, 1, 64, 8, 8, 1, 2) == 0


def noalloc(lib, T=64, G=2, C=16, q=P[0], B=1, H=1, m=8, n=8, din=0):
    return lib.sfda_chunk_fwd_segmented_noalloc(q, *P[1:], B, H, T, m, n, C, G, din, 0, None)


def test_noalloc_argument_errors(lib):
    """The allocation-free segmented entry point validates every argument before it touches
    the device, and refuses a workspace beyond its static scratch (CPU only)."""
    assert noalloc(lib, G=0) == 2
    assert noalloc(lib, T=48, G=2, C=16) == 2
    assert noalloc(lib, q=None) == 1
    assert noalloc(lib, C=8) == 3 and noalloc(lib, din=3) == 4
    assert noalloc(lib, B=0, q=None) == 0
    # 64 heads x 8 segments x (64 x 64 + 2 x 64 x 64) complex float32 = 48 MiB > 32 MiB
    assert lib.sfda_chunk_fwd_segmented_workspace_bytes(1, 64, 8 * 16, 64, 64, 8, 0) > (32 << 20)
    assert noalloc(lib, T=8 * 16, G=8, H=64, m=64, n=64) == 8
    assert lib.sfda_status_string(8).startswith(b"the call needs more workspace")


def test_segmented_argument_errors(lib):
    assert seg(lib, G=0) == 2
    assert seg(lib, T=48, G=2, C=16) == 2             # T not a multiple of G * C
    assert seg(lib, ws=None) == 1
    assert seg(lib, ws=A * 20 + 8) == 5
    assert seg(lib, nws=100) == 2                     # workspace too small
    assert seg(lib, ws=P[2]) == 6                     # workspace on top of v
    assert seg(lib, q=None) == 1
    assert seg(lib, C=8) == 3 and seg(lib, din=3) == 4
    assert seg(lib, B=0, q=None, ws=None) == 0        # nothing to do


def gated(lib, amin=0.9, amax=1.0, tmax=0.5, eps=0.0, C=16, q=P[0]):
    f = ctypes.c_float
    return lib.sfda_chunk_fwd_gated(q, *P[1:], 1, 1, 4, 8, 8, C, f(amin), f(amax), f(tmax), f(eps),
                                    0, 0, None)


def test_gated_argument_errors(lib):
    assert gated(lib, amin=0.0) == 2                   # alpha must stay positive
    assert gated(lib, amin=0.0042) == 2                # alpha_min^16 < 2^-126: outside the block range
    assert gated(lib, amin=0.95, amax=0.9) == 2
    assert gated(lib, amax=1.5) == 2
    assert gated(lib, tmax=-0.1) == 2
    assert gated(lib, eps=float("nan")) == 2 and gated(lib, tmax=float("inf")) == 2
    assert gated(lib, q=None) == 1 and gated(lib, C=8) == 3


def test_step_argument_errors(lib):
    assert step(lib, S=None) == 1
    assert step(lib, m=0) == 2 and step(lib, m=65) == 2 and step(lib, n=0) == 2
    assert step(lib, n=1 << 22) == 2                  # state rows use 32-bit offsets
    assert step(lib, din=5) == 4
    assert step(lib, v=P[2] + 4) == 5
    assert step(lib, o=P[6]) == 6                     # o on top of S
    assert step(lib, S=P[0]) == 6                     # S on top of q
    assert step(lib, H=0) == 0


def test_binding_fails_loudly_without_library(tmp_path):
    from paper_2607_11897_amd import sfda
    with pytest.raises(RuntimeError):
        old = sfda._lib
        sfda._lib = None
        try:
            sfda.load_library(str(tmp_path / "missing.so"))
        finally:
            sfda._lib = old


# --------------------------------------------------------------------------- backward
PB = [A * (i + 1) for i in range(17)]       # 16 tensors + workspace


def bwd(lib, ptrs=None, B=1, H=1, T=40, m=8, n=8, C=16, din=0, dout=0, ws_bytes=None):
    p = list(PB if ptrs is None else ptrs)
    need = lib.sfda_chunk_bwd_workspace_bytes(max(B, 1), max(H, 1), T, m, n, C)
    ws = need if ws_bytes is None else ws_bytes
    return lib.sfda_chunk_bwd(*p[:16], B, H, T, m, n, C, din, dout, p[16], ws, None)


def test_bwd_workspace_bytes(lib):
    # per chunk: two m x n and two C x n complex float32 blocks; every C runs 16-token chunks
    assert lib.sfda_chunk_bwd_workspace_bytes(8, 16, 4096, 64, 64, 16) == 8 * 16 * 256 * (2 * 64 * 64 + 2 * 16 * 64) * 8
    for C in (32, 64, 128):
        assert lib.sfda_chunk_bwd_workspace_bytes(8, 16, 4096, 64, 64, C) == \
            lib.sfda_chunk_bwd_workspace_bytes(8, 16, 4096, 64, 64, 16)
    assert lib.sfda_chunk_bwd_workspace_bytes(1, 1, 65, 8, 8, 64) == 5 * (2 * 8 * 8 + 2 * 16 * 8) * 8
    assert lib.sfda_chunk_bwd_workspace_bytes(1, 1, 65, 8, 8, 16) == 5 * (2 * 8 * 8 + 2 * 16 * 8) * 8
    assert lib.sfda_chunk_bwd_workspace_bytes(1, 1, 0, 8, 8, 16) == 0
    for bad in [(0, 1, 4, 8, 8, 16), (1, 1, 4, 65, 8, 16), (1, 1, 4, 8, 0, 16), (1, 1, 4, 8, 8, 48)]:
        assert lib.sfda_chunk_bwd_workspace_bytes(*bad) == 0


def test_bwd_argument_errors(lib):
    assert bwd(lib, B=0) == 0                                  # nothing to do
    assert bwd(lib, C=48) == 3
    assert bwd(lib, din=5) == 4
    assert bwd(lib, m=65) == 2
    assert bwd(lib, T=-1) == 2
    assert bwd(lib, m=1, n=1 << 23, C=64) == 2                 # 32 * n * 8 >= 2^31 (32-bit row offsets)
    for idx in list(range(6)) + [7] + list(range(9, 15)):     # required: inputs, dO, gradients
        p = list(PB)
        p[idx] = 0
        assert bwd(lib, p) == 1, idx
    p = list(PB)
    p[16] = 0
    assert bwd(lib, p) == 1                                    # workspace needed
    p = list(PB)
    p[9] += 8
    assert bwd(lib, p) == 5                                    # misaligned dq
    assert bwd(lib, ws_bytes=100) == 2                         # workspace too small
    p = list(PB)
    p[9] = p[0]
    assert bwd(lib, p) == 6                                    # dq over q
    p = list(PB)
    p[16] = p[12]
    assert bwd(lib, p) == 6                                    # workspace over dtheta
    p = list(PB)
    p[15] = p[8]
    assert bwd(lib, p) == 6                                    # dS0 over dS_T


def test_decoupled_argument_errors(lib):
    def dec(q=P[0], k=P[1], r=A * 20, v=P[2], a=P[3], th=P[4], eta=P[5], b=A * 21, s0=P[6], o=P[7], st=P[8],
            B=1, H=1, T=4, m=8, n=8, C=16, din=0, dout=0):
        return lib.sfda_chunk_fwd_decoupled(q, k, r, v, a, th, eta, b, s0, o, st, B, H, T, m, n, C, din, dout, None)
    assert dec(B=0) == 0
    assert dec(C=256) == 3
    assert dec(C=48) == 3
    assert dec(r=0) == 1
    assert dec(b=0) == 1
    assert dec(eta=0) == 1
    assert dec(b=A * 21 + 4) == 5
    assert dec(o=A * 20) == 6          # o over r
    assert dec(st=A * 21) == 6         # S_T over beta
    assert dec(m=65) == 2


def test_binding_checks_shapes_and_devices(lib):
    """The ctypes binding refuses tensors whose shapes do not match q's sizes and host
    tensors before any call reaches the library (CPU only)."""
    import torch
    from paper_2607_11897_amd import sfda
    B, H, T, m, n = 1, 2, 8, 8, 4
    q = torch.zeros(B, H, T, m, 2)
    k = torch.zeros(B, H, T, m, 2)
    v = torch.zeros(B, H, T, n, 2)
    a = torch.ones(B, H, T, m)
    th = torch.zeros(B, H, T, m)
    b = torch.zeros(B, H, T)
    with pytest.raises(ValueError, match="shape"):
        sfda.chunk_fwd(q, k[:, :, :4], v, a, th, b, C=16)
    with pytest.raises(ValueError, match="shape"):
        sfda.chunk_fwd(q, k, v, a, th, b, torch.zeros(B, H, m, n + 1, 2), C=16)
    with pytest.raises(ValueError, match="shape"):
        sfda.chunk_fwd(q, k, v, a, th, b, C=16, o=torch.zeros(B, H, T - 1, n, 2))
    with pytest.raises(ValueError, match="GPU tensor"):
        sfda.chunk_fwd(q, k, v, a, th, b, C=16)
    with pytest.raises(ValueError, match="shape"):
        sfda.step(q[:, :, 0], k[:, :, 0], v[:, :, 0], a[:, :, 0], th[:, :, 0], b[:, :, 0],
                  torch.zeros(B, H, m, n, 2), o=torch.zeros(B, H, n + 1, 2))
    with pytest.raises(ValueError, match="GPU tensor"):
        sfda.step(q[:, :, 0], k[:, :, 0], v[:, :, 0], a[:, :, 0], th[:, :, 0], b[:, :, 0],
                  torch.zeros(B, H, m, n, 2))
    with pytest.raises(ValueError, match="shape"):
        sfda.chunk_bwd(q, k, v, a, th, b, None, torch.zeros(B, H, T, n + 1, 2), C=16)


def test_binding_checks_state_and_output_dtypes(lib):
    """A caller-supplied S_T (or S, dS_T) of half width would be overrun by the library's
    m * n * 8 bytes per head; the binding refuses it, and an o of an unsupported dtype,
    before any call (CPU only)."""
    import torch
    from paper_2607_11897_amd import sfda
    B, H, T, m, n = 1, 2, 8, 8, 4
    q = torch.zeros(B, H, T, m, 2)
    k = torch.zeros(B, H, T, m, 2)
    v = torch.zeros(B, H, T, n, 2)
    a = torch.ones(B, H, T, m)
    th = torch.zeros(B, H, T, m)
    b = torch.zeros(B, H, T)
    half_state = torch.zeros(B, H, m, n, 2, dtype=torch.bfloat16)
    with pytest.raises(TypeError, match="S_T must be float32"):
        sfda.chunk_fwd(q, k, v, a, th, b, C=16, S_T=half_state)
    with pytest.raises(TypeError, match="S0 must be float32"):
        sfda.chunk_fwd(q, k, v, a, th, b, half_state, C=16)
    with pytest.raises(TypeError, match="S_T must be float32"):
        sfda.chunk_fwd_gated(q, k, v, a, th, b, C=16, alpha_min=0.5, alpha_max=1.0, theta_max=1.0,
                             eps=0.0, S_T=half_state)
    with pytest.raises(TypeError, match="S_T must be float32"):
        sfda.chunk_fwd_decoupled(q, k, k, v, a, th, b, b, C=16, S_T=half_state)
    with pytest.raises(TypeError, match="unsupported dtype"):
        sfda.chunk_fwd(q, k, v, a, th, b, C=16, o=torch.zeros(B, H, T, n, 2, dtype=torch.float16))
    with pytest.raises(TypeError, match="dS_T must be float32"):
        sfda.chunk_bwd(q, k, v, a, th, b, None, torch.zeros(B, H, T, n, 2), half_state, C=16)
    with pytest.raises(TypeError, match="S must be float32"):
        sfda.step(q[:, :, 0], k[:, :, 0], v[:, :, 0], a[:, :, 0], th[:, :, 0], b[:, :, 0], half_state)
    with pytest.raises(TypeError, match="unsupported dtype"):
        sfda.step(q[:, :, 0], k[:, :, 0], v[:, :, 0], a[:, :, 0], th[:, :, 0], b[:, :, 0],
                  torch.zeros(B, H, m, n, 2), o=torch.zeros(B, H, n, 2, dtype=torch.float16))


def monitor(lib, k=P[1], a=P[3], th=P[4], b=P[5], res=P[6], ln=P[7], B=1, H=1, T=32, m=8, din=0):
    return lib.sfda_chunk_solve_monitor(k, a, th, b, res, ln, B, H, T, m, din, None)


def test_solve_monitor_argument_errors(lib):
    assert monitor(lib, din=2) == 4
    assert monitor(lib, m=0) == 2 and monitor(lib, m=65) == 2 and monitor(lib, T=-1) == 2
    assert monitor(lib, k=None) == 1 and monitor(lib, res=None, ln=None) == 1
    assert monitor(lib, k=P[1] + 4) == 5
    assert monitor(lib, res=P[1]) == 6            # over k
    assert monitor(lib, ln=P[6]) == 6             # over residual
    assert monitor(lib, B=0, k=None) == 0 and monitor(lib, T=0, k=None) == 0
