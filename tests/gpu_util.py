"""Helpers shared by the GPU tests: upload stored inputs, run the library, compare with the
oracle.  The error measure is max |x - ref| / max |ref| over a whole tensor."""
from __future__ import annotations

import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2607_11897_amd import inputs as I  # noqa: E402


def ensure_built():
    from paper_2607_11897_amd import build, sfda
    if not os.path.exists(sfda.LIB_PATH):
        build.build(verbose=False)
    return sfda.load_library()


def to_device(a: np.ndarray, dtype: str, device="cuda"):
    """Stored numpy buffer (float32 or bf16 bits as uint16) -> torch tensor on the device."""
    import torch
    if a is None:
        return None
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


def upload(x: "I.ChunkInputs", device="cuda"):
    st = x.storage()
    d = {k: to_device(st[k], x.dtype, device) for k in ("q", "k", "v", "alpha", "theta", "beta")}
    d["S0"] = None if st["S0"] is None else to_device(st["S0"], "f32", device)
    return d


def to_complex(t) -> np.ndarray:
    a = t.float().cpu().numpy().astype(np.float64)
    return a[..., 0] + 1j * a[..., 1]


def rel_err(x: np.ndarray, ref: np.ndarray) -> float:
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    num = float(np.max(np.abs(x - ref))) if ref.size else 0.0
    return num / den if den > 0 else num


def run_chunk(x: "I.ChunkInputs", C: int, out_dtype=None, slice=None, device="cuda", segments="auto"):
    import torch
    from paper_2607_11897_amd import sfda
    d = upload(x, device)
    od = None if out_dtype is None else {"f32": torch.float32, "bf16": torch.bfloat16}[out_dtype]
    o, S = sfda.chunk_fwd(d["q"], d["k"], d["v"], d["alpha"], d["theta"], d["beta"], d["S0"],
                          C=C, out_dtype=od, slice=slice, segments=segments)
    torch.cuda.synchronize()
    return to_complex(o), to_complex(S)


def run_oracle(x: "I.ChunkInputs"):
    import oracle
    return oracle.recurrence(x.q, x.k, x.v, x.alpha, x.theta, x.beta, x.S0)
