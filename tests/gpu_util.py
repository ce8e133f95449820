"""Helpers shared by the GPU tests: device transfer of the seeded inputs and
the parity measures (relative Frobenius errors per matrix)."""
from __future__ import annotations

import numpy as np
import pytest

from oracle import muon_ref as ref

# Official gates (relative Frobenius error per matrix).
TOL = {"bf16": 2e-2, "f32": 1e-4}
MOMENTUM_TOL = 1e-6   # fp32 FMA against fp64
# bf16 storage of X, A and B rounds each stage to 8 significant bits (unit
# roundoff u = 2^-9).  With many singular values the rounding errors average
# out and the error stays near 1.1-1.4e-2; a matrix whose short side is tiny
# has one or a few singular values that absorb every rounding coherently:
# four roundings per step over K = 5 steps bound it by 4*K*u = 3.9e-2.
BF16_FEW_SV_TOL = 4 * 5 * 2.0 ** -9


def tol_for(prec: str, shape) -> float:
    if prec == "bf16" and min(shape[-2:]) < 16:
        return BF16_FEW_SV_TOL
    return TOL[prec]


def require_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    from paper_2609_21594_amd import binding
    binding.load_library()  # raises when the HIP library is missing
    return torch


def to_dev(a, dtype: str):
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint16).view(np.int16)).view(torch.bfloat16)
    elif dtype == "f32":
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    else:
        raise ValueError(dtype)
    return t.cuda()


def to_host(t) -> np.ndarray:
    """Exact fp64 copy of a device tensor (bf16 or fp32)."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return ref.decode_bf16(t.view(torch.int16).numpy().view(np.uint16))
    return t.numpy().astype(np.float64)


def to_bits(t) -> np.ndarray:
    """Raw bits of a device tensor, for bitwise comparisons."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().copy()
    return t.view(torch.int32).numpy().copy()


def decode(a, dtype: str) -> np.ndarray:
    return ref.decode_bf16(a) if dtype == "bf16" else np.asarray(a, dtype=np.float64)


def rel(a, b) -> float:
    nb = float(np.linalg.norm(b))
    return float(np.linalg.norm(np.asarray(a) - np.asarray(b))) / (nb if nb > 0 else 1.0)


def w_gate(W_gpu, W_ref, W0, dtype):
    """(error, floor): ||W_gpu - W_ref|| / ||W_ref - W0|| and the storage
    rounding floor ||round(W_ref) - W_ref|| / ||W_ref - W0||."""
    d = float(np.linalg.norm(W_ref - W0))
    err = float(np.linalg.norm(W_gpu - W_ref)) / d
    rho = float(np.linalg.norm(ref.round_to(W_ref, dtype) - W_ref)) / d
    return err, rho


def o_gate(O_gpu, O_ref, dtype):
    """(error, floor) for an orthogonalised output stored in `dtype`."""
    err = rel(O_gpu, O_ref)
    rho = rel(ref.round_to(O_ref, dtype), O_ref)
    return err, rho
