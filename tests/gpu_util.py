"""Helpers shared by the GPU tests: device transfer of the seeded inputs and
the parity measures (relative Frobenius errors per matrix)."""
from __future__ import annotations

import functools

import numpy as np
import pytest

from oracle import muon_ref as ref

# Official gates (relative Frobenius error per matrix).
TOL = {"bf16": 2e-2, "f32": 1e-4}
MOMENTUM_TOL = 1e-6   # fp32 FMA against fp64


@functools.lru_cache(maxsize=None)
def _worst_storage_error(shape, ns_steps, coeffs):
    from tests.bf16_pipeline import worst_storage_error
    return worst_storage_error(shape, ns_steps, None if coeffs is None else [list(r) for r in coeffs])


def tol_for(prec: str, shape, ns_steps: int = 5, coeffs=None, G=None) -> float:
    """Gate for one matrix.  The flat gates of the target, except on the bf16
    path for a short side below 16: there a few singular values take every
    bf16 rounding coherently, and the gate is 1.25 times the worst error that
    bf16 storage alone reaches on that shape and on the tested input G
    (tests/bf16_pipeline.py, a CPU emulation of the bf16 pipeline measured
    against the oracle), never below 2e-2."""
    shape = tuple(int(v) for v in shape[-2:])
    if prec == "bf16" and min(shape) < 16:
        from tests.bf16_pipeline import FEW_SV_MARGIN, storage_error
        key = None if coeffs is None else tuple(tuple(float(v) for v in r) for r in coeffs)
        worst = _worst_storage_error(shape, ns_steps, key)
        if G is not None:
            worst = max(worst, storage_error(np.asarray(G, dtype=np.float64), ns_steps, coeffs))
        return max(TOL["bf16"], FEW_SV_MARGIN * worst)
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


def o_gate(O_gpu, O_ref, dtype, prec, ns_steps: int = 5, coeffs=None, G=None):
    """(error, gate) for an orthogonalised output stored in `dtype` from NS
    in precision `prec` on input G: the gate of `prec` (tol_for), plus the
    storage floor ||round(O_ref) - O_ref|| / ||O_ref|| only where the output
    is stored coarser than the NS precision (bf16 output of fp32 NS)."""
    err = rel(O_gpu, O_ref)
    gate = tol_for(prec, np.shape(O_ref), ns_steps, coeffs, G)
    if dtype == "bf16" and prec == "f32":
        gate += rel(ref.round_to(O_ref, dtype), O_ref)
    return err, gate
