"""Seeded synthetic inputs for the Muon-step workloads.

This module is shared by the tests, the benchmark and the smoke check: both
the HIP path and the CPU oracle consume exactly the bits it produces.  It
holds no step of the Muon method itself, only the workload shapes, the
random draws and their conversion to the storage types.

Every array comes from its own PCG64 stream seeded with
SeedSequence([260921594, workload, step, matrix index, kind]), kind 0 = the
parameter W, 1 = the gradient g, 2 = the momentum buffer.  Values are drawn
as binary32 standard normals times sigma (binary32 product); bf16 arrays are
those binary32 values rounded to bfloat16 (nearest, ties to even) and are
returned as uint16 bit patterns.

Workloads (shapes are [rows, cols] = [out_features, in_features]):

1. one 256x128 fp32 matrix; W, g, momentum ~ N(0, 1); beta 0.95 Nesterov,
   lr 0.02, wd 0; 5 fp32 Newton-Schulz steps; one step;
2. one transformer block, hidden 2048, FFN 5632 (Q, K, V, O 2048x2048; gate,
   up 5632x2048; down 2048x5632); bf16 W and g ~ N(0, 0.02); fp32 momentum
   starting at zero; three steps with a fresh gradient each step;
3. a 7B-like per-device share: 8 layers of hidden 4096, FFN 11008 (56
   matrices); bf16 g ~ N(0, 1e-3), fp32 momentum ~ N(0, 1e-3), bf16 W ~
   N(0, 0.02); one step;
4. a mixed-shape batch: 96 x 1024x4096, 96 x 4096x1024, 256 x 512x512,
   64 x 128x2048, in that order; bf16 entries ~ N(0, 1), every 7th matrix
   (0-based index i with (i+1) % 7 == 0) scaled by 1e-4; these are the inputs
   of a standalone batched orthogonalisation;
5. a 70B-like per-device share: 4 layers of hidden 8192, FFN 28672 with GQA
   K/V 1024x8192 (28 matrices); bf16 g ~ N(0, 1e-3), fp32 momentum ~
   N(0, 1e-3), bf16 W ~ N(0, 0.02); one step.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

ROOT_SEED = 260921594
KIND_PARAM, KIND_GRAD, KIND_MOMENTUM = 0, 1, 2


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    rows: int
    cols: int
    batch: int = 1          # > 1: an [E, rows, cols] stack of independent matrices
    scale: float = 1.0      # extra factor on the draw (workload 4's 1e-4 matrices)

    @property
    def numel(self) -> int:
        return self.batch * self.rows * self.cols


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    matrices: Sequence[MatrixSpec]
    param_dtype: str          # "bf16" | "f32"
    grad_dtype: str
    ns_precision: str         # "bf16" | "f32"
    sigma_param: float
    sigma_grad: float
    sigma_momentum: float     # 0 -> momentum starts at zero
    steps: int = 1
    lr: float = 0.02
    beta: float = 0.95
    weight_decay: float = 0.0
    ns_steps: int = 5
    nesterov: bool = True
    orthogonalize_only: bool = False   # workload 4: inputs of the standalone NS

    @property
    def n_matrices(self) -> int:
        return sum(m.batch for m in self.matrices)


def _layers(n_layers: int, hidden: int, ffn: int, kv: Optional[int] = None) -> List[MatrixSpec]:
    kv = hidden if kv is None else kv
    out: List[MatrixSpec] = []
    for layer in range(n_layers):
        p = f"l{layer}."
        out += [MatrixSpec(p + "q", hidden, hidden), MatrixSpec(p + "k", kv, hidden),
                MatrixSpec(p + "v", kv, hidden), MatrixSpec(p + "o", hidden, hidden),
                MatrixSpec(p + "gate", ffn, hidden), MatrixSpec(p + "up", ffn, hidden),
                MatrixSpec(p + "down", hidden, ffn)]
    return out


def _mixed() -> List[MatrixSpec]:
    shapes = [(1024, 4096)] * 96 + [(4096, 1024)] * 96 + [(512, 512)] * 256 + [(128, 2048)] * 64
    return [MatrixSpec(f"m{i}", r, c, 1, 1e-4 if (i + 1) % 7 == 0 else 1.0)
            for i, (r, c) in enumerate(shapes)]


WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "single-256x128-fp32", [MatrixSpec("w", 256, 128)], "f32", "f32", "f32",
                1.0, 1.0, 1.0),
    2: Workload(2, "block-h2048-ffn5632-3steps", _layers(1, 2048, 5632), "bf16", "bf16", "bf16",
                0.02, 0.02, 0.0, steps=3),
    3: Workload(3, "7b-share-8x(h4096,ffn11008)", _layers(8, 4096, 11008), "bf16", "bf16", "bf16",
                0.02, 1e-3, 1e-3),
    4: Workload(4, "mixed-512-grouped", _mixed(), "bf16", "bf16", "bf16",
                1.0, 1.0, 0.0, orthogonalize_only=True),
    5: Workload(5, "70b-share-4x(h8192,ffn28672,kv1024)", _layers(4, 8192, 28672, kv=1024),
                "bf16", "bf16", "bf16", 0.02, 1e-3, 1e-3),
}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """binary32 -> bfloat16 bit patterns, round to nearest even (finite input)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def rng_for(workload: int, step: int, index: int, kind: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([ROOT_SEED, workload, step, index, kind])))


def draw(shape, sigma: float, dtype: str, rng: np.random.Generator,
         extra_scale: float = 1.0) -> np.ndarray:
    """N(0, sigma^2) draw in the storage dtype ("f32" array or "bf16" bits)."""
    x = rng.standard_normal(shape, dtype=np.float32)
    x *= np.float32(sigma)
    if extra_scale != 1.0:
        x *= np.float32(extra_scale)
    if dtype == "f32":
        return x
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    raise ValueError(dtype)


@dataclass
class MatrixInputs:
    spec: MatrixSpec
    W: Optional[np.ndarray]      # param (bf16 bits or f32), None for orthogonalize-only
    g: np.ndarray                # gradient / NS input (bf16 bits or f32)
    buf: Optional[np.ndarray]    # fp32 momentum, None for orthogonalize-only


def _shape(spec: MatrixSpec):
    return (spec.rows, spec.cols) if spec.batch == 1 else (spec.batch, spec.rows, spec.cols)


def make_matrix(wl: Workload, index: int, step: int = 0, with_state: bool = True) -> MatrixInputs:
    """Inputs of matrix `index` at `step`.  W and the momentum are drawn at
    step 0 only (later steps carry state); gradients are fresh every step."""
    spec = wl.matrices[index]
    shp = _shape(spec)
    g = draw(shp, wl.sigma_grad, wl.grad_dtype, rng_for(wl.index, step, index, KIND_GRAD),
             spec.scale)
    if wl.orthogonalize_only or not with_state:
        return MatrixInputs(spec, None, g, None)
    W = draw(shp, wl.sigma_param, wl.param_dtype, rng_for(wl.index, 0, index, KIND_PARAM))
    if wl.sigma_momentum == 0.0:
        buf = np.zeros(shp, dtype=np.float32)
    else:
        buf = draw(shp, wl.sigma_momentum, "f32", rng_for(wl.index, 0, index, KIND_MOMENTUM))
    return MatrixInputs(spec, W, g, buf)


def make_workload(wl: Workload, step: int = 0, with_state: bool = True,
                  indices: Optional[Sequence[int]] = None,
                  threads: Optional[int] = None) -> List[MatrixInputs]:
    """All (or the listed) matrices of a workload, generated in parallel
    threads (NumPy's bulk draws release the GIL; every matrix has its own
    stream, so the result does not depend on the thread count)."""
    idx = list(range(len(wl.matrices))) if indices is None else list(indices)
    threads = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(max_workers=threads) as ex:
        return list(ex.map(lambda i: make_matrix(wl, i, step, with_state), idx))


# --------------------------------------------------------------------------
# Work accounting for the measurement (shapes only)
# --------------------------------------------------------------------------
def ns_dense_flops(rows: int, cols: int, ns_steps: int) -> float:
    """Dense flop count of ns_steps Newton-Schulz steps on the short-side-first
    matrix s x l: X X^T (2 s^2 l) + A A (2 s^3) + B X (2 s^2 l) per step."""
    s, l = min(rows, cols), max(rows, cols)
    return float(ns_steps) * (4.0 * s * s * l + 2.0 * float(s) ** 3)


def workload_ns_flops(wl: Workload) -> float:
    return sum(m.batch * ns_dense_flops(m.rows, m.cols, wl.ns_steps) for m in wl.matrices)
