"""An emulation of the bf16 Newton-Schulz pipeline on the CPU (test helper).

It computes the iteration of Eq. (1) the way the bf16 path stores it: X, A
and B rounded to bfloat16 (nearest, ties to even) after every product, the
products of bf16 operands accumulated in binary32.  It is not the oracle:
the oracle is exact fp64, and the gates measure the GPU path against it.
This emulation measures how far the bf16 storage itself takes a result from
the exact one on a given shape, which is what a tolerance on the bf16 path
has to allow.  It shares nothing with the HIP library.

Why it is needed: with many singular values the roundings of X, A and B
average out and the error of the bf16 path stays near 1.1-1.4e-2; a matrix
whose short side is tiny has one or a few singular values, which absorb
every rounding coherently, so the storage alone can exceed 2e-2 there.
"""
from __future__ import annotations

import numpy as np

from oracle import muon_ref as ref

FLAT_BF16_TOL = 2e-2
FEW_SV_SHORT_SIDE = 16     # short side below which the few-value gate applies
FEW_SV_SEEDS = 64          # inputs per shape the few-value gate is taken over
# The kernels round in another order than the emulation (the sums of each
# product, and X~ = u rounded before 1/||u|| is applied on the first step),
# so their result is one more draw of the same storage error; the gate
# allows a quarter more than the worst emulated draw.
FEW_SV_MARGIN = 1.25


def _f32(x):
    return np.asarray(x, dtype=np.float32)


def emulate_orthogonalize(G, ns_steps: int = 5, ns_coeffs=None, eps: float = 1e-7):
    """Transpose-first NS with bf16 storage of X, A and B and binary32
    accumulation of every product; returns fp64 values of bf16 numbers."""
    rb = ref.round_to_bf16
    G = np.asarray(G, dtype=np.float64)
    t = G.shape[0] > G.shape[1]
    Y = G.T if t else G
    X = rb(Y / (np.sqrt(np.sum(Y * Y)) + eps))
    for a, b, c in ref.coefficient_table(ns_steps, ns_coeffs):
        A = rb(_f32(X) @ _f32(X).T)
        B = rb(c * (_f32(A) @ _f32(A)).astype(np.float64) + b * A)
        X = rb(a * X + (_f32(B) @ _f32(X)).astype(np.float64))
    return X.T if t else X


def storage_error(G, ns_steps: int = 5, ns_coeffs=None) -> float:
    """Relative Frobenius distance of the emulated bf16 result from the
    exact one (the oracle) for one input."""
    want = ref.orthogonalize(G, ns_steps, ns_coeffs)
    got = emulate_orthogonalize(G, ns_steps, ns_coeffs)
    return float(np.linalg.norm(got - want) / np.linalg.norm(want))


def worst_storage_error(shape, ns_steps: int = 5, ns_coeffs=None) -> float:
    """The worst storage error the emulation reaches on FEW_SV_SEEDS bf16
    standard normal inputs of this shape."""
    worst = 0.0
    for seed in range(FEW_SV_SEEDS):
        rng = np.random.default_rng([0xB16, seed, *shape])
        G = ref.round_to_bf16(rng.standard_normal(shape))
        worst = max(worst, storage_error(G, ns_steps, ns_coeffs))
    return worst


def few_sv_tol(shape, ns_steps: int = 5, ns_coeffs=None, G=None) -> float:
    """Gate of the bf16 path for a matrix with a short side below 16:
    FEW_SV_MARGIN times the worst emulated storage error over FEW_SV_SEEDS
    inputs of this shape and, when given, the tested input G itself; never
    below the flat 2e-2."""
    worst = worst_storage_error(tuple(shape), ns_steps, ns_coeffs)
    if G is not None:
        worst = max(worst, storage_error(G, ns_steps, ns_coeffs))
    return max(FLAT_BF16_TOL, FEW_SV_MARGIN * worst)
