"""Oracle for the per-device Muon step: a plain, slow, fp64 CPU definition.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: it exists so that tests, the smoke check and the CPU
baseline leg of the benchmark can compare the HIP kernels against the paper's
definition.  It shares no code with the HIP library, and it never consumes a
value the HIP library produced.

What is computed (paper: HyperParallel-FSDP, arXiv 2609.21594):

* Sec. 2.3, Eq. (1): Muon accumulates momentum G, normalises it,
  X_0 = G / (||G||_F + eps), and runs k Newton-Schulz steps
  X_{k+1} = a_k X_k + b_k (X_k X_k^T) X_k + c_k (X_k X_k^T)^2 X_k,
  which approximates msign(G) = U V^T.  The result is multiplied by the
  RMS-matching factor 0.2 * sqrt(max(m, n)) so AdamW learning rates carry over.
* Sec. 6.6: when a matrix has more rows than columns the iteration runs on its
  transpose, so the Gram product sits on the short side.
* Sec. 6.3: a fused expert weight [E, M, N] is E independent [M, N] matrices;
  it is never flattened.
* Sec. 6.4 and Fig. "muon-grouping": the update is applied together with
  decoupled weight decay; one-dimensional and scalar parameters leave Muon
  for AdamW through a chained optimizer (adamw_step at the end).

Readings where the paper is silent (each is listed in the design notes):

* momentum is the EMA form buf' = beta*buf + (1-beta)*g, and the Nesterov
  blend is u = (1-beta)*g + beta*buf' (Sec. 7.4 runs Nesterov with beta 0.95
  but prints no recurrence);
* eps = 1e-7 is added to the Frobenius norm, outside the square root, as in
  Eq. (1)'s placement;
* weight decay is multiplicative on the old W and simultaneous with the
  update: W' = (1 - lr*wd) W - lr * 0.2*sqrt(max(m,n)) * O;
* a square matrix is not transposed ("more rows than columns" is strict);
* the default coefficient table is the constant quintic (3.4445, -4.7750,
  2.0315) of the original Muon method the paper cites as its legacy set; the
  paper prints neither that set nor its asymmetric five-step default, so any
  per-step table can be passed in;
* scale_mode 2, sqrt(max(1, m/n)), is the original Muon method's scale,
  which the paper keeps as a configurable legacy stage without printing it;
* AdamW (which the paper names but does not define) has exponential moments,
  bias correction by 1 - beta^t and decoupled decay on the old value.

Every floating-point step runs in fp64.  Inputs are decoded exactly; results
are rounded once, from fp64, to the storage type (round to nearest, ties to
even).  The module uses only NumPy; matrix products are plain dense ``@``
products with no use of the symmetry of X X^T.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

# Constant-coefficient quintic of the original Muon method (the "legacy"
# coefficient set of Sec. 2.3 / Sec. 6.6, values from the cited method).
LEGACY_QUINTIC: Tuple[float, float, float] = (3.4445, -4.7750, 2.0315)
DEFAULT_EPS = 1e-7
# RMS-matching constant of Sec. 2.3.
RMS_MATCH = 0.2


# --------------------------------------------------------------------------
# Storage codecs (exact decode, single rounding on store)
# --------------------------------------------------------------------------
def decode_bf16(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exact fp64 values.

    A bfloat16 number is the upper half of an IEEE binary32 number, so
    shifting the 16 bits into the top of a 32-bit word gives the binary32
    pattern of the same value, which widens to fp64 exactly.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def round_to_bf16(x) -> np.ndarray:
    """Round fp64 values to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits and binary32's exponent range, so for
    x = m * 2**e (0.5 <= |m| < 1) the spacing of representable values is
    2**(e-8), and never finer than the subnormal spacing 2**-133.  Scaling by
    a power of two is exact, and ``np.rint`` rounds half to even, so the
    rounding happens once, directly from fp64 (no detour through binary32,
    which could round twice).  Magnitudes that round to 2**128 or beyond
    overflow to infinity; NaN and infinities pass through.
    """
    x = np.asarray(x, dtype=np.float64)
    out = x.copy()
    fin = np.isfinite(x)
    xf = x[fin]
    _, e = np.frexp(xf)
    q = np.maximum(e - 8, -133)
    y = np.ldexp(np.rint(np.ldexp(xf, -q)), q)
    y = np.where(np.abs(y) >= 2.0 ** 128, np.copysign(np.inf, xf), y)
    out[fin] = y
    return out


def encode_bf16(x) -> np.ndarray:
    """fp64 values -> bfloat16 bit patterns, rounding as ``round_to_bf16``."""
    r = round_to_bf16(x).astype(np.float32)  # exact: r is a bfloat16 value
    return (r.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def round_to_f32(x) -> np.ndarray:
    """Round fp64 values to binary32 (NumPy's cast rounds to nearest even)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(x, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_to_bf16(x)
    if dtype == "f32":
        return round_to_f32(x)
    raise ValueError(f"unknown storage dtype {dtype!r}")


# --------------------------------------------------------------------------
# The Muon step, one matrix at a time
# --------------------------------------------------------------------------
@dataclass
class MuonHParams:
    lr: float = 0.02
    beta: float = 0.95
    weight_decay: float = 0.0
    eps: float = DEFAULT_EPS
    ns_steps: int = 5
    nesterov: bool = True
    # Per-step (a_k, b_k, c_k); None selects LEGACY_QUINTIC at every step.
    ns_coeffs: Optional[Sequence[Tuple[float, float, float]]] = None
    # 0: multiply by 0.2*sqrt(max(m, n)) (Sec. 2.3); 1: no rescale;
    # 2: sqrt(max(1, m/n)) (the original Muon rule; see rms_scale).
    scale_mode: int = 0
    # Post-processing after the update (Sec. 6.2 lists it among the
    # pluggable stages, QK-clip being the example): the updated matrix is
    # multiplied by this factor, which the caller derives (for QK-clip, per
    # attention head from its logits).  1: none.
    post_scale: float = 1.0

    def coefficient_table(self) -> List[Tuple[float, float, float]]:
        return coefficient_table(self.ns_steps, self.ns_coeffs)


def coefficient_table(ns_steps: int,
                      ns_coeffs: Optional[Sequence[Sequence[float]]] = None
                      ) -> List[Tuple[float, float, float]]:
    """The K rows (a_k, b_k, c_k) of Eq. (1); None means the legacy quintic."""
    if ns_steps < 0:
        raise ValueError("ns_steps must be >= 0")
    if ns_coeffs is None:
        return [LEGACY_QUINTIC] * ns_steps
    rows = [tuple(float(v) for v in r) for r in ns_coeffs]
    if len(rows) != ns_steps or any(len(r) != 3 for r in rows):
        raise ValueError("ns_coeffs must hold ns_steps rows of (a, b, c)")
    return rows


def momentum_update(g: np.ndarray, buf: np.ndarray, beta: float,
                    nesterov: bool = True) -> Tuple[np.ndarray, np.ndarray]:
    """Momentum accumulation of Sec. 2.3 (EMA form) with the Nesterov blend.

    Returns (buf', u): buf' = beta*buf + (1-beta)*g is the new state, u is the
    direction handed to the orthogonalisation: (1-beta)*g + beta*buf' with
    Nesterov, buf' without.
    """
    g = np.asarray(g, dtype=np.float64)
    buf = np.asarray(buf, dtype=np.float64)
    buf_new = beta * buf + (1.0 - beta) * g
    u = (1.0 - beta) * g + beta * buf_new if nesterov else buf_new
    return buf_new, u


def frobenius_normalize(G: np.ndarray, eps: float = DEFAULT_EPS) -> np.ndarray:
    """X_0 = G / (||G||_F + eps), Eq. (1)."""
    G = np.asarray(G, dtype=np.float64)
    norm = np.sqrt(np.sum(G * G))
    return G / (norm + eps)


def newton_schulz(X0: np.ndarray, coeffs: Iterable[Sequence[float]]) -> np.ndarray:
    """The quintic iteration of Eq. (1), one step per coefficient row.

    A = X X^T, then X <- a X + (b A + c A A) X, with plain dense products.
    """
    X = np.asarray(X0, dtype=np.float64)
    for a, b, c in coeffs:
        A = X @ X.T
        B = b * A + c * (A @ A)
        X = a * X + B @ X
    return X


def orthogonalize(G: np.ndarray, ns_steps: int = 5,
                  ns_coeffs: Optional[Sequence[Sequence[float]]] = None,
                  eps: float = DEFAULT_EPS) -> np.ndarray:
    """NS orthogonalisation of one matrix, transpose-first (Sec. 6.6).

    If G has more rows than columns the iteration runs on G^T (so the Gram
    matrix is min(m,n) square) and the result is transposed back, so the
    output always has G's shape.
    """
    G = np.asarray(G, dtype=np.float64)
    if G.ndim != 2:
        raise ValueError("orthogonalize takes one matrix")
    transposed = G.shape[0] > G.shape[1]
    Y = G.T if transposed else G
    X = newton_schulz(frobenius_normalize(Y, eps), coefficient_table(ns_steps, ns_coeffs))
    return X.T if transposed else X


def rms_scale(rows: int, cols: int, scale_mode: int = 0) -> float:
    """Update scale of the m x n matrix.

    0: the RMS-matching factor 0.2*sqrt(max(m, n)) of Sec. 2.3;
    1: no rescale;
    2: sqrt(max(1, m/n)), the factor of the original Muon method, which
       Sec. 2.3 and Sec. 6.2 keep as a configurable legacy stage.
    """
    if scale_mode == 0:
        return RMS_MATCH * float(np.sqrt(max(rows, cols)))
    if scale_mode == 1:
        return 1.0
    if scale_mode == 2:
        return float(np.sqrt(max(1.0, rows / cols)))
    raise ValueError("scale_mode must be 0, 1 or 2")


def apply_update(W: np.ndarray, O: np.ndarray, lr: float, weight_decay: float,
                 scale: float, post_scale: float = 1.0) -> np.ndarray:
    """Decoupled weight decay and update, W' = (1 - lr*wd) W - lr*scale*O,
    then the post-processing stage (Sec. 6.2): W' multiplied by post_scale."""
    W = np.asarray(W, dtype=np.float64)
    W_new = (1.0 - lr * weight_decay) * W - lr * scale * np.asarray(O, dtype=np.float64)
    return W_new if post_scale == 1.0 else post_scale * W_new


@dataclass
class StepResult:
    W_new: np.ndarray      # fp64, before storage rounding
    buf_new: np.ndarray    # fp64, before storage rounding
    O: np.ndarray          # orthogonalised update, the matrix's own shape


def muon_step_matrix(W, g, buf, hp: MuonHParams) -> StepResult:
    """One Muon step on one 2-D matrix (Sec. 2.3 with the readings above)."""
    W = np.asarray(W, dtype=np.float64)
    if W.ndim != 2:
        raise ValueError("muon_step_matrix takes one matrix")
    buf_new, u = momentum_update(g, buf, hp.beta, hp.nesterov)
    O = orthogonalize(u, hp.ns_steps, hp.ns_coeffs, hp.eps)
    scale = rms_scale(W.shape[0], W.shape[1], hp.scale_mode)
    return StepResult(apply_update(W, O, hp.lr, hp.weight_decay, scale, hp.post_scale), buf_new, O)


def muon_step(params: Sequence[np.ndarray], grads: Sequence[np.ndarray],
              bufs: Sequence[np.ndarray], hp: MuonHParams) -> List[StepResult]:
    """Muon step over a list of parameters; each is [M, N] or [E, M, N].

    A 3-D parameter is E independent matrices (Sec. 6.3): each plane is updated
    on its own and the results are stacked back.
    """
    out: List[StepResult] = []
    for W, g, b in zip(params, grads, bufs):
        W = np.asarray(W, dtype=np.float64)
        if W.ndim == 2:
            out.append(muon_step_matrix(W, g, b, hp))
        elif W.ndim == 3:
            planes = [muon_step_matrix(W[e], np.asarray(g)[e], np.asarray(b)[e], hp)
                      for e in range(W.shape[0])]
            out.append(StepResult(np.stack([p.W_new for p in planes]),
                                  np.stack([p.buf_new for p in planes]),
                                  np.stack([p.O for p in planes])))
        else:
            raise ValueError("Muon takes matrices or stacks of matrices only")
    return out



# ---------------------------------------------------------------------------
# AdamW for the parameters Muon does not take.  Sec. 6.4 (and the decision
# flow of Fig. "muon-grouping") sends one-dimensional and scalar parameters to
# AdamW through a chained optimizer, with decoupled weight decay.  The paper
# prints no formula, so this is AdamW as commonly defined: exponential
# moments, bias correction by 1 - beta^t, decoupled decay on the old value.
# ---------------------------------------------------------------------------
@dataclass
class AdamWHParams:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.0


def adamw_step(p, g, m, v, step: int, hp: AdamWHParams):
    """One AdamW step (t = step >= 1) on arrays of any shape; returns
    (p', m', v') in fp64:
        m' = beta1 m + (1 - beta1) g,   v' = beta2 v + (1 - beta2) g^2,
        p' = (1 - lr wd) p - lr * (m' / (1 - beta1^t)) / (sqrt(v' / (1 - beta2^t)) + eps).
    """
    if step < 1:
        raise ValueError("step must be >= 1")
    p, g, m, v = (np.asarray(a, dtype=np.float64) for a in (p, g, m, v))
    m_new = hp.beta1 * m + (1.0 - hp.beta1) * g
    v_new = hp.beta2 * v + (1.0 - hp.beta2) * g * g
    m_hat = m_new / (1.0 - hp.beta1 ** step)
    v_hat = v_new / (1.0 - hp.beta2 ** step)
    p_new = (1.0 - hp.lr * hp.weight_decay) * p - hp.lr * m_hat / (np.sqrt(v_hat) + hp.eps)
    return p_new, m_new, v_new
