"""The bf16 storage error on the CPU (tests/bf16_pipeline.py), which the
gates of the bf16 path rest on.

* Shapes with many singular values (every configuration matrix has a short
  side of 128 or more) stay well inside the flat 2e-2 gate from bf16 storage
  alone, so that gate has room for the kernels' own rounding order.
* Vectors and other shapes with a short side below 16 exceed 2e-2 from bf16
  storage alone on some inputs: the flat gate cannot hold there, which is why
  such shapes take the worst emulated error over 64 inputs as their gate.
"""
import numpy as np
import pytest

from oracle import muon_ref as ref
from tests import bf16_pipeline as bp


def test_emulation_follows_the_scalar_map_on_a_1x1_input():
    # a 1 x 1 input is one singular value: the emulation is the scalar map of
    # Eq. (1) with each stage rounded to 8 significant bits, so it stays within
    # four roundings per step of the exact value
    G = np.array([[3.0]])
    got = bp.emulate_orthogonalize(G)[0, 0]
    want = ref.orthogonalize(G, 5)[0, 0]
    assert abs(got - want) / want < 4 * 5 * 2.0 ** -9


@pytest.mark.parametrize("shape", [(128, 256), (256, 128), (128, 512)])
def test_many_singular_values_stay_inside_the_flat_gate(shape):
    errs = []
    for seed in range(4):
        rng = np.random.default_rng([7, seed, *shape])
        G = ref.round_to_bf16(rng.standard_normal(shape))
        errs.append(bp.storage_error(G))
    assert max(errs) < 0.75 * bp.FLAT_BF16_TOL, errs


def test_vectors_exceed_the_flat_gate_from_storage_alone():
    worst = 0.0
    for seed in range(bp.FEW_SV_SEEDS):
        rng = np.random.default_rng([0xB16, seed, 1, 7])
        G = ref.round_to_bf16(rng.standard_normal((1, 7)))
        worst = max(worst, bp.storage_error(G))
    assert worst > bp.FLAT_BF16_TOL
    assert bp.few_sv_tol((1, 7)) == bp.FEW_SV_MARGIN * worst


def test_few_sv_gate_is_never_below_the_flat_gate():
    assert bp.few_sv_tol((1, 1)) == bp.FLAT_BF16_TOL
