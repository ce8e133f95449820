"""Planted mistakes in the oracle must each break at least one pin (CPU only).

Each case swaps one oracle function for a plausible wrong version (a dropped
term, a wrong sign, a transposed operand, eps in the wrong place, the other
momentum convention, decay applied in the wrong order, rounding twice), or
one digit of the default coefficient table for another, and runs the pins;
the case passes when some pin fails.
"""
import numpy as np
import pytest

from oracle import muon_ref as ref
import tests.test_oracle_pins as pins


def _ns_drop_c(X0, coeffs):
    X = X0
    for a, b, c in coeffs:
        A = X @ X.T
        X = a * X + (b * A) @ X
    return X


def _ns_wrong_sign(X0, coeffs):
    X = X0
    for a, b, c in coeffs:
        A = X @ X.T
        X = a * X - (b * A + c * A @ A) @ X
    return X


def _ns_gram_transposed(X0, coeffs):
    X = X0
    for a, b, c in coeffs:
        A = X.T @ X
        B = b * A + c * A @ A
        X = a * X + B @ X
    return X


def _ns_right_multiply(X0, coeffs):
    # B applied on the wrong side: only shape-compatible for square X
    X = X0
    for a, b, c in coeffs:
        A = X @ X.T
        B = b * A + c * A @ A
        X = a * X + X @ B
    return X


def _ns_c_uses_A(X0, coeffs):
    X = X0
    for a, b, c in coeffs:
        A = X @ X.T
        X = a * X + (b * A + c * A) @ X
    return X


def _normalize_eps_in_sqrt(G, eps=ref.DEFAULT_EPS):
    G = np.asarray(G, dtype=np.float64)
    return G / np.sqrt(np.sum(G * G) + eps)


def _normalize_no_eps(G, eps=ref.DEFAULT_EPS):
    G = np.asarray(G, dtype=np.float64)
    return G / np.sqrt(np.sum(G * G))


def _momentum_sgd(g, buf, beta, nesterov=True):
    g = np.asarray(g, float); buf = np.asarray(buf, float)
    bn = beta * buf + g
    return bn, (g + beta * bn if nesterov else bn)


def _momentum_bad_nesterov(g, buf, beta, nesterov=True):
    g = np.asarray(g, float); buf = np.asarray(buf, float)
    bn = beta * buf + (1 - beta) * g
    return bn, ((1 - beta) * g + beta * buf if nesterov else bn)


def _scale_min_side(rows, cols, scale_mode=0):
    return 0.2 * float(np.sqrt(min(rows, cols))) if scale_mode == 0 else 1.0


def _apply_decay_after(W, O, lr, weight_decay, scale, post_scale=1.0):
    return post_scale * (1.0 - lr * weight_decay) * (np.asarray(W, float) - lr * scale * np.asarray(O, float))


def _apply_post_scale_update_only(W, O, lr, weight_decay, scale, post_scale=1.0):
    return (1.0 - lr * weight_decay) * np.asarray(W, float) - post_scale * lr * scale * np.asarray(O, float)


def _apply_post_scale_decay_only(W, O, lr, weight_decay, scale, post_scale=1.0):
    return post_scale * (1.0 - lr * weight_decay) * np.asarray(W, float) - lr * scale * np.asarray(O, float)


def _round_bf16_via_f32(x):
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = x32.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def _run_all_pins():
    """Run every pin test function; return the names that failed."""
    failed = []
    cases = [
        ("momentum_hand", pins.test_momentum_hand_example, {}),
        ("momentum_closed", pins.test_momentum_constant_gradient_closed_form, {}),
        ("whole_step_hand", pins.test_whole_step_hand_example, {}),
        ("bf16_hand", pins.test_bf16_round_hand_cases, {}),
        ("eps_small_norm", pins.test_ns_spectral_small_norm_exposes_eps_placement, {}),
        ("vector", pins.test_ns_vector_and_scalar, {"shape": (1, 50)}),
        ("diag", pins.test_ns_diagonal_reduces_to_scalars, {}),
        ("apply_scale", pins.test_apply_scale_uses_long_side, {"shape": (6, 9)}),
        ("zero_update", pins.test_apply_zero_update_is_pure_decay, {}),
        ("post_scale_hand", pins.test_post_scale_hand_example, {}),
        ("post_scale_decay", pins.test_post_scale_applies_to_the_decayed_weight, {}),
        ("legacy_orthogonal", pins.test_legacy_values_on_orthogonal_input, {"n": 128}),
        ("legacy_vector", pins.test_legacy_value_on_vectors, {"shape": (1, 37)}),
        ("legacy_rank_one", pins.test_legacy_value_on_rank_one, {}),
        ("legacy_slope", pins.test_legacy_slope_at_zero, {}),
    ]
    for shape in [(8, 5), (5, 8), (6, 6)]:
        cases.append((f"spectral{shape}", pins.test_ns_spectral_closed_form,
                      {"shape": shape, "table": "legacy"}))
    for name, fn, kw in cases:
        try:
            fn(**kw)
        except Exception:  # assertion or shape error: the pin caught it
            failed.append(name)
    return failed


MUTANTS = {
    "drop_c_term": ("newton_schulz", _ns_drop_c),
    "wrong_sign": ("newton_schulz", _ns_wrong_sign),
    "gram_transposed": ("newton_schulz", _ns_gram_transposed),
    "right_multiply": ("newton_schulz", _ns_right_multiply),
    "c_uses_A": ("newton_schulz", _ns_c_uses_A),
    "eps_in_sqrt": ("frobenius_normalize", _normalize_eps_in_sqrt),
    "no_eps": ("frobenius_normalize", _normalize_no_eps),
    "sgd_momentum": ("momentum_update", _momentum_sgd),
    "nesterov_old_buf": ("momentum_update", _momentum_bad_nesterov),
    "scale_min_side": ("rms_scale", _scale_min_side),
    "decay_after_update": ("apply_update", _apply_decay_after),
    "post_scale_update_only": ("apply_update", _apply_post_scale_update_only),
    "post_scale_decay_only": ("apply_update", _apply_post_scale_decay_only),
    "bf16_double_round": ("round_to_bf16", _round_bf16_via_f32),
    # one digit off in each coefficient of the default table
    "legacy_a_typo": ("LEGACY_QUINTIC", (3.4454, -4.7750, 2.0315)),
    "legacy_b_typo": ("LEGACY_QUINTIC", (3.4445, -4.7705, 2.0315)),
    "legacy_c_typo": ("LEGACY_QUINTIC", (3.4445, -4.7750, 2.0351)),
    "legacy_c_last_digit": ("LEGACY_QUINTIC", (3.4445, -4.7750, 2.0316)),
}


def test_unmutated_oracle_passes_all_pins():
    assert _run_all_pins() == []


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    attr, fn = MUTANTS[mutant]
    monkeypatch.setattr(ref, attr, fn)
    assert _run_all_pins(), f"no pin caught the planted mistake {mutant}"
