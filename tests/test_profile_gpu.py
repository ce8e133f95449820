"""Launch accounting and workspace reservation through the C ABI.

With profiling on, every launch is bracketed by events on its stream and
counted under its kernel family; the flop figures are the ones the bench's
roofline divides by the measured time, so they are checked here against the
dense count of Eq. 1 (2 s^2 l per Gram and update product, 2 s^3 per
polynomial product) and against the MFMA work of the 256 x 256 kernel
(upper tiles of the symmetric products).  Profiling must not change results.
"""
import numpy as np
import pytest

from paper_2609_21594_amd import synth
from tests.gpu_util import require_gpu, to_bits, to_dev

pytestmark = pytest.mark.gpu


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([9191, *key])))


def inputs(shapes):
    W = [to_dev(synth.draw(s, 0.02, "bf16", rng(i, 0)), "bf16") for i, s in enumerate(shapes)]
    G = [to_dev(synth.draw(s, 1e-3, "bf16", rng(i, 1)), "bf16") for i, s in enumerate(shapes)]
    M = [to_dev(synth.draw(s, 1e-3, "f32", rng(i, 2)), "f32") for i, s in enumerate(shapes)]
    return W, G, M


def test_profile_counts_and_flops_and_no_effect_on_results():
    require_gpu()
    import torch
    from paper_2609_21594_amd.binding import Muon
    K = 5
    s, l, n = 512, 1024, 3  # one chunk of three 512 x 1024 matrices on the 256 x 256 kernel
    shapes = [(s, l)] * n
    plain = Muon(0)
    prof = Muon(0)
    try:
        W1, G1, M1 = inputs(shapes)
        W2, G2, M2 = inputs(shapes)
        plain.step(W1, G1, M1, ns_steps=K)
        prof.profile(True)
        prof.profile_read(reset=True)
        prof.step(W2, G2, M2, ns_steps=K)
        st = prof.profile_read(reset=True)
        torch.cuda.synchronize()
        for a, b in zip(W1 + M1, W2 + M2):
            np.testing.assert_array_equal(to_bits(a), to_bits(b))
    finally:
        plain.close()
        prof.close()
    launches = {k: v["launches"] for k, v in st.items()}
    assert launches["momentum_norm"] == 1 and launches["norm_finalize"] == 1 and launches["rescale"] == 1
    assert launches["gram_syrk"] == K and launches["poly_syrk"] == K
    assert launches["update_gemm"] == K - 1 and launches["update_apply_gemm"] == 1
    assert launches["apply_x0"] == 0 and launches["adamw"] == 0
    for k, v in st.items():
        assert v["total_ms"] >= 0 and (v["launches"] > 0 or v["total_ms"] == 0), k
        if v["flops"]:
            assert v["total_ms"] > 0, k
    t = s // 256
    upper = (t * (t + 1) // 2) / (t * t)
    assert st["gram_syrk"]["flops"] == pytest.approx(K * n * 2 * s * s * l, rel=1e-12)
    assert st["gram_syrk"]["exec_flops"] == pytest.approx(K * n * 2 * s * s * l * upper, rel=1e-12)
    assert st["poly_syrk"]["flops"] == pytest.approx(K * n * 2 * s ** 3, rel=1e-12)
    assert st["poly_syrk"]["exec_flops"] == pytest.approx(K * n * 2 * s ** 3 * upper, rel=1e-12)
    assert st["update_gemm"]["flops"] == pytest.approx((K - 1) * n * 2 * s * s * l, rel=1e-12)
    assert st["update_apply_gemm"]["flops"] == pytest.approx(n * 2 * s * s * l, rel=1e-12)
    assert st["update_gemm"]["exec_flops"] == st["update_gemm"]["flops"]


def test_reserve_presizes_the_workspace():
    require_gpu()
    import torch
    from paper_2609_21594_amd.binding import Muon
    shapes = [(512, 1024)] * 2 + [(256, 256)]
    m = Muon(0)
    try:
        m.reserve(64 << 20)
        assert m.workspace_bytes >= 64 << 20
        before = m.workspace_bytes
        W, G, M = inputs(shapes)
        m.step(W, G, M)
        torch.cuda.synchronize()
        assert m.workspace_bytes == before  # the plan fitted: nothing was reallocated
    finally:
        m.close()
    from paper_2609_21594_amd.binding import MuonError
    capped = Muon(0)
    try:
        capped.set_workspace_limit(1 << 20)
        with pytest.raises(MuonError) as e:
            capped.reserve(2 << 20)
        assert e.value.status == 3 and capped.workspace_bytes == 0
    finally:
        capped.close()
