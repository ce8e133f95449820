"""Grouped launches (muon_set_grouping, calls on one stream): chunks that
leave compute units idle and share the 256 x 256 kernels, the step count and
the parameter dtype run each product of each step as one launch over all
their tiles.  Every case is compared bit for bit with the same call run chunk
by chunk, and the grouped results with the oracle."""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import MOMENTUM_TOL, TOL, decode, o_gate, rel, require_gpu, to_bits, to_dev, to_host, w_gate

pytestmark = pytest.mark.gpu

# three shape buckets, each a chunk whose Gram launch fills few of the CUs:
# 3 x 512^2 (9 upper tiles), 3 x 512 x 1536 in both orientations (9), and
# 2 x 768 x 1024 (12)
SHAPES = [(512, 512)] * 3 + [(1536, 512), (512, 1536), (1536, 512)] + [(768, 1024)] * 2


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    m.set_streams(1)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([synth.ROOT_SEED, 7400, *key])))


def inputs(shapes, pdts=None, key=0):
    pdts = pdts or ["bf16"] * len(shapes)
    W = [synth.draw(s, 0.02, p, rng(key, i, 0)) for i, (s, p) in enumerate(zip(shapes, pdts))]
    G = [synth.draw(s, 1e-3, "bf16", rng(key, i, 1)) for i, s in enumerate(shapes)]
    B = [synth.draw(s, 1e-3, "f32", rng(key, i, 2)) for i, s in enumerate(shapes)]
    return W, G, B, pdts


def run_step(muon, W, G, B, pdts, grouping, **kw):
    import torch
    muon.set_grouping(grouping)
    dW = [to_dev(w, p) for w, p in zip(W, pdts)]
    dG = [to_dev(g, "bf16") for g in G]
    dB = [to_dev(b, "f32") for b in B]
    muon.step(dW, dG, dB, lr=0.02, beta=0.95, weight_decay=0.01, **kw)
    torch.cuda.synchronize()
    return dW, dB


def test_grouped_step_equals_chunk_by_chunk_and_oracle(muon):
    W, G, B, pdts = inputs(SHAPES)
    gw, gb = run_step(muon, W, G, B, pdts, True)
    sw, sb = run_step(muon, W, G, B, pdts, False)
    for i in range(len(SHAPES)):
        assert np.array_equal(to_bits(gw[i]), to_bits(sw[i])), i
        assert np.array_equal(to_bits(gb[i]), to_bits(sb[i])), i
    hp = ref.MuonHParams(lr=0.02, beta=0.95, weight_decay=0.01)
    for i in (0, 3, 4, 6):
        W0 = decode(W[i], "bf16")
        r = ref.muon_step_matrix(W0, decode(G[i], "bf16"), np.asarray(B[i], np.float64), hp)
        err, rho = w_gate(to_host(gw[i]), r.W_new, W0, "bf16")
        print(f"grouped step {SHAPES[i]}: W err {err:.3e} (rho {rho:.1e})", flush=True)
        assert err <= TOL["bf16"] + rho, (i, err, rho)
        assert rel(to_host(gb[i]), r.buf_new) <= MOMENTUM_TOL


def test_grouped_orthogonalize_equals_chunk_by_chunk_and_oracle(muon):
    import torch
    G = [synth.draw(s, 1.0, "bf16", rng(1, i)) for i, s in enumerate(SHAPES)]
    ins = [to_dev(g, "bf16") for g in G]
    outs = {}
    for grouping in (True, False):
        muon.set_grouping(grouping)
        o = [torch.full_like(t, float("nan")) for t in ins]
        muon.orthogonalize(ins, o)
        torch.cuda.synchronize()
        outs[grouping] = o
    for i in range(len(SHAPES)):
        assert np.array_equal(to_bits(outs[True][i]), to_bits(outs[False][i])), i
    for i in (0, 4, 7):
        x = decode(G[i], "bf16")
        err, gate = o_gate(to_host(outs[True][i]), ref.orthogonalize(x, 5), "bf16", "bf16", G=x)
        assert err <= gate, (i, err, gate)


def test_one_launch_per_product_and_step(muon):
    W, G, B, pdts = inputs(SHAPES, key=2)
    counts = {}
    for grouping in (True, False):
        muon.profile(True)
        muon.profile_read(reset=True)
        run_step(muon, W, G, B, pdts, grouping)
        st = muon.profile_read(reset=True)
        muon.profile(False)
        counts[grouping] = {k: v["launches"] for k, v in st.items()}
        flops = {k: v["flops"] for k, v in st.items()}
        counts[grouping]["_flops"] = flops
    print(counts, flush=True)
    g, s = counts[True], counts[False]
    # three chunks, five steps: 5 grouped launches per product against 15
    assert g["gram_syrk"] == 5 and g["poly_syrk"] == 5 and g["update_gemm"] == 4 and g["update_apply_gemm"] == 1
    assert s["gram_syrk"] == 15 and s["poly_syrk"] == 15 and s["update_gemm"] == 12 and s["update_apply_gemm"] == 3
    # the prologue stays per chunk; the work counted is the same
    assert g["momentum_norm"] == s["momentum_norm"] == 3
    for k in ("gram_syrk", "poly_syrk", "update_gemm", "update_apply_gemm"):
        assert g["_flops"][k] == pytest.approx(s["_flops"][k], rel=1e-12)


def test_groups_split_by_parameter_dtype_and_step_count(muon):
    # fp32 parameters form their own group; entries with a 3-step table form
    # theirs; results equal the chunk-by-chunk run
    shapes = SHAPES + [(512, 512)] * 2
    pdts = ["bf16"] * 3 + ["f32"] * 3 + ["bf16"] * 2 + ["bf16"] * 2
    W, G, B, _ = inputs(shapes, pdts, key=3)
    coeffs = [None] * 8 + [[[3.4445, -4.7750, 2.0315]] * 3] * 2
    gw, gb = run_step(muon, W, G, B, pdts, True, entry_coeffs=coeffs)
    sw, sb = run_step(muon, W, G, B, pdts, False, entry_coeffs=coeffs)
    for i in range(len(shapes)):
        assert np.array_equal(to_bits(gw[i]), to_bits(sw[i])), i
        assert np.array_equal(to_bits(gb[i]), to_bits(sb[i])), i


def test_workspace_limit_below_a_group_runs_chunk_by_chunk(muon):
    # a limit (20 MiB) that holds the largest chunk (3 x 512 x 1536: two X of
    # 4.5 MiB, A and B of 1.5 MiB) but not the three chunks' regions together
    # (28.5 MiB)
    import torch
    from paper_2609_21594_amd.binding import Muon
    W, G, B, pdts = inputs(SHAPES, key=4)
    want_w, want_b = run_step(muon, W, G, B, pdts, False)
    m = Muon(0)
    try:
        m.set_streams(1)
        m.set_grouping(True)
        m.set_workspace_limit(20 << 20)
        dW = [to_dev(w, "bf16") for w in W]
        dG = [to_dev(g, "bf16") for g in G]
        dB = [to_dev(b, "f32") for b in B]
        m.step(dW, dG, dB, lr=0.02, beta=0.95, weight_decay=0.01)
        torch.cuda.synchronize()
        assert m.workspace_bytes <= 20 << 20
        for i in range(len(SHAPES)):
            assert np.array_equal(to_bits(dW[i]), to_bits(want_w[i])), i
            assert np.array_equal(to_bits(dB[i]), to_bits(want_b[i])), i
    finally:
        m.close()
