"""Parity of the HIP path with the fp64 oracle, called through the C ABI.

Sizes span several 128-wide tiles and ragged tails; every case compares each
matrix with the oracle at the gates of the method: relative Frobenius error
<= 2e-2 on the bf16 Newton-Schulz path, <= 1e-4 on the fp32 path (plus the
storage-rounding floor of the output dtype), momentum <= 1e-6.
"""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import (MOMENTUM_TOL, TOL, decode, o_gate, rel, require_gpu, to_bits,
                            to_dev, to_host, tol_for, w_gate)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([4242, *key])))


def gen(shape, sigma, dtype, *key):
    return synth.draw(shape, sigma, dtype, rng(*key))


SHAPES = [(1, 1), (1, 7), (7, 1), (17, 33), (33, 17), (64, 64), (128, 256), (256, 128),
          (129, 257), (300, 200), (130, 1000), (384, 384)]


def run_orth(muon, shapes, dtype, prec, ns_steps=5, coeffs=None, eps=1e-7, sigma=1.0, key=0):
    import torch
    G = [gen(s, sigma, dtype, key, i) for i, s in enumerate(shapes)]
    ins = [to_dev(g, dtype) for g in G]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_steps=ns_steps, ns_coeffs=coeffs, eps=eps, ns_precision=prec)
    torch.cuda.synchronize()
    return G, outs


@pytest.mark.parametrize("dtype,prec", [("bf16", "bf16"), ("f32", "f32"), ("bf16", "f32"),
                                        ("f32", "bf16")])
def test_orthogonalize_matches_oracle(muon, dtype, prec):
    G, outs = run_orth(muon, SHAPES, dtype, prec, key=1)
    for s, g, o in zip(SHAPES, G, outs):
        want = ref.orthogonalize(decode(g, dtype), 5)
        err, gate = o_gate(to_host(o), want, dtype, prec, G=decode(g, dtype))
        print(f"orthogonalize {dtype}/{prec} {s}: O err {err:.3e} (gate {gate:.2e})", flush=True)
        assert err <= gate, (s, err, gate)


@pytest.mark.parametrize("nesterov", [True, False])
@pytest.mark.parametrize("pdt,gdt,prec", [("bf16", "bf16", "bf16"), ("f32", "f32", "f32"),
                                          ("f32", "bf16", "bf16"), ("bf16", "f32", "f32")])
def test_muon_step_matches_oracle(muon, pdt, gdt, prec, nesterov):
    import torch
    shapes = [(17, 33), (33, 17), (128, 256), (300, 200), (64, 64), (1, 50)]
    hp = ref.MuonHParams(lr=0.02, beta=0.9, weight_decay=0.1, nesterov=nesterov)
    Ws = [gen(s, 0.02, pdt, 2, i, 0) for i, s in enumerate(shapes)]
    gs = [gen(s, 1e-3, gdt, 2, i, 1) for i, s in enumerate(shapes)]
    bs = [gen(s, 1e-3, "f32", 2, i, 2) for i, s in enumerate(shapes)]
    dW = [to_dev(w, pdt) for w in Ws]
    dg = [to_dev(g, gdt) for g in gs]
    db = [to_dev(b, "f32") for b in bs]
    muon.step(dW, dg, db, lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay,
              nesterov=nesterov, ns_precision=prec)
    torch.cuda.synchronize()
    for s, W, g, b, w_dev, b_dev in zip(shapes, Ws, gs, bs, dW, db):
        W0 = decode(W, pdt)
        r = ref.muon_step_matrix(W0, decode(g, gdt), np.asarray(b, np.float64), hp)
        err, rho = w_gate(to_host(w_dev), r.W_new, W0, pdt)
        gate = tol_for(prec, s, G=ref.momentum_update(decode(g, gdt), b, hp.beta, nesterov)[1])
        print(f"step {pdt}/{gdt}/{prec} {s}: W err {err:.3e} (gate {gate:.2e} + rho {rho:.1e})", flush=True)
        assert err <= gate + rho, (s, err, gate, rho)
        assert rel(to_host(b_dev), r.buf_new) <= MOMENTUM_TOL, s


# Padded extents that are multiples of 256 on both sides take the 256 x 256
# path with upper-triangle storage of A and B (read back transposed below the
# diagonal) and X read through transposing LDS reads.  Several tile rows, so
# every operand mode and mode change occurs; one transposed parameter.
UPPER_SHAPES = [(512, 1024), (1024, 512), (768, 768), (500, 1200)]


@pytest.mark.parametrize("pdt,gdt", [("bf16", "bf16"), ("f32", "f32")])
def test_upper_tile_path_step_matches_oracle(muon, pdt, gdt):
    # bf16 parameters take the staged in-place update for interior blocks and
    # the per-vector one at ragged edges; fp32 parameters always the latter
    import torch
    hp = ref.MuonHParams(lr=0.02, beta=0.95, weight_decay=0.01, nesterov=True)
    Ws = [gen(s, 0.02, pdt, 20, i, 0) for i, s in enumerate(UPPER_SHAPES)]
    gs = [gen(s, 1e-3, gdt, 20, i, 1) for i, s in enumerate(UPPER_SHAPES)]
    bs = [gen(s, 1e-3, "f32", 20, i, 2) for i, s in enumerate(UPPER_SHAPES)]
    dW = [to_dev(w, pdt) for w in Ws]
    dg = [to_dev(g, gdt) for g in gs]
    db = [to_dev(b, "f32") for b in bs]
    muon.step(dW, dg, db, lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, ns_precision="bf16")
    torch.cuda.synchronize()
    for s, W, g, b, w_dev, b_dev in zip(UPPER_SHAPES, Ws, gs, bs, dW, db):
        W0 = decode(W, pdt)
        r = ref.muon_step_matrix(W0, decode(g, gdt), np.asarray(b, np.float64), hp)
        err, rho = w_gate(to_host(w_dev), r.W_new, W0, pdt)
        print(f"upper-tile path {s}: W err {err:.3e} (rho {rho:.1e})", flush=True)
        assert err <= tol_for("bf16", s) + rho, (s, err, rho)
        assert rel(to_host(b_dev), r.buf_new) <= MOMENTUM_TOL, s


def test_upper_tile_path_orthogonalize_matches_oracle(muon):
    G, outs = run_orth(muon, UPPER_SHAPES, "bf16", "bf16", key=21)
    for s, g, o in zip(UPPER_SHAPES, G, outs):
        want = ref.orthogonalize(decode(g, "bf16"), 5)
        err, gate = o_gate(to_host(o), want, "bf16", "bf16")
        assert err <= gate, (s, err, gate)


def test_upper_tile_path_zero_c_steps_match_oracle(muon):
    # Steps with c = 0 (the cubic iteration) read the polynomial's A term in
    # the epilogue; steps with c != 0 add it to the accumulators in the main
    # loop.  Both kinds in one schedule.
    coeffs = [(3.4445, -4.7750, 2.0315)] * 3 + [(1.5, -0.5, 0.0)] * 3
    G, outs = run_orth(muon, UPPER_SHAPES, "bf16", "bf16", ns_steps=len(coeffs), coeffs=coeffs, key=22)
    for s, g, o in zip(UPPER_SHAPES, G, outs):
        want = ref.orthogonalize(decode(g, "bf16"), len(coeffs), coeffs)
        err, gate = o_gate(to_host(o), want, "bf16", "bf16", len(coeffs), coeffs)
        print(f"zero-c schedule {s}: err {err:.3e} (gate {gate:.1e})", flush=True)
        assert err <= gate, (s, err, gate)


def test_rows_past_the_tile_kernel_offsets(muon):
    # Rows of 2^22 + 256 bf16 elements are too long for the 256 x 256
    # kernel's 32-bit row offsets, so this step runs on the 128 x 128 kernel.
    # The gradient's rows have disjoint supports (row i holds v_i on column
    # block i and zeros elsewhere), so the iteration acts on every row alone:
    # the update keeps that pattern exactly, and row i's value follows from
    # the oracle on the 256 x 256 diagonal matrix with the same singular
    # values (v_i sqrt(blk)), divided by sqrt(blk).
    import torch
    s, blk = 256, 16385
    l = s * blk
    assert l * 2 * 256 >= 2 ** 31
    vb = synth.draw((s,), 1.0, "bf16", rng(23))
    v = decode(vb, "bf16")
    lr = 0.02
    G = torch.zeros((s, s, blk), dtype=torch.bfloat16, device="cuda")
    ar = torch.arange(s, device="cuda")
    G[ar, ar, :] = to_dev(vb, "bf16").view(s, 1)
    G = G.view(s, l)
    W = torch.zeros_like(G)
    M = torch.zeros((s, l), dtype=torch.float32, device="cuda")
    muon.step([W], [G], [M], lr=lr, beta=0.95, weight_decay=0.0, ns_precision="bf16")
    torch.cuda.synchronize()
    del G, M
    W3 = W.view(s, s, blk)
    dblk = W3[ar, ar, :]
    assert bool((dblk == dblk[:, :1]).all())
    assert int(torch.count_nonzero(W)) == int(torch.count_nonzero(dblk))
    got = to_host(dblk[:, 0].contiguous())
    # u = (1 - beta)(1 + beta) g is a multiple of g, so X0 is the same
    O_small = ref.orthogonalize(np.diag(v * np.sqrt(blk)), 5)
    want = -lr * 0.2 * np.sqrt(l) * np.diag(O_small) / np.sqrt(blk)
    rho = rel(ref.round_to(want, "bf16"), want)
    err = rel(got, want)
    print(f"long rows ({s} x {l}): err {err:.3e} (rho {rho:.1e})", flush=True)
    assert err <= TOL["bf16"] + rho


def test_fp32_step_recovers_orthogonalised_update(muon):
    # fp32 parameters: O = (decay*W - W') / (lr*scale) is checked at 1e-4.
    import torch
    shape = (256, 128)
    hp = ref.MuonHParams(lr=0.02, beta=0.95, weight_decay=0.0)
    W, g, b = (gen(shape, 1.0, "f32", 3, k) for k in range(3))
    dW, dg, db = to_dev(W, "f32"), to_dev(g, "f32"), to_dev(b, "f32")
    muon.step([dW], [dg], [db], lr=0.02, beta=0.95, ns_precision="f32")
    torch.cuda.synchronize()
    r = ref.muon_step_matrix(W.astype(np.float64), g, b, hp)
    scale = 0.2 * np.sqrt(256)
    O_gpu = (W.astype(np.float64) - to_host(dW)) / (0.02 * scale)
    assert rel(O_gpu, r.O) <= 1e-4


def test_custom_per_step_coefficients(muon):
    # a convergent quintic for 12 steps: the output approaches U V^T
    coeffs = [(15 / 8, -10 / 8, 3 / 8)] * 6 + [(3.4445, -4.7750, 2.0315)] * 2 + [(1.5, -0.5, 0.0)] * 4
    shapes = [(96, 160), (200, 130)]
    G, outs = run_orth(muon, shapes, "f32", "f32", ns_steps=len(coeffs), coeffs=coeffs, key=4)
    for g, o in zip(G, outs):
        want = ref.orthogonalize(g.astype(np.float64), len(coeffs), coeffs)
        assert rel(to_host(o), want) <= 1e-4


@pytest.mark.parametrize("prec", ["bf16", "f32"])
@pytest.mark.parametrize("steps", [1, 2])
def test_one_and_two_steps_match_oracle(muon, steps, prec):
    # K = 1: the first step is also the last, so the last-step kernel applies
    # the norm scale r itself (on the 256 x 256 kernel for the bf16 upper
    # shapes, on the 128 x 128 kernel otherwise); K = 2: one exchange of the
    # ping-pong iterates.  Both the parameter update and the standalone
    # orthogonalisation, whose last kernel writes O.
    import torch
    shapes = UPPER_SHAPES + [(300, 200), (129, 257)]
    # lr large enough that one step's update stands well above the bf16
    # rounding of W (X1 is still far from orthogonal, so O is small)
    hp = ref.MuonHParams(lr=0.5, beta=0.95, weight_decay=0.01, ns_steps=steps)
    Ws = [gen(s, 0.02, "bf16", 24, steps, i, 0) for i, s in enumerate(shapes)]
    gs = [gen(s, 1e-3, "bf16", 24, steps, i, 1) for i, s in enumerate(shapes)]
    bs = [gen(s, 1e-3, "f32", 24, steps, i, 2) for i, s in enumerate(shapes)]
    dW, dg, db = [to_dev(w, "bf16") for w in Ws], [to_dev(g, "bf16") for g in gs], [to_dev(b, "f32") for b in bs]
    muon.step(dW, dg, db, lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, ns_steps=steps,
              ns_precision=prec)
    torch.cuda.synchronize()
    for s, W, g, b, w_dev, b_dev in zip(shapes, Ws, gs, bs, dW, db):
        W0 = decode(W, "bf16")
        r = ref.muon_step_matrix(W0, decode(g, "bf16"), np.asarray(b, np.float64), hp)
        err, rho = w_gate(to_host(w_dev), r.W_new, W0, "bf16")
        print(f"K={steps} {prec} step {s}: W err {err:.3e} (rho {rho:.1e})", flush=True)
        assert err <= tol_for(prec, s) + rho, (s, err, rho)
        assert rel(to_host(b_dev), r.buf_new) <= MOMENTUM_TOL, s
    G, outs = run_orth(muon, shapes, "bf16", prec, ns_steps=steps, key=25 + steps)
    for s, g, o in zip(shapes, G, outs):
        want = ref.orthogonalize(decode(g, "bf16"), steps)
        err, gate = o_gate(to_host(o), want, "bf16", prec, steps)
        print(f"K={steps} {prec} orthogonalize {s}: O err {err:.3e} (gate {gate:.1e})", flush=True)
        assert err <= gate, (s, err, gate)


def test_zero_steps_returns_normalised_input(muon):
    G, outs = run_orth(muon, [(40, 70), (70, 40)], "f32", "f32", ns_steps=0, key=5)
    for g, o in zip(G, outs):
        want = ref.orthogonalize(g.astype(np.float64), 0)
        assert rel(to_host(o), want) <= 1e-6


def test_zero_input_and_pure_decay(muon):
    import torch
    W = gen((100, 60), 1.0, "f32", 6, 0)
    dW = to_dev(W, "f32")
    dg = torch.zeros_like(dW)
    db = torch.zeros_like(dW)
    muon.step([dW], [dg], [db], lr=0.1, weight_decay=0.5, ns_precision="f32")
    torch.cuda.synchronize()
    # the decay factor 1 - lr*wd is an fp32 constant; one rounding of its product
    decay = np.float64(np.float32(1.0 - np.float64(np.float32(0.1)) * np.float64(np.float32(0.5))))
    np.testing.assert_array_equal(to_host(dW), ref.round_to_f32(decay * W.astype(np.float64)))
    # a zero input gives O = 0: the fused small-matrix launch (33 x 9) and the
    # tile kernels (512 x 768)
    for shape in ((33, 9), (512, 768)):
        z = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
        o = torch.full_like(z, 7.0)
        muon.orthogonalize([z], [o])
        torch.cuda.synchronize()
        assert (to_host(o) == 0).all(), shape


@pytest.mark.parametrize("prec,shape", [("f32", (64, 96)),      # fused small-matrix launch
                                        ("bf16", (64, 96)),     # its bf16 form
                                        ("bf16", (512, 1024)),  # 256 x 256 tile kernels
                                        ("bf16", (300, 200))])  # 128 x 128 kernel
def test_nan_propagates_to_its_matrix_only(muon, prec, shape):
    # R13: a NaN in one matrix makes that matrix's output NaN and leaves the
    # other matrices of the call (same chunk, same launches) as the oracle has them
    import torch
    g1 = gen(shape, 1.0, "f32", 7, 0)
    g2 = gen(shape, 1.0, "f32", 7, 1)
    g1[3, 5] = np.nan
    dt = "f32" if prec == "f32" else "bf16"
    if dt == "bf16":
        g1 = decode(synth.f32_to_bf16_bits(g1), "bf16").astype(np.float32)
        g2 = decode(synth.f32_to_bf16_bits(g2), "bf16").astype(np.float32)
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    ins = [torch.from_numpy(g1).to(tdt).cuda(), torch.from_numpy(g2).to(tdt).cuda()]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_precision=prec)
    torch.cuda.synchronize()
    assert np.isnan(to_host(outs[0])).all()
    assert rel(to_host(outs[1]), ref.orthogonalize(g2.astype(np.float64), 5)) <= TOL[prec]


def test_tiny_and_scaled_inputs(muon):
    # 1e-4-scaled and 1e-30-scaled matrices normalise like unit ones (P8)
    import torch
    shapes = [(48, 80)] * 3
    base = gen((48, 80), 1.0, "f32", 8, 0)
    ins = [to_dev(base * np.float32(s), "f32") for s in (1.0, 1e-4, 1e-12)]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_precision="f32", eps=0.0)
    torch.cuda.synchronize()
    want = ref.orthogonalize(base.astype(np.float64), 5, eps=0.0)
    for o in outs:
        assert rel(to_host(o), want) <= 1e-4


@pytest.mark.parametrize("shape", [(48, 80), (160, 600)])
@pytest.mark.parametrize("prec", ["f32", "bf16"])
def test_norms_outside_the_folded_range(muon, prec, shape):
    # The first Newton-Schulz step applies r = 1/(||u|| + eps) to products of
    # u itself while r lies in [2^-40, 2^40]; beyond that X0 = r*u is written
    # out first.  Power-of-two scales keep the inputs exact in both dtypes:
    # ||u|| ~ 2^-44, 2^56, 2^76 (u^2 past the binary32 range: the norm sums
    # run in fp64) and 2^127 (r below the normal binary32 range: applied as
    # two factors).  eps = 0 makes the result scale-invariant.  48 x 80 runs
    # on the fused small-matrix launch, 160 x 600 on the tile kernels.
    import torch
    base = gen(shape, 1.0, "f32", 28, 0)
    base /= np.float32(np.abs(base).max())   # |entries| <= 1, so 2^126 x base stays finite
    if prec == "bf16":
        base = decode(synth.f32_to_bf16_bits(base), "bf16").astype(np.float32)
    want = ref.orthogonalize(base.astype(np.float64), 5, eps=0.0)
    scales = (1.0, 2.0 ** -50, 2.0 ** 50, 2.0 ** 70, 2.0 ** 126)
    dt = torch.float32 if prec == "f32" else torch.bfloat16
    ins = [torch.from_numpy(base * np.float32(sc)).to(dt).cuda() for sc in scales]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_precision=prec, eps=0.0)
    torch.cuda.synchronize()
    for sc, o in zip(scales, outs):
        err = rel(to_host(o), want)
        print(f"norm scale 2^{int(np.log2(sc))} {prec} {shape}: O err {err:.3e}", flush=True)
        assert err <= TOL[prec], sc
    # the same through muon_step: zero momentum, beta = 0, no decay, lr = 1
    # and no rescale, so W' = W - O
    Ws = [torch.zeros(*shape, dtype=dt, device="cuda") for _ in scales]
    Ms = [torch.zeros(*shape, dtype=torch.float32, device="cuda") for _ in scales]
    muon.step(Ws, ins, Ms, lr=1.0, beta=0.0, weight_decay=0.0, eps=0.0, ns_precision=prec, scale_mode=1)
    torch.cuda.synchronize()
    for sc, w in zip(scales, Ws):
        assert rel(-to_host(w), want) <= TOL[prec], sc


def test_orthogonal_input_closed_form(muon):
    import torch
    Q, _ = np.linalg.qr(rng(9).standard_normal((256, 256)))
    f = Q.astype(np.float32)
    out = torch.empty((256, 256), dtype=torch.float32, device="cuda")
    muon.orthogonalize([to_dev(f, "f32")], [out], ns_precision="f32")
    torch.cuda.synchronize()
    s = 1.0 / (16.0 + 1e-7)
    for a, b, c in [ref.LEGACY_QUINTIC] * 5:
        s = a * s + b * s ** 3 + c * s ** 5
    assert rel(to_host(out), s * f.astype(np.float64)) <= 1e-4


# ---------------------------------------------------------------------------
# Invariants of the batching (Sec. 6.6) and determinism
# ---------------------------------------------------------------------------
def _step_bits(muon, shapes, dtypes=("bf16", "bf16"), prec="bf16", key=10, **kw):
    import torch
    pdt, gdt = dtypes
    dW = [to_dev(gen(s, 0.02, pdt, key, i, 0), pdt) for i, s in enumerate(shapes)]
    dg = [to_dev(gen(s, 1e-3, gdt, key, i, 1), gdt) for i, s in enumerate(shapes)]
    db = [to_dev(gen(s, 1e-3, "f32", key, i, 2), "f32") for i, s in enumerate(shapes)]
    muon.step(dW, dg, db, ns_precision=prec, **kw)
    torch.cuda.synchronize()
    return [to_bits(t) for t in dW], [to_bits(t) for t in db]


@pytest.mark.parametrize("shapes", [[(256, 384), (384, 256), (200, 200)], UPPER_SHAPES])
def test_deterministic_repeat(muon, shapes):
    a = _step_bits(muon, shapes)
    b = _step_bits(muon, shapes)
    for x, y in zip(a[0] + a[1], b[0] + b[1]):
        np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("shapes", [[(256, 384), (384, 256), (200, 200), (256, 384)],
                                    [(512, 1024), (768, 768), (1024, 512), (512, 1024)]])
def test_batched_equals_single(muon, shapes):
    # a matrix's bits do not depend on which other matrices share the call
    import torch
    together = _step_bits(muon, shapes)
    for i, s in enumerate(shapes):
        dW = to_dev(gen(s, 0.02, "bf16", 10, i, 0), "bf16")
        dg = to_dev(gen(s, 1e-3, "bf16", 10, i, 1), "bf16")
        db = to_dev(gen(s, 1e-3, "f32", 10, i, 2), "f32")
        muon.step([dW], [dg], [db])
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_bits(dW), together[0][i])
        np.testing.assert_array_equal(to_bits(db), together[1][i])


def test_chunk_cap_does_not_change_results(muon):
    shapes = [(128, 256)] * 5 + [(64, 64)] * 3
    full = _step_bits(muon, shapes, key=11)
    tiny = _step_bits(muon, shapes, key=11, max_chunk_elems=1)
    for x, y in zip(full[0] + full[1], tiny[0] + tiny[1]):
        np.testing.assert_array_equal(x, y)


def test_expert_stack_is_independent_matrices(muon):
    import torch
    E, M, N = 3, 96, 160
    W = gen((E, M, N), 0.02, "bf16", 12, 0)
    g = gen((E, M, N), 1e-3, "bf16", 12, 1)
    b = gen((E, M, N), 1e-3, "f32", 12, 2)
    dW, dg, db = to_dev(W, "bf16"), to_dev(g, "bf16"), to_dev(b, "f32")
    muon.step([dW], [dg], [db])
    torch.cuda.synchronize()
    Wh = to_bits(dW)
    hp = ref.MuonHParams()
    for e in range(E):
        pw, pg, pb = to_dev(W[e], "bf16"), to_dev(g[e], "bf16"), to_dev(b[e], "f32")
        muon.step([pw], [pg], [pb])
        torch.cuda.synchronize()
        np.testing.assert_array_equal(to_bits(pw), Wh[e])
        r = ref.muon_step_matrix(decode(W[e], "bf16"), decode(g[e], "bf16"), b[e].astype(np.float64), hp)
        err, rho = w_gate(to_host(pw), r.W_new, decode(W[e], "bf16"), "bf16")
        assert err <= TOL["bf16"] + rho


def test_three_steps_equal_one_plus_resume(muon):
    import torch
    shapes = [(160, 96), (96, 96)]
    W = [gen(s, 0.02, "bf16", 13, i, 0) for i, s in enumerate(shapes)]
    b = [gen(s, 1e-3, "f32", 13, i, 2) for i, s in enumerate(shapes)]
    grads = [[to_dev(gen(s, 1e-3, "bf16", 13, i, 10 + t), "bf16") for i, s in enumerate(shapes)]
             for t in range(3)]
    dW = [to_dev(w, "bf16") for w in W]
    db = [to_dev(x, "f32") for x in b]
    for t in range(3):
        muon.step(dW, grads[t], db, weight_decay=0.1)
    torch.cuda.synchronize()
    dW2 = [to_dev(w, "bf16") for w in W]
    db2 = [to_dev(x, "f32") for x in b]
    muon.step(dW2, grads[0], db2, weight_decay=0.1)
    torch.cuda.synchronize()
    saved = [(t.cpu().clone(), m.cpu().clone()) for t, m in zip(dW2, db2)]
    del dW2, db2
    dW3 = [w.cuda() for w, _ in saved]
    db3 = [m.cuda() for _, m in saved]
    for t in (1, 2):
        muon.step(dW3, grads[t], db3, weight_decay=0.1)
    torch.cuda.synchronize()
    for x, y in zip(dW + db, dW3 + db3):
        np.testing.assert_array_equal(to_bits(x), to_bits(y))


def test_unaligned_views_take_the_scalar_path(muon):
    import torch
    rows, cols = 37, 45
    n = rows * cols
    Wf = gen((n + 3,), 0.02, "bf16", 14, 0)
    gf = gen((n + 5,), 1e-3, "bf16", 14, 1)
    bf = gen((n + 1,), 1e-3, "f32", 14, 2)
    dWf, dgf, dbf = to_dev(Wf, "bf16"), to_dev(gf, "bf16"), to_dev(bf, "f32")
    dW = dWf[3:3 + n].view(rows, cols)
    dg = dgf[5:5 + n].view(rows, cols)
    db = dbf[1:1 + n].view(rows, cols)
    muon.step([dW], [dg], [db])
    torch.cuda.synchronize()
    W0 = decode(Wf[3:3 + n], "bf16").reshape(rows, cols)
    r = ref.muon_step_matrix(W0, decode(gf[5:5 + n], "bf16").reshape(rows, cols),
                             bf[1:1 + n].astype(np.float64).reshape(rows, cols), ref.MuonHParams())
    err, rho = w_gate(to_host(dW), r.W_new, W0, "bf16")
    assert err <= TOL["bf16"] + rho
    assert (to_host(dWf[:3]) == decode(Wf[:3], "bf16")).all()  # neighbours untouched


def test_in_place_orthogonalize(muon):
    import torch
    g = gen((150, 90), 1.0, "bf16", 15, 0)
    t = to_dev(g, "bf16")
    muon.orthogonalize([t], [t])
    torch.cuda.synchronize()
    err, gate = o_gate(to_host(t), ref.orthogonalize(decode(g, "bf16"), 5), "bf16", "bf16")
    assert err <= gate, (err, gate)


def test_non_default_stream(muon):
    import torch
    shapes = [(256, 384)]
    base = _step_bits(muon, shapes, key=16)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        dW = [to_dev(gen(shapes[0], 0.02, "bf16", 16, 0, 0), "bf16")]
        dg = [to_dev(gen(shapes[0], 1e-3, "bf16", 16, 0, 1), "bf16")]
        db = [to_dev(gen(shapes[0], 1e-3, "f32", 16, 0, 2), "f32")]
        muon.step(dW, dg, db, stream=s)
    s.synchronize()
    np.testing.assert_array_equal(to_bits(dW[0]), base[0][0])


def test_second_stream_gives_the_same_bits(muon):
    # every bucket here fills few tiles, so its chunks alternate between the
    # caller's stream and the handle's second one; on a non-default caller
    # stream too, and with a workspace limit that leaves room for one slot
    # only (everything then runs on the caller's stream)
    import torch
    from paper_2609_21594_amd import binding as B
    shapes = [(512, 1024)] * 3 + [(768, 768)] + [(256, 256)] * 2 + [(200, 300)]
    muon.set_streams(1)
    try:
        base = _step_bits(muon, shapes, key=27)
    finally:
        muon.set_streams(2)
    two = _step_bits(muon, shapes, key=27)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        other = _step_bits(muon, shapes, key=27, stream=s)
    W = [to_dev(gen(sh, 0.02, "bf16", 27, i, 0), "bf16") for i, sh in enumerate(shapes)]
    arr, keep = B.params_array(W, W, [torch.zeros(sh, device="cuda") for sh in shapes])
    hp, keep2 = B.make_hparams()
    _, _, one_slot, _ = B.plan_step(list(arr)[:len(shapes)], hp)
    lim = B.Muon(0)
    try:
        lim.set_workspace_limit(one_slot)
        limited = _step_bits(lim, shapes, key=27)
    finally:
        lim.close()
    for run in (two, other, limited):
        for x, y in zip(base[0] + base[1], run[0] + run[1]):
            np.testing.assert_array_equal(x, y)
    with pytest.raises(B.MuonError):
        muon.set_streams(3)


def test_workspace_growth_between_calls_on_two_streams():
    # one handle and no host synchronisation between its calls: a small call
    # on a side stream, a larger one on the current stream (the workspace
    # grows: the handle waits for its own earlier call before freeing the old
    # one), and the small one again on the side stream; each result equals
    # the same call made alone on a fresh handle
    import torch
    from paper_2609_21594_amd.binding import Muon
    require_gpu()
    small = [(256, 512), (512, 256)]
    large = [(1024, 2048), (2048, 1024), (768, 768)]
    calls = [(small, 41), (large, 42), (small, 43)]
    want = []
    for shapes, key in calls:
        ref_h = Muon(0)
        try:
            want.append(_step_bits(ref_h, shapes, key=key))
        finally:
            ref_h.close()
    args = [([to_dev(gen(s, 0.02, "bf16", key, i, 0), "bf16") for i, s in enumerate(shapes)],
             [to_dev(gen(s, 1e-3, "bf16", key, i, 1), "bf16") for i, s in enumerate(shapes)],
             [to_dev(gen(s, 1e-3, "f32", key, i, 2), "f32") for i, s in enumerate(shapes)])
            for shapes, key in calls]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    h = Muon(0)
    try:
        sizes = []
        for (W, g, m), st in zip(args, (side, None, side)):
            h.step(W, g, m, ns_precision="bf16", stream=st)
            sizes.append(h.workspace_bytes)
        torch.cuda.synchronize()
    finally:
        h.close()
    assert sizes[1] > sizes[0] and sizes[2] == sizes[1]
    for (W, g, m), (wW, wm) in zip(args, want):
        for x, y in zip([to_bits(t) for t in W] + [to_bits(t) for t in m], wW + wm):
            np.testing.assert_array_equal(x, y)


def test_errors_leave_buffers_untouched(muon):
    import torch
    from paper_2609_21594_amd.binding import Muon, MuonError
    W = gen((64, 64), 0.02, "bf16", 17, 0)
    dW = to_dev(W, "bf16")
    dg = to_dev(gen((64, 64), 1e-3, "bf16", 17, 1), "bf16")
    db = to_dev(gen((64, 64), 1e-3, "f32", 17, 2), "f32")
    with pytest.raises(MuonError) as e:
        muon.step([dW], [dg], [db], ns_steps=-1)
    assert e.value.status == 1
    with pytest.raises(MuonError) as e:
        muon.step([dW], [dW], [db])  # grad aliases param
    assert e.value.status == 1
    small = Muon(0)
    small.set_workspace_limit(1024)
    with pytest.raises(MuonError) as e:
        small.step([dW], [dg], [db])
    assert e.value.status == 3
    small.close()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_bits(dW), to_bits(to_dev(W, "bf16")))
