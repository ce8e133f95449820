"""Per-parameter stages (Sec. 6.2: step count, coefficients and scaling are
configurable per parameter), through the C ABI.

One call with per-entry coefficient tables and scale modes must give every
entry the bits a call that uses those settings for all its entries gives it
(a matrix's result does not depend on what shares its call), and each entry
must match the oracle with its own settings.
"""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import MOMENTUM_TOL, decode, rel, require_gpu, to_bits, to_dev, to_host, tol_for, w_gate

pytestmark = pytest.mark.gpu

QUINTIC = (3.4445, -4.7750, 2.0315)
CUBIC3 = [(1.5, -0.5, 0.0)] * 3
MIXED8 = [(15 / 8, -10 / 8, 3 / 8)] * 4 + [QUINTIC] * 4


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([6262, *key])))


def inputs(shapes, key):
    W = [synth.draw(s, 0.02, "bf16", rng(key, i, 0)) for i, s in enumerate(shapes)]
    g = [synth.draw(s, 1e-3, "bf16", rng(key, i, 1)) for i, s in enumerate(shapes)]
    m = [synth.draw(s, 1e-3, "f32", rng(key, i, 2)) for i, s in enumerate(shapes)]
    return W, g, m


def device(W, g, m):
    return [to_dev(a, "bf16") for a in W], [to_dev(a, "bf16") for a in g], [to_dev(a, "f32") for a in m]


@pytest.mark.parametrize("shapes", [[(512, 1024), (1024, 512), (512, 1024), (1024, 512)],
                                    [(200, 300), (300, 200), (200, 300), (300, 200)]])
def test_per_entry_options_match_uniform_calls_and_oracle(muon, shapes):
    import torch
    # lr large enough that the update stands well above the bf16 rounding of
    # W for every scale rule
    hpk = dict(lr=0.2, beta=0.95, weight_decay=0.01, ns_precision="bf16")
    W, g, m = inputs(shapes, (len(shapes), shapes[0][0]))
    # entry 0: the call's table and scale; entry 1: the cubic table and the
    # original Muon scale; entry 2: an 8-step table; entry 3: no steps
    # (O = X0) without any rescale
    opts = [(None, None), (CUBIC3, 2), (MIXED8, None), ([], 1)]  # the last: K = 0
    Wd, gd, md = device(W, g, m)
    muon.step(Wd, gd, md, entry_coeffs=[o[0] for o in opts], entry_scale_modes=[o[1] for o in opts],
              **hpk)
    for i, (coeffs, smode) in enumerate(opts):
        Wu, gu, mu = device([W[i]], [g[i]], [m[i]])
        kw = dict(hpk)
        if coeffs is not None:
            kw.update(ns_coeffs=coeffs if coeffs else None, ns_steps=len(coeffs))
        if smode is not None:
            kw.update(scale_mode=smode)
        muon.step(Wu, gu, mu, **kw)
        torch.cuda.synchronize()
        assert np.array_equal(to_bits(Wd[i]), to_bits(Wu[0])), i
        assert np.array_equal(to_bits(md[i]), to_bits(mu[0])), i
        hp = ref.MuonHParams(lr=0.2, beta=0.95, weight_decay=0.01,
                             ns_steps=len(coeffs) if coeffs is not None else 5, ns_coeffs=coeffs,
                             scale_mode=smode or 0)
        W0 = decode(W[i], "bf16")
        r = ref.muon_step_matrix(W0, decode(g[i], "bf16"), np.asarray(m[i], np.float64), hp)
        err, rho = w_gate(to_host(Wd[i]), r.W_new, W0, "bf16")
        print(f"entry {i} {shapes[i]}: err {err:.3e} (rho {rho:.1e})", flush=True)
        assert err <= tol_for("bf16", shapes[i]) + rho, (i, err, rho)
        assert rel(to_host(md[i]), r.buf_new) <= MOMENTUM_TOL


def test_original_muon_scale_on_the_call(muon):
    # scale_mode 2 for a whole call: a tall matrix is scaled by
    # sqrt(rows / cols), a wide one by 1
    import torch
    shapes = [(1024, 256), (256, 768)]
    W, g, m = inputs(shapes, (9,))
    Wd, gd, md = device(W, g, m)
    muon.step(Wd, gd, md, lr=0.2, beta=0.95, weight_decay=0.0, ns_precision="bf16", scale_mode=2)
    torch.cuda.synchronize()
    hp = ref.MuonHParams(lr=0.2, beta=0.95, weight_decay=0.0, scale_mode=2)
    for i, s in enumerate(shapes):
        W0 = decode(W[i], "bf16")
        r = ref.muon_step_matrix(W0, decode(g[i], "bf16"), np.asarray(m[i], np.float64), hp)
        err, rho = w_gate(to_host(Wd[i]), r.W_new, W0, "bf16")
        print(f"scale mode 2 {s}: err {err:.3e} (rho {rho:.1e})", flush=True)
        assert err <= tol_for("bf16", s) + rho, (s, err, rho)


@pytest.mark.parametrize("hd,d", [(64, 256), (256, 1024)])
def test_post_scale_per_head_qk_clip(muon, hd, d):
    # A QK-clip-style post-processing stage (Sec. 6.2): each head's query and
    # key slices of a fused [H, 3, hd, d] QKV weight are separate entries
    # (zero-copy views) with their own factor; values take none.  64 x 256
    # runs on the fused small-matrix launch, 256 x 1024 on the tile kernels.
    import torch
    H = 4
    shape = (H, 3, hd, d)
    Wf = synth.draw(shape, 0.02, "bf16", rng(90, hd, 0))
    gf = synth.draw(shape, 1e-3, "bf16", rng(90, hd, 1))
    mf = synth.draw(shape, 1e-3, "f32", rng(90, hd, 2))
    eta = [0.5, 0.8, 1.0, 0.65]                      # per-head clip factors
    post = [[np.sqrt(e), np.sqrt(e), None] for e in eta]
    hp = ref.MuonHParams(lr=0.02, beta=0.95, weight_decay=0.01)
    results = {}
    for use in (True, False):
        Wd, gd, md = to_dev(Wf, "bf16"), to_dev(gf, "bf16"), to_dev(mf, "f32")
        P = [Wd[h, j] for h in range(H) for j in range(3)]
        G = [gd[h, j] for h in range(H) for j in range(3)]
        M = [md[h, j] for h in range(H) for j in range(3)]
        scales = [post[h][j] for h in range(H) for j in range(3)] if use else None
        muon.step(P, G, M, lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, entry_post_scales=scales)
        torch.cuda.synchronize()
        results[use] = (to_host(Wd), to_bits(Wd), to_host(md))
    W0 = decode(Wf, "bf16")
    for h in range(H):
        for j in range(3):
            r = ref.muon_step_matrix(W0[h, j], decode(gf[h, j], "bf16"), np.asarray(mf[h, j], np.float64),
                                     ref.MuonHParams(lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay,
                                                     post_scale=post[h][j] or 1.0))
            err, rho = w_gate(results[True][0][h, j], r.W_new, W0[h, j], "bf16")
            # the gate is relative to this entry's change, which the factor makes large
            print(f"post scale {post[h][j]} head {h} slice {j} ({hd}x{d}): W err {err:.3e} (rho {rho:.1e})", flush=True)
            assert err <= tol_for("bf16", (hd, d)) + rho, (h, j, err, rho)
            assert rel(results[True][2][h, j], r.buf_new) <= MOMENTUM_TOL
            if post[h][j] is None:   # untouched entries: the bits of the plain call
                assert np.array_equal(results[True][1][h, j], results[False][1][h, j]), (h, j)
    # the momentum does not depend on the stage
    assert np.array_equal(results[True][2], results[False][2])
