"""The fused small-matrix launch (short side <= 128; always for fp32
Newton-Schulz, for bf16 when the short side is <= 64 or the long side <= 512):
element-wise parity with the oracle over short sides 1..128 and long sides
128..2048, both orientations, K = 0, 1 and 5; many matrices sharing groups of
workgroups; batching and repeat determinism.  The bf16 shapes cover both the
fused launch and, for 128 x 2048 and 2048 x 128, the 128 x 128 tile kernel,
against the bf16 gate."""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import MOMENTUM_TOL, TOL, decode, o_gate, rel, require_gpu, to_bits, to_dev, to_host, tol_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([synth.ROOT_SEED, 7100, *key])))


SHORT = [1, 7, 64, 128]
LONG = [128, 300, 2048]
LONG_BF16 = [128, 300, 512, 2048]


@pytest.mark.parametrize("steps", [5, 1, 0])
def test_small_orthogonalize_matches_oracle(muon, steps):
    import torch
    shapes = [(s, l) for s in SHORT for l in LONG] + [(l, s) for s in (7, 128) for l in LONG]
    G = [synth.draw(sh, 1.0, "f32", rng(steps, i)) for i, sh in enumerate(shapes)]
    ins = [to_dev(g, "f32") for g in G]
    outs = [torch.full_like(t, float("nan")) for t in ins]
    muon.orthogonalize(ins, outs, ns_steps=steps, ns_precision="f32")
    torch.cuda.synchronize()
    for sh, g, o in zip(shapes, G, outs):
        err = rel(to_host(o), ref.orthogonalize(decode(g, "f32"), steps))
        print(f"small fp32 K={steps} {sh}: O err {err:.2e}", flush=True)
        assert err <= TOL["f32"], (sh, err)


@pytest.mark.parametrize("steps", [5, 1, 0])
def test_small_shapes_bf16_path_match_oracle(muon, steps):
    # K = 0 writes X0 = r u from the prologue; K = 1 applies r in the last
    # step's products themselves
    import torch
    shapes = [(s, l) for s in SHORT for l in LONG_BF16] + [(l, s) for s in (7, 128) for l in LONG_BF16]
    G = [synth.draw(sh, 1.0, "bf16", rng(50, steps, i)) for i, sh in enumerate(shapes)]
    ins = [to_dev(g, "bf16") for g in G]
    outs = [torch.full_like(t, float("nan")) for t in ins]
    muon.orthogonalize(ins, outs, ns_steps=steps, ns_precision="bf16")
    torch.cuda.synchronize()
    for sh, g, o in zip(shapes, G, outs):
        x = decode(g, "bf16")
        err, gate = o_gate(to_host(o), ref.orthogonalize(x, steps), "bf16", "bf16", steps, G=x)
        print(f"small bf16 K={steps} {sh}: O err {err:.2e} (gate {gate:.2e})", flush=True)
        assert err <= gate, (sh, err, gate)


@pytest.mark.parametrize("pdt", ["f32", "bf16"])
def test_small_step_matches_oracle(muon, pdt):
    import torch
    shapes = [(256, 128), (128, 256), (7, 2048), (2048, 7), (64, 300), (1, 128)]
    hp = ref.MuonHParams(lr=0.02, beta=0.95, weight_decay=0.1, nesterov=True)
    Ws = [synth.draw(sh, 0.02 if pdt == "bf16" else 1.0, pdt, rng(30, i, 0)) for i, sh in enumerate(shapes)]
    gs = [synth.draw(sh, 1.0, "f32", rng(30, i, 1)) for i, sh in enumerate(shapes)]
    bs = [synth.draw(sh, 1.0, "f32", rng(30, i, 2)) for i, sh in enumerate(shapes)]
    dW, dg, db = [to_dev(w, pdt) for w in Ws], [to_dev(g, "f32") for g in gs], [to_dev(b, "f32") for b in bs]
    muon.step(dW, dg, db, lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, ns_precision="f32")
    torch.cuda.synchronize()
    for sh, W, g, b, w_dev, b_dev in zip(shapes, Ws, gs, bs, dW, db):
        W0 = decode(W, pdt)
        r = ref.muon_step_matrix(W0, decode(g, "f32"), np.asarray(b, np.float64), hp)
        d = np.linalg.norm(r.W_new - W0)
        err = np.linalg.norm(to_host(w_dev) - r.W_new) / d
        rho = np.linalg.norm(ref.round_to(r.W_new, pdt) - r.W_new) / d
        print(f"small step {pdt} {sh}: W err {err:.2e} (rho {rho:.1e})", flush=True)
        assert err <= TOL["f32"] + rho, (sh, err, rho)
        assert rel(to_host(b_dev), r.buf_new) <= MOMENTUM_TOL, sh


def test_small_many_matrices_share_groups_and_match_single_calls(muon):
    # 70 matrices: more than one matrix per group of workgroups; each result
    # equal, bit for bit, to the same matrix in a call of its own
    import torch
    shapes = [(96, 160)] * 40 + [(160, 96)] * 30
    G = [synth.draw(sh, 1.0, "f32", rng(40, i)) for i, sh in enumerate(shapes)]
    ins = [to_dev(g, "f32") for g in G]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_precision="f32")
    torch.cuda.synchronize()
    for i in (0, 17, 39, 40, 69):
        one = torch.empty_like(ins[i])
        muon.orthogonalize([ins[i]], [one], ns_precision="f32")
        torch.cuda.synchronize()
        assert np.array_equal(to_bits(one), to_bits(outs[i])), i
        assert rel(to_host(outs[i]), ref.orthogonalize(decode(G[i], "f32"), 5)) <= TOL["f32"]
    again = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, again, ns_precision="f32")
    torch.cuda.synchronize()
    assert all(np.array_equal(to_bits(a), to_bits(b)) for a, b in zip(outs, again))


@pytest.mark.parametrize("prec", ["bf16", "f32"])
def test_small_step_with_bf16_grads(muon, prec):
    # muon_step over bf16 parameters and gradients, the Newton-Schulz products
    # in either precision: the fused launch (and the tile path for 128 x 2048)
    import torch
    shapes = [(64, 300), (300, 64), (7, 2048), (128, 512), (512, 128), (1, 128), (128, 2048)]
    hp = ref.MuonHParams(lr=0.02, beta=0.95, weight_decay=0.1, nesterov=True)
    Ws = [synth.draw(sh, 0.02, "bf16", rng(60, i, 0)) for i, sh in enumerate(shapes)]
    gs = [synth.draw(sh, 1e-3, "bf16", rng(60, i, 1)) for i, sh in enumerate(shapes)]
    bs = [synth.draw(sh, 1e-3, "f32", rng(60, i, 2)) for i, sh in enumerate(shapes)]
    dW, dg, db = [to_dev(w, "bf16") for w in Ws], [to_dev(g, "bf16") for g in gs], [to_dev(b, "f32") for b in bs]
    muon.step(dW, dg, db, lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, ns_precision=prec)
    torch.cuda.synchronize()
    for sh, W, g, b, w_dev, b_dev in zip(shapes, Ws, gs, bs, dW, db):
        W0 = decode(W, "bf16")
        r = ref.muon_step_matrix(W0, decode(g, "bf16"), np.asarray(b, np.float64), hp)
        d = np.linalg.norm(r.W_new - W0)
        err = np.linalg.norm(to_host(w_dev) - r.W_new) / d
        rho = np.linalg.norm(ref.round_to(r.W_new, "bf16") - r.W_new) / d
        gate = tol_for(prec, sh)
        print(f"small step bf16 params, {prec} NS {sh}: W err {err:.2e} (gate {gate:.1e} + rho {rho:.1e})", flush=True)
        assert err <= gate + rho, (sh, err, gate, rho)
        assert rel(to_host(b_dev), r.buf_new) <= MOMENTUM_TOL, sh


def test_small_bf16_batching_and_repeats_are_bitwise_stable(muon):
    # bf16 Newton-Schulz on the fused launch: each matrix of a 60-matrix call
    # equal, bit for bit, to the same matrix alone, and to a repeat
    import torch
    shapes = [(64, 300)] * 30 + [(300, 48)] * 20 + [(128, 512)] * 10
    G = [synth.draw(sh, 1.0, "bf16", rng(70, i)) for i, sh in enumerate(shapes)]
    ins = [to_dev(g, "bf16") for g in G]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_precision="bf16")
    torch.cuda.synchronize()
    for i in (0, 29, 30, 49, 50, 59):
        one = torch.empty_like(ins[i])
        muon.orthogonalize([ins[i]], [one], ns_precision="bf16")
        torch.cuda.synchronize()
        assert np.array_equal(to_bits(one), to_bits(outs[i])), i
        x = decode(G[i], "bf16")
        err, gate = o_gate(to_host(outs[i]), ref.orthogonalize(x, 5), "bf16", "bf16", G=x)
        assert err <= gate, (i, err, gate)
    again = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, again, ns_precision="bf16")
    torch.cuda.synchronize()
    assert all(np.array_equal(to_bits(a), to_bits(b)) for a, b in zip(outs, again))


def test_workload1_speed_record(muon):
    # not a gate: the fused launch's time for the 256 x 128 fp32 step, printed
    import time
    import torch
    wl = synth.WORKLOADS[1]
    m = synth.make_matrix(wl, 0)
    dW, dg, db = to_dev(m.W, "f32"), to_dev(m.g, "f32"), to_dev(m.buf, "f32")
    kw = dict(lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay, ns_precision="f32")
    for _ in range(5):
        muon.step([dW], [dg], [db], **kw)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(50):
        muon.step([dW], [dg], [db], **kw)
    torch.cuda.synchronize()
    print(f"workload 1: {(time.perf_counter() - t0) / 50 * 1e3:.3f} ms per step", flush=True)
