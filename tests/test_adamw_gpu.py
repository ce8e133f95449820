"""AdamW for the parameters Muon does not take (Sec. 6.4 chains it for the
one-dimensional and scalar ones), through the C ABI, against the oracle.

Each step starts the oracle from the values the GPU holds, so every step is
compared on identical inputs.  Moments are fp32 on the GPU: relative error
<= 1e-6.  The parameter's change matches the oracle's change to 1e-5
(fp32 parameters), or within the bf16 rounding floor plus 1e-5 (bf16).
"""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import decode, rel, require_gpu, to_bits, to_dev, to_host

pytestmark = pytest.mark.gpu

# scalars, an unaligned tail, block boundaries (8192 per workgroup), and
# several blocks
SIZES = [1, 7, 8, 8191, 8192, 8193, 100003, 1 << 20]
HP = ref.AdamWHParams(lr=3e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([7373, *key])))


def call(muon, ps, gs, ms, vs, t, hp=HP):
    muon.adamw_step(ps, gs, ms, vs, t, lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                    weight_decay=hp.weight_decay)


@pytest.mark.parametrize("pdt,gdt", [("bf16", "bf16"), ("f32", "f32"), ("f32", "bf16"), ("bf16", "f32")])
def test_adamw_matches_oracle(muon, pdt, gdt):
    import torch
    ps = [to_dev(synth.draw((n,), 0.02, pdt, rng(n, 0)), pdt) for n in SIZES]
    ms = [torch.zeros(n, dtype=torch.float32, device="cuda") for n in SIZES]
    vs = [torch.zeros(n, dtype=torch.float32, device="cuda") for n in SIZES]
    for t in (1, 2, 3):
        gn = [synth.draw((n,), 1e-3, gdt, rng(n, t)) for n in SIZES]
        gs = [to_dev(g, gdt) for g in gn]
        before = [(to_host(p), to_host(m), to_host(v)) for p, m, v in zip(ps, ms, vs)]
        call(muon, ps, gs, ms, vs, t)
        torch.cuda.synchronize()
        for n, (p0, m0, v0), g, p, m, v in zip(SIZES, before, gn, ps, ms, vs):
            pr, mr, vr = ref.adamw_step(p0, decode(g, gdt), m0, v0, t, HP)
            assert rel(to_host(m), mr) <= 1e-6, (n, t)
            assert rel(to_host(v), vr) <= 1e-6, (n, t)
            d = float(np.linalg.norm(pr - p0))
            err = float(np.linalg.norm(to_host(p) - pr)) / d
            rho = float(np.linalg.norm(ref.round_to(pr, pdt) - pr)) / d
            assert err <= 1e-5 + rho, (n, t, err, rho)


def test_vector_and_element_paths_agree_bitwise(muon):
    # the same values, once 16-byte aligned (8 elements per thread) and once
    # one element off (element by element)
    import torch
    n = 3 * 8192 + 40
    pn = synth.draw((n,), 0.02, "bf16", rng(1, 0))
    gn = synth.draw((n,), 1e-3, "bf16", rng(1, 1))
    mn = synth.draw((n,), 1e-4, "f32", rng(1, 2))
    vn = np.abs(synth.draw((n,), 1e-6, "f32", rng(1, 3)))
    out = []
    for off in (0, 1):
        def place(a, dt):
            big = to_dev(np.concatenate([np.zeros(off, a.dtype), a]), dt)
            return big[off:]
        p, g, m, v = place(pn, "bf16"), place(gn, "bf16"), place(mn, "f32"), place(vn, "f32")
        assert (p.data_ptr() % 16 == 0) == (off == 0)
        call(muon, [p], [g], [m], [v], 4)
        torch.cuda.synchronize()
        out.append([to_bits(x.contiguous()) for x in (p, m, v)])
    for a, b in zip(*out):
        assert np.array_equal(a, b)


def test_zero_gradient_is_pure_decay(muon):
    import torch
    n = 5000
    pn = synth.draw((n,), 1.0, "f32", rng(2, 0))
    p = to_dev(pn, "f32")
    z = lambda: torch.zeros(n, dtype=torch.float32, device="cuda")
    m, v = z(), z()
    call(muon, [p], [z()], [m], [v], 1)
    torch.cuda.synchronize()
    want = (1 - HP.lr * HP.weight_decay) * pn.astype(np.float64)
    assert rel(to_host(p), want) <= 1e-7
    assert not to_host(m).any() and not to_host(v).any()


def test_errors_leave_buffers_untouched(muon):
    import torch
    from paper_2609_21594_amd.binding import MuonError
    p = to_dev(synth.draw((64,), 1.0, "f32", rng(3, 0)), "f32")
    g = to_dev(synth.draw((64,), 1.0, "f32", rng(3, 1)), "f32")
    m = torch.zeros(64, dtype=torch.float32, device="cuda")
    before = to_bits(p)
    for kw in (dict(step=0), dict(betas=(1.0, 0.9)), dict(eps=0.0), dict(lr=float("nan"))):
        args = dict(step=1, lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
        args.update(kw)
        with pytest.raises(MuonError):
            muon.adamw_step([p], [g], [m], [m], **args)  # also: m given twice
    with pytest.raises(MuonError):
        muon.adamw_step([p], [g], [m], [m], 1)  # the two moments overlap
    torch.cuda.synchronize()
    assert np.array_equal(to_bits(p), before)
