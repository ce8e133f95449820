"""A repeated request reuses the handle's cached checks and plan: results
must equal, bit for bit, those of a fresh handle (which plans from scratch),
call after call, with eager work and host synchronisations in between; lr
and weight decay may change from call to call, and a different request in
between takes its own plan."""
import numpy as np
import pytest

from paper_2609_21594_amd import synth
from tests.gpu_util import require_gpu, to_bits, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([synth.ROOT_SEED, 7300, *key])))


@pytest.mark.parametrize("shapes,prec", [
    ([(512, 1024), (1024, 512), (768, 768), (256, 256), (256, 256)], "bf16"),   # tile kernels, two streams
    ([(300, 200), (129, 257)], "bf16"),                                          # 128 x 128 kernel
    ([(256, 128), (64, 300), (7, 90)], "f32"),                                   # fused small launch
])
def test_cached_request_equals_fresh_plans(muon, shapes, prec):
    import torch
    from paper_2609_21594_amd.binding import Muon
    W = [synth.draw(s, 0.02, "bf16", rng(len(shapes), i, 0)) for i, s in enumerate(shapes)]
    G = [synth.draw(s, 1e-3, "bf16", rng(len(shapes), i, 1)) for i, s in enumerate(shapes)]
    B = [synth.draw(s, 1e-3, "f32", rng(len(shapes), i, 2)) for i, s in enumerate(shapes)]
    dev = [[to_dev(w, "bf16") for w in W], [to_dev(g, "bf16") for g in G], [to_dev(b, "f32") for b in B]]
    dev2 = [[t.clone() for t in lst] for lst in dev]
    other = [torch.zeros(64, 96, dtype=torch.bfloat16, device="cuda") for _ in range(3)]
    other[2] = other[2].float()
    scratch = torch.zeros(1 << 20, device="cuda")
    for step, lr in enumerate([0.02, 0.02, 0.015, 0.01, 0.02]):
        kw = dict(lr=lr, beta=0.95, weight_decay=0.05 * step, ns_precision=prec)
        muon.step(*dev, **kw)                 # cached from the second call on
        fresh = Muon(0)
        fresh.step(*dev2, **kw)
        fresh.close()
        if step == 2:                         # another request in between
            muon.step([other[0]], [other[1]], [other[2]], lr=0.01)
        scratch.add_(1.0)
        torch.cuda.synchronize()
        for a, b in zip(dev[0] + dev[2], dev2[0] + dev2[2]):
            assert np.array_equal(to_bits(a), to_bits(b)), (step, a.shape)


def test_cached_orthogonalize_equals_fresh(muon):
    import torch
    from paper_2609_21594_amd.binding import Muon
    for shapes in ([(512, 1024), (256, 768)], [(512, 1024), (256, 768)], [(384, 384)], [(512, 1024), (256, 768)]):
        G = [to_dev(synth.draw(s, 1.0, "bf16", rng(9, i)), "bf16") for i, s in enumerate(shapes)]
        o1 = [torch.empty_like(t) for t in G]
        o2 = [torch.empty_like(t) for t in G]
        muon.orthogonalize(G, o1)
        fresh = Muon(0)
        fresh.orthogonalize(G, o2)
        fresh.close()
        torch.cuda.synchronize()
        for a, b in zip(o1, o2):
            assert np.array_equal(to_bits(a), to_bits(b))
