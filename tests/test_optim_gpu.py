"""The torch optimizer over the library (Muon for matrices, chained AdamW
for the rest, Sec. 6.4): its steps equal direct library calls bit for bit,
per group and with parameters whose first gradient comes late, and its
state_dict restores a run exactly."""
import copy

import numpy as np
import pytest

from paper_2609_21594_amd import synth
from tests.gpu_util import require_gpu, to_bits

pytestmark = pytest.mark.gpu

SHAPES = [(256, 512), (768, 256), (3, 128, 64), (512,), (256,), ()]


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([8181, *key])))


def tensor(shape, sigma, key, dtype):
    import torch
    a = synth.draw(shape if shape else (1,), sigma, "f32", rng(*key)).reshape(shape)
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype=dtype, device="cuda")


def make_params(dtype):
    import torch
    return [torch.nn.Parameter(tensor(s, 0.02, (i, 0), dtype)) for i, s in enumerate(SHAPES)]


def set_grads(params, t):
    for i, p in enumerate(params):
        p.grad = tensor(tuple(p.shape), 1e-3, (i, 1, t), p.dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_optimizer_equals_direct_calls(dtype):
    require_gpu()
    import torch
    from paper_2609_21594_amd.binding import Muon
    from paper_2609_21594_amd.optim import MuonAdamW
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    P = make_params(dt)
    P0 = [p.detach().clone() for p in P]
    Q = [torch.nn.Parameter(p.detach().clone()) for p in P]
    opt = MuonAdamW(P, lr=0.03, weight_decay=0.01, adamw_lr=1e-3, adamw_weight_decay=0.1)
    lib = Muon(0)
    mats = [q for q in Q if q.dim() in (2, 3)]
    vecs = [q for q in Q if q.dim() not in (2, 3)]
    moms = [torch.zeros(q.shape, dtype=torch.float32, device="cuda") for q in mats]
    ms = [torch.zeros(q.shape, dtype=torch.float32, device="cuda") for q in vecs]
    vs = [torch.zeros(q.shape, dtype=torch.float32, device="cuda") for q in vecs]
    try:
        for t in (1, 2, 3):
            set_grads(P, t)
            set_grads(Q, t)
            opt.step()
            lib.step(mats, [q.grad for q in mats], moms, lr=0.03, beta=0.95, weight_decay=0.01)
            lib.adamw_step(vecs, [q.grad for q in vecs], ms, vs, t, lr=1e-3, betas=(0.9, 0.95),
                           weight_decay=0.1)
        torch.cuda.synchronize()
        for p, q, p0 in zip(P, Q, P0):
            np.testing.assert_array_equal(to_bits(p.detach()), to_bits(q.detach()))
            assert not torch.equal(p.detach(), p0)  # it moved
        for p, m in zip([p for p in P if p.dim() in (2, 3)], moms):
            np.testing.assert_array_equal(to_bits(opt.state[p]["momentum_buffer"]), to_bits(m))
    finally:
        opt.close()
        lib.close()


def test_groups_late_parameters_and_state_dict():
    require_gpu()
    import torch
    from paper_2609_21594_amd.optim import MuonAdamW
    P = make_params(torch.bfloat16)
    # two groups: the first matrix with its own lr and forced to AdamW
    groups = [{"params": P[:1], "lr": 0.05, "use_muon": False}, {"params": P[1:]}]
    opt = MuonAdamW(groups, lr=0.02, adamw_lr=2e-3)
    try:
        for t in (1, 2):
            set_grads(P, t)
            P[3].grad = None if t == 1 else P[3].grad  # the (512,) vector joins at step 2
            opt.step()
        assert int(opt.state[P[0]]["step"]) == 2 and "momentum_buffer" not in opt.state[P[0]]
        assert int(opt.state[P[3]]["step"]) == 1 and int(opt.state[P[4]]["step"]) == 2
        saved = copy.deepcopy(opt.state_dict())  # state_dict() holds live references
        snap = [p.detach().clone() for p in P]
        set_grads(P, 3)
        opt.step()
        after = [to_bits(p.detach()) for p in P]
        # restore parameters and optimizer state into a fresh optimizer
        with torch.no_grad():
            for p, s in zip(P, snap):
                p.copy_(s)
        opt2 = MuonAdamW(groups, lr=0.02, adamw_lr=2e-3)
        try:
            opt2.load_state_dict(saved)
            set_grads(P, 3)
            opt2.step()
            torch.cuda.synchronize()
            for p, a in zip(P, after):
                np.testing.assert_array_equal(to_bits(p.detach()), a)
            for p in P:  # the moments came back fp32
                for k, v in opt2.state[p].items():
                    assert k == "step" or v.dtype == torch.float32
        finally:
            opt2.close()
    finally:
        opt.close()


def test_trains_a_small_mlp():
    # autograd forward/backward in torch (fp32), updates by the library: the
    # weights (2-D) take Muon, the biases AdamW; a fixed random target
    # function is fitted, and the loss must fall well below where it starts
    require_gpu()
    import torch
    from paper_2609_21594_amd.optim import MuonAdamW
    g = torch.Generator(device="cpu").manual_seed(1234)
    X = torch.randn(512, 64, generator=g).cuda()
    A, Bm = torch.randn(64, 48, generator=g).cuda() / 8, torch.randn(48, 16, generator=g).cuda() / 7
    Y = torch.tanh(X @ A) @ Bm
    torch.manual_seed(0)
    model = torch.nn.Sequential(torch.nn.Linear(64, 128), torch.nn.Tanh(), torch.nn.Linear(128, 16)).cuda()
    opt = MuonAdamW(model.parameters(), lr=0.02, weight_decay=0.0, adamw_lr=3e-3)
    start = [p.detach().clone() for p in model.parameters()]
    losses = []
    try:
        for _ in range(60):
            loss = torch.nn.functional.mse_loss(model(X), Y)
            opt.zero_grad()
            loss.backward()
            opt.step()
            losses.append(float(loss.detach()))
    finally:
        opt.close()
    print(f"mlp loss {losses[0]:.4f} -> {losses[-1]:.4f}", flush=True)
    assert losses[-1] < 0.25 * losses[0], losses[::10]
    for p, p0 in zip(model.parameters(), start):
        assert not torch.equal(p.detach(), p0)
