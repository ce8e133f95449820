"""Pins of the oracle's AdamW (the optimizer Sec. 6.4 chains for the
parameters Muon does not take) to things other than itself: torch's own
AdamW in float64 on the CPU (an independent library routine), hand-worked
first steps, and pure decay under a zero gradient."""
import numpy as np
import pytest

from oracle import muon_ref as ref


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_matches_torch_adamw_over_several_steps(wd):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(31)
    shapes = [(7,), (3, 5), (1,)]
    ps = [rng.standard_normal(s) for s in shapes]
    hp = ref.AdamWHParams(lr=0.01, beta1=0.8, beta2=0.95, eps=1e-6, weight_decay=wd)
    tp = [torch.tensor(p, dtype=torch.float64, requires_grad=True) for p in ps]
    opt = torch.optim.AdamW(tp, lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.eps,
                            weight_decay=wd, foreach=False)
    ms = [np.zeros(s) for s in shapes]
    vs = [np.zeros(s) for s in shapes]
    for t in range(1, 5):
        gs = [rng.standard_normal(s) for s in shapes]
        for x, g in zip(tp, gs):
            x.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        for i in range(len(shapes)):
            ps[i], ms[i], vs[i] = ref.adamw_step(ps[i], gs[i], ms[i], vs[i], t, hp)
        for i, x in enumerate(tp):
            st = opt.state[x]
            np.testing.assert_allclose(ps[i], x.detach().numpy(), rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(ms[i], st["exp_avg"].numpy(), rtol=1e-13, atol=1e-15)
            np.testing.assert_allclose(vs[i], st["exp_avg_sq"].numpy(), rtol=1e-13, atol=1e-15)


def test_first_step_by_hand():
    # t = 1 from zero moments: m_hat = g and v_hat = g^2, so the step is
    # lr * g / (|g| + eps): with g = 2, -0.5, 0, lr = 0.1, eps = 1e-8 the
    # changes are -0.1 * 2/(2 + 1e-8), +0.1 * 0.5/(0.5 + 1e-8) and 0
    hp = ref.AdamWHParams(lr=0.1, beta1=0.9, beta2=0.999, eps=1e-8)
    p = np.array([1.0, 1.0, 1.0])
    g = np.array([2.0, -0.5, 0.0])
    p1, m1, v1 = ref.adamw_step(p, g, np.zeros(3), np.zeros(3), 1, hp)
    np.testing.assert_allclose(p1 - p, [-0.1 * 2 / (2 + 1e-8), 0.1 * 0.5 / (0.5 + 1e-8), 0.0],
                               rtol=1e-14, atol=0)
    np.testing.assert_allclose(m1, [0.2, -0.05, 0.0], rtol=1e-15)
    np.testing.assert_allclose(v1, [0.004, 0.00025, 0.0], rtol=1e-12)


def test_zero_gradient_and_moments_is_pure_decay():
    hp = ref.AdamWHParams(lr=0.02, weight_decay=0.5)
    p = np.linspace(-1, 1, 9)
    z = np.zeros(9)
    p1, m1, v1 = ref.adamw_step(p, z, z, z, 3, hp)
    np.testing.assert_array_equal(p1, (1 - 0.02 * 0.5) * p)
    np.testing.assert_array_equal(m1, 0.0)
    np.testing.assert_array_equal(v1, 0.0)


def test_step_must_be_positive():
    with pytest.raises(ValueError):
        ref.adamw_step(np.ones(2), np.ones(2), np.zeros(2), np.zeros(2), 0, ref.AdamWHParams())
