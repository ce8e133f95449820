"""Logical matrices as zero-copy views of a physical parameter (Sec. 6.6:
the matrix Muon sees is defined apart from the storage layout), through the
C ABI.

Each case steps strided views of one physical weight (its gradient and
momentum), and the same logical matrices as dense copies in a second call.
The two must agree bit for bit, since they run the same kernels on the same
values.  One matrix is also checked against the oracle.  Every element
outside the views must keep its bits.
"""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import MOMENTUM_TOL, decode, rel, require_gpu, to_bits, to_dev, to_host, tol_for, w_gate

pytestmark = pytest.mark.gpu

HP = dict(lr=0.02, beta=0.95, weight_decay=0.01, nesterov=True)


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([5151, *key])))


def physical(shape, pdt, key):
    """Seeded param, grad (param dtype) and fp32 momentum of one weight."""
    W = synth.draw(shape, 0.02, pdt, rng(key, 0))
    g = synth.draw(shape, 1e-3, pdt, rng(key, 1))
    m = synth.draw(shape, 1e-3, "f32", rng(key, 2))
    return W, g, m


def oracle_check(W_dev, W0, g, m0, m_dev, pdt):
    hp = ref.MuonHParams(**HP)
    r = ref.muon_step_matrix(decode(W0, pdt), decode(g, pdt), np.asarray(m0, np.float64), hp)
    err, rho = w_gate(to_host(W_dev), r.W_new, decode(W0, pdt), pdt)
    assert err <= tol_for("bf16", W0.shape) + rho, (err, rho)
    assert rel(to_host(m_dev), r.buf_new) <= MOMENTUM_TOL


# (8, 128, 512): q and k are 1024 x 512, tall, so they are transposed first
# and their last step writes W blocks back transposed through the row blocks
@pytest.mark.parametrize("H,hd,d", [(4, 64, 256), (3, 40, 200), (8, 128, 512)])
def test_interleaved_heads_of_fused_qkv(muon, H, hd, d):
    # [3*H*hd, d] with rows grouped per head as (q_h, k_h, v_h); q and k are
    # [H*hd, d] logical matrices of H row blocks each; v is left alone
    import torch
    from paper_2609_21594_amd.binding import RowBlocks
    Wn, gn, mn = physical((3 * H * hd, d), "bf16", (1, H, hd, d))
    Wp, Gp, Mp = to_dev(Wn, "bf16"), to_dev(gn, "bf16"), to_dev(mn, "f32")
    W0, G0, M0 = Wp.clone(), Gp.clone(), Mp.clone()
    heads = lambda T, j: T.view(H, 3, hd, d)[:, j]
    dense = lambda T, j: heads(T, j).reshape(H * hd, d).clone()
    Wd, Gd, Md = ([dense(T, j) for j in (0, 1)] for T in (Wp, Gp, Mp))
    muon.step([RowBlocks(heads(Wp, j)) for j in (0, 1)], [RowBlocks(heads(Gp, j)) for j in (0, 1)],
              [RowBlocks(heads(Mp, j)) for j in (0, 1)], ns_precision="bf16", **HP)
    muon.step(Wd, Gd, Md, ns_precision="bf16", **HP)
    torch.cuda.synchronize()
    for j in (0, 1):
        assert np.array_equal(to_bits(dense(Wp, j)), to_bits(Wd[j])), j
        assert np.array_equal(to_bits(dense(Mp, j)), to_bits(Md[j])), j
    assert np.array_equal(to_bits(heads(Wp, 2).contiguous()), to_bits(heads(W0, 2).contiguous()))
    assert np.array_equal(to_bits(heads(Mp, 2).contiguous()), to_bits(heads(M0, 2).contiguous()))
    assert np.array_equal(to_bits(Gp), to_bits(G0))
    sel = lambda a: a.reshape(H, 3, hd, d)[:, 0].reshape(H * hd, d)
    oracle_check(Wd[0], sel(Wn), sel(gn), sel(mn), Md[0], "bf16")


@pytest.mark.parametrize("pdt", ["bf16", "f32"])
# (2, 1024, 256): tall 1024 x 256 halves, transposed first, on the 256 x 256
# kernel with a column-range view
@pytest.mark.parametrize("E,d,f", [(2, 512, 256), (2, 256, 384), (2, 1024, 256)])
def test_gate_up_halves_of_packed_expert_weights(muon, pdt, E, d, f):
    # [E, d, 2f] packed gate|up: two stacked [E, d, f] views (ld = 2f, plane
    # stride d*2f).  The gate's momentum shares the view; the up half keeps
    # its momentum as a dense [E, d, f] tensor.
    import torch
    Wn, gn, mn = physical((E, d, 2 * f), pdt, (2, E, d, f))
    Wp, Gp, Mp = to_dev(Wn, pdt), to_dev(gn, pdt), to_dev(mn, "f32")
    M0 = Mp.clone()
    M_up = Mp[:, :, f:].contiguous()
    half = lambda T, j: T[:, :, j * f:(j + 1) * f]
    Wd, Gd = ([half(T, j).contiguous() for j in (0, 1)] for T in (Wp, Gp))
    Md = [half(Mp, 0).contiguous(), M_up.clone()]
    muon.step([half(Wp, 0), half(Wp, 1)], [half(Gp, 0), half(Gp, 1)], [half(Mp, 0), M_up],
              ns_precision="bf16", **HP)
    muon.step(Wd, Gd, Md, ns_precision="bf16", **HP)
    torch.cuda.synchronize()
    for j in (0, 1):
        assert np.array_equal(to_bits(half(Wp, j).contiguous()), to_bits(Wd[j])), j
    assert np.array_equal(to_bits(half(Mp, 0).contiguous()), to_bits(Md[0]))
    assert np.array_equal(to_bits(M_up), to_bits(Md[1]))
    assert np.array_equal(to_bits(half(Mp, 1).contiguous()), to_bits(half(M0, 1).contiguous()))
    e = E - 1
    oracle_check(Wd[0][e], Wn[e, :, :f], gn[e, :, :f], mn[e, :, :f], Md[0][e], pdt)


@pytest.mark.parametrize("prec,steps", [("f32", 5), ("bf16", 0), ("f32", 0)])
def test_views_on_the_other_paths(muon, prec, steps):
    # fp32 Newton-Schulz (the 128 x 128 kernel's last-step epilogue writes
    # through the view) and K = 0 (the update from X0 alone), on interleaved
    # row blocks and a column range, against dense copies bit for bit
    import torch
    from paper_2609_21594_amd.binding import RowBlocks
    H, hd, d = 3, 64, 192
    Wn, gn, mn = physical((3 * H * hd, d), "bf16", (4, steps))
    Wp, Gp, Mp = to_dev(Wn, "bf16"), to_dev(gn, "bf16"), to_dev(mn, "f32")
    W0 = Wp.clone()
    blocks = lambda T: RowBlocks(T.view(H, 3, hd, d)[:, 1])
    dense_b = lambda T: T.view(H, 3, hd, d)[:, 1].reshape(H * hd, d).clone()
    cols = lambda T: T[2 * hd:3 * hd, 8:8 + 96]  # head 0's v rows, a column range
    Wd = [dense_b(Wp), cols(Wp).contiguous()]
    Gd = [dense_b(Gp), cols(Gp).contiguous()]
    Md = [dense_b(Mp), cols(Mp).contiguous()]
    kw = dict(ns_precision=prec, ns_steps=steps, **HP)
    muon.step([blocks(Wp), cols(Wp)], [blocks(Gp), cols(Gp)], [blocks(Mp), cols(Mp)], **kw)
    muon.step(Wd, Gd, Md, **kw)
    torch.cuda.synchronize()
    assert np.array_equal(to_bits(dense_b(Wp)), to_bits(Wd[0]))
    assert np.array_equal(to_bits(cols(Wp).contiguous()), to_bits(Wd[1]))
    assert np.array_equal(to_bits(dense_b(Mp)), to_bits(Md[0]))
    assert np.array_equal(to_bits(cols(Mp).contiguous()), to_bits(Md[1]))
    # untouched: the q heads
    q = W0.view(H, 3, hd, d)[:, 0].contiguous()
    assert np.array_equal(to_bits(Wp.view(H, 3, hd, d)[:, 0].contiguous()), to_bits(q))


def test_unaligned_column_range(muon):
    # a column range starting 3 elements into each row: no 16-byte vector
    # access applies; compared with the oracle, and the columns around it
    # keep their bits
    import torch
    rows, cols, c0, n = 200, 136, 3, 120
    Wn, gn, mn = physical((rows, cols), "bf16", (3,))
    Wp, Gp, Mp = to_dev(Wn, "bf16"), to_dev(gn, "bf16"), to_dev(mn, "f32")
    W0, M0 = Wp.clone(), Mp.clone()
    sl = slice(c0, c0 + n)
    muon.step([Wp[:, sl]], [Gp[:, sl]], [Mp[:, sl]], ns_precision="bf16", **HP)
    torch.cuda.synchronize()
    oracle_check(Wp[:, sl].contiguous(), Wn[:, sl], gn[:, sl], mn[:, sl], Mp[:, sl].contiguous(), "bf16")
    for T, T0 in ((Wp, W0), (Mp, M0)):
        for outside in (slice(0, c0), slice(c0 + n, cols)):
            assert np.array_equal(to_bits(T[:, outside].contiguous()), to_bits(T0[:, outside].contiguous()))
