"""Seeded random cases against the oracle, through the C ABI: shapes from 1
to 1300 on a side (tall, wide, square, and multiples of 128 and 256 so that
every kernel path is taken: the fused small-matrix launch, the 128 x 128
and 256 x 256 tile kernels, grouped launches), random parameter and
gradient dtypes, both Newton-Schulz precisions, 0 to 5 steps, per-entry
coefficient tables, scale modes and post-processing factors, some entries
as column-range views of a wider weight.  Every matrix of a call is compared with the oracle at
the gates of its precision."""
import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.gpu_util import MOMENTUM_TOL, decode, o_gate, rel, require_gpu, to_dev, to_host, tol_for, w_gate

pytestmark = pytest.mark.gpu

QUINTIC = (3.4445, -4.7750, 2.0315)
# per-entry coefficient tables (None: the call's step count with the constant quintic)
TABLES = [None, None, [(1.5, -0.5, 0.0)] * 3, [(15 / 8, -10 / 8, 3 / 8)] * 2 + [QUINTIC] * 2, []]


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def rng(*key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([synth.ROOT_SEED, 7700, *key])))


def side(r):
    pick = r.integers(4)
    if pick == 0:
        return int(r.integers(1, 130))               # fused launch sizes
    if pick == 1:
        return int(256 * r.integers(1, 5))           # 256-multiples: the 256 x 256 kernels
    if pick == 2:
        return int(128 * r.integers(1, 9))          # 128-multiples
    return int(r.integers(130, 1301))                # ragged


@pytest.mark.parametrize("case", range(6))
def test_random_calls_match_oracle(muon, case):
    import torch
    r = rng(case)
    prec = ["bf16", "f32"][case % 2]
    steps = [5, 5, 2, 1, 0, 3][case]
    muon.set_streams(1 if case in (1, 4) else 2)
    muon.set_grouping(case != 2)
    n = 6
    # lr large enough that the change of a bf16 parameter stands above its rounding
    hp = ref.MuonHParams(lr=0.2, beta=0.95, weight_decay=0.05, ns_steps=steps, nesterov=bool(case % 3))
    dev, host = [], []
    for i in range(n):
        rows, cols = side(r), side(r)
        pdt = ["bf16", "f32"][int(r.integers(2))]
        gdt = ["bf16", "f32"][int(r.integers(2))]
        smode = [None, 0, 1, 2][int(r.integers(4))]
        post = [None, None, float(r.uniform(0.5, 1.0))][int(r.integers(3))]
        view = bool(r.integers(3) == 0)
        width = cols + (int(r.integers(1, 65)) if view else 0)   # a column range of a wider weight
        table = TABLES[int(r.integers(len(TABLES)))]
        Wp = synth.draw((rows, width), 0.02, pdt, rng(case, i, 0))
        gp = synth.draw((rows, width), 1e-3, gdt, rng(case, i, 1))
        mp = synth.draw((rows, width), 1e-3, "f32", rng(case, i, 2))
        dW, dg, dm = to_dev(Wp, pdt), to_dev(gp, gdt), to_dev(mp, "f32")
        off = width - cols
        dev.append((dW, dg, dm, dW[:, off:], dg[:, off:], dm[:, off:]))
        host.append((Wp, gp, mp, off, rows, cols, pdt, gdt, smode, post, table))
    muon.step([d[3] for d in dev], [d[4] for d in dev], [d[5] for d in dev],
              lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, ns_steps=steps,
              nesterov=hp.nesterov, ns_precision=prec,
              entry_scale_modes=[h[8] for h in host], entry_post_scales=[h[9] for h in host],
              entry_coeffs=[h[10] for h in host])
    torch.cuda.synchronize()
    for i, ((dW, dg, dm, *_), (Wp, gp, mp, off, rows, cols, pdt, gdt, smode, post, table)) in enumerate(zip(dev, host)):
        W0 = decode(Wp, pdt)
        k_i = steps if table is None else len(table)
        hpi = ref.MuonHParams(lr=hp.lr, beta=hp.beta, weight_decay=hp.weight_decay, ns_steps=k_i,
                              ns_coeffs=table, nesterov=hp.nesterov, scale_mode=0 if smode is None else smode,
                              post_scale=1.0 if post is None else post)
        res = ref.muon_step_matrix(W0[:, off:], decode(gp, gdt)[:, off:], np.asarray(mp[:, off:], np.float64), hpi)
        got = to_host(dW)
        err, rho = w_gate(got[:, off:], res.W_new, W0[:, off:], pdt)
        u = ref.momentum_update(decode(gp, gdt)[:, off:], np.asarray(mp[:, off:], np.float64), hp.beta, hp.nesterov)[1]
        gate = tol_for(prec, (rows, cols), k_i, table, u)
        print(f"case {case} {prec} K={k_i} entry {i}: {rows}x{cols} {pdt}/{gdt} view={off > 0} "
              f"scale={smode} post={post}: W err {err:.2e} (gate {gate:.1e} + {rho:.1e})", flush=True)
        assert err <= gate + rho, (i, rows, cols, err, gate, rho)
        assert rel(to_host(dm)[:, off:], res.buf_new) <= MOMENTUM_TOL, i
        if off:   # the columns outside the view keep their values
            np.testing.assert_array_equal(got[:, :off], W0[:, :off])
            np.testing.assert_array_equal(to_host(dm)[:, :off], mp[:, :off])
    muon.set_streams(2)
    muon.set_grouping(True)


@pytest.mark.parametrize("case", range(4))
def test_random_orthogonalize_matches_oracle(muon, case):
    import torch
    r = rng(100, case)
    prec = ["bf16", "f32"][case % 2]
    steps = [5, 5, 1, 3][case]
    dt = ["bf16", "f32"][case // 2]
    shapes = [(side(r), side(r)) for _ in range(5)]
    G = [synth.draw(s, 1e-3, dt, rng(100, case, i)) for i, s in enumerate(shapes)]
    ins = [to_dev(a, dt) for a in G]
    outs = [torch.empty_like(a) for a in ins]
    muon.orthogonalize(ins, outs, ns_steps=steps, ns_precision=prec)
    torch.cuda.synchronize()
    for i, s in enumerate(shapes):
        Gd = decode(G[i], dt)
        O = ref.orthogonalize(Gd, steps)
        err, gate = o_gate(to_host(outs[i]), O, dt, prec, steps, None, Gd)
        print(f"orthogonalize case {case} {prec} K={steps} {dt} {s}: err {err:.2e} (gate {gate:.1e})", flush=True)
        assert err <= gate, (i, s, err, gate)
