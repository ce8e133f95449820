"""Full-size parity on the five synthetic workloads, in the launch
configuration the benchmark times (one call over every matrix, default
2^29-element chunk cap).

Workload 1 (one 256x128 fp32 matrix) is compared with the oracle run here.
Workloads 2-5 are compared at seeded sample positions with oracle values that
tests/golden/make_golden.py computed (fp64, whole matrices) from the same
seeded inputs; the relative error over the samples estimates the relative
Frobenius error per matrix.
"""
import os

import numpy as np
import pytest

from oracle import muon_ref as ref
from paper_2609_21594_amd import synth
from tests.golden.make_golden import NSAMP, golden_path, sample_indices
from tests.gpu_util import MOMENTUM_TOL, TOL, decode, o_gate, rel, require_gpu, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def muon():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    yield m
    m.close()


def _gather(t, idx):
    import torch
    flat = t.reshape(-1)
    return to_host(flat[torch.from_numpy(idx).to(flat.device)])


def test_workload1_single_fp32_matrix(muon):
    import torch
    wl = synth.WORKLOADS[1]
    m = synth.make_matrix(wl, 0)
    dW, dg, db = to_dev(m.W, "f32"), to_dev(m.g, "f32"), to_dev(m.buf, "f32")
    muon.step([dW], [dg], [db], lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay,
              ns_steps=wl.ns_steps, nesterov=wl.nesterov, ns_precision="f32")
    torch.cuda.synchronize()
    hp = ref.MuonHParams(lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay, ns_steps=5)
    W0 = m.W.astype(np.float64)
    r = ref.muon_step_matrix(W0, m.g, m.buf, hp)
    scale = ref.rms_scale(256, 128)
    O_gpu = (W0 - to_host(dW)) / (wl.lr * scale)   # wd = 0
    print(f"workload 1: O rel err {rel(O_gpu, r.O):.3e}", flush=True)
    assert rel(O_gpu, r.O) <= TOL["f32"]
    assert rel(to_host(db), r.buf_new) <= MOMENTUM_TOL


def _load_golden(workload):
    path = golden_path(workload)
    if not os.path.exists(path):
        pytest.fail(f"{path} missing: run tests/golden/make_golden.py {workload}")
    return np.load(path, allow_pickle=False)


@pytest.mark.parametrize("workload", [2, 3, 5])
def test_workload_muon_step_sampled(muon, workload):
    import torch
    wl = synth.WORKLOADS[workload]
    gold = _load_golden(workload)
    n = len(wl.matrices)
    ns = NSAMP[workload]
    W, G, B, W0s, idxs = [], [], [], [], []
    for lo in range(0, n, 8):  # bounded host memory
        for m in synth.make_workload(wl, 0, indices=range(lo, min(n, lo + 8))):
            i = len(W)
            idx = sample_indices(workload, i, m.spec.rows * m.spec.cols, ns)
            idxs.append(idx)
            W0s.append(decode(m.W.reshape(-1)[idx], wl.param_dtype))
            W.append(to_dev(m.W, wl.param_dtype))
            G.append(to_dev(m.g, wl.grad_dtype))
            B.append(to_dev(m.buf, "f32"))
    hp = dict(lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay, ns_steps=wl.ns_steps,
              nesterov=wl.nesterov, ns_precision=wl.ns_precision)
    for t in range(wl.steps):
        if t > 0:
            G = [to_dev(synth.make_matrix(wl, i, t, with_state=False).g, wl.grad_dtype)
                 for i in range(n)]
        muon.step(W, G, B, **hp)
        torch.cuda.synchronize()
        print(f"workload {workload}: step {t + 1}/{wl.steps} done", flush=True)
    worst_w = worst_b = 0.0
    for i in range(n):
        dW = _gather(W[i], idxs[i]) - W0s[i]
        err = rel(dW, gold["dW"][i].astype(np.float64))
        berr = rel(_gather(B[i], idxs[i]), gold["buf"][i].astype(np.float64))
        worst_w, worst_b = max(worst_w, err), max(worst_b, berr)
        assert err <= TOL[wl.ns_precision] + gold["rho"][i], (i, err, gold["rho"][i])
        assert berr <= 1e-5, (i, berr)  # float32 storage of the expected samples
    print(f"workload {workload}: worst sampled W err {worst_w:.3e}, momentum {worst_b:.2e}", flush=True)


def test_workload4_orthogonalize_sampled(muon):
    import torch
    wl = synth.WORKLOADS[4]
    gold = _load_golden(4)
    ins = [to_dev(m.g, "bf16") for m in synth.make_workload(wl, 0)]
    outs = [torch.empty_like(t) for t in ins]
    muon.orthogonalize(ins, outs, ns_steps=wl.ns_steps, ns_precision="bf16")
    torch.cuda.synchronize()
    worst = 0.0
    for i, o in enumerate(outs):
        spec = wl.matrices[i]
        idx = sample_indices(4, i, spec.rows * spec.cols, NSAMP[4])
        err, rho = o_gate(_gather(o, idx), gold["O"][i].astype(np.float64), "bf16")
        worst = max(worst, err)
        assert err <= TOL["bf16"] + rho, (i, spec, err, rho)
    print(f"workload 4: worst sampled O err {worst:.3e}", flush=True)
