"""Writes sampled oracle results for the full-size workloads.

    python tests/golden/make_golden.py [2 3 4 5] [--threads N]

For every matrix of a workload the fp64 oracle (oracle/muon_ref.py) runs the
whole Muon step (or, for workload 4, the standalone orthogonalisation) on the
seeded inputs of paper_2609_21594_amd/synth.py, one matrix at a time, and the
values at NSAMP seeded positions are stored in tests/golden/workload<k>_samples.npz:

  dW     W_final - W_initial at the sampled positions (float32)   [Muon steps]
  buf    final momentum at the sampled positions (float32)        [Muon steps]
  O      orthogonalised update of the last step (float32)
  rho    storage-rounding floor per matrix: sum over steps of the norm of
         (bf16 rounding of W_t - W_t) at the samples, over the norm of dW
  scale  RMS of O over the samples (sanity)

The oracle keeps its state in fp64 across steps (no intermediate rounding);
rho bounds the rounding a bf16-stored trajectory adds.  Only oracle/ and the
input generator are imported.
"""
from __future__ import annotations

import argparse
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import muon_ref as ref  # noqa: E402
from paper_2609_21594_amd import synth  # noqa: E402

NSAMP = {2: 1024, 3: 512, 4: 256, 5: 512}
SAMPLE_STREAM = 777


def sample_indices(workload: int, index: int, numel: int, n: int) -> np.ndarray:
    """Seeded flat positions (with replacement, sorted) inside one matrix."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([synth.ROOT_SEED, workload, SAMPLE_STREAM, index])))
    return np.sort(rng.integers(0, numel, size=n))


def decode(x, dtype):
    return ref.decode_bf16(x) if dtype == "bf16" else np.asarray(x, dtype=np.float64)


def golden_path(workload: int) -> str:
    return os.path.join(HERE, f"workload{workload}_samples.npz")


def run_matrix(wl: synth.Workload, i: int):
    spec = wl.matrices[i]
    ns = NSAMP[wl.index]
    idx = sample_indices(wl.index, i, spec.rows * spec.cols, ns)
    hp = ref.MuonHParams(lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay,
                         ns_steps=wl.ns_steps, nesterov=wl.nesterov)
    if wl.orthogonalize_only:
        G = decode(synth.make_matrix(wl, i, 0).g, wl.grad_dtype)
        O = ref.orthogonalize(G, wl.ns_steps)
        o = O.ravel()[idx]
        return dict(O=o.astype(np.float32), dW=np.zeros(0, np.float32),
                    buf=np.zeros(0, np.float32), rho=0.0)
    inp = synth.make_matrix(wl, i, 0)
    W = decode(inp.W, wl.param_dtype)
    buf = np.asarray(inp.buf, dtype=np.float64)
    W0 = W.ravel()[idx].copy()
    resid = 0.0
    for t in range(wl.steps):
        g = decode(inp.g if t == 0 else synth.make_matrix(wl, i, t, with_state=False).g,
                   wl.grad_dtype)
        r = ref.muon_step_matrix(W, g, buf, hp)
        W, buf, O = r.W_new, r.buf_new, r.O
        ws = W.ravel()[idx]
        resid += float(np.linalg.norm(ref.round_to(ws, wl.param_dtype) - ws))
    dW = W.ravel()[idx] - W0
    return dict(O=O.ravel()[idx].astype(np.float32), dW=dW.astype(np.float32),
                buf=buf.ravel()[idx].astype(np.float32),
                rho=resid / max(float(np.linalg.norm(dW)), 1e-300))


def make(workload: int):
    wl = synth.WORKLOADS[workload]
    n = len(wl.matrices)
    cols = {k: [] for k in ("O", "dW", "buf", "rho")}
    t0 = time.time()
    for i in range(n):
        res = run_matrix(wl, i)
        for k in cols:
            cols[k].append(res[k])
        print(f"workload {workload}: matrix {i + 1}/{n} {wl.matrices[i].rows}x{wl.matrices[i].cols} "
              f"done at {time.time() - t0:.0f}s", flush=True)
    np.savez_compressed(golden_path(workload), O=np.stack(cols["O"]), dW=np.stack(cols["dW"]),
                        buf=np.stack(cols["buf"]), rho=np.array(cols["rho"]),
                        nsamp=NSAMP[workload], workload=workload)
    print(f"wrote {golden_path(workload)} in {time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("workloads", nargs="*", type=int, default=[2, 4, 3, 5])
    args = ap.parse_args()
    for w in args.workloads:
        make(w)
