"""Writes sampled oracle results for the full-size workloads.

    python tests/golden/make_golden.py [2 3 4 5] [--threads N]

For every matrix of a workload the fp64 oracle (oracle/muon_ref.py) runs the
whole Muon step (or, for workload 4, the standalone orthogonalisation) on the
seeded inputs of paper_2609_21594_amd/synth.py, one matrix at a time, and the
values at seeded positions are stored in tests/golden/workload<k>_samples.npz.
The positions are stratified over the 256 x 256 tiles of the matrix (edge
tiles clipped): every tile holds at least TILE_SAMPLES of them, and at least
MIN_SAMPLES fall in every matrix, so an error confined to any one output tile
of the kernels is sampled.

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

TILE = 256
TILE_SAMPLES = 2
MIN_SAMPLES = 256
SAMPLE_STREAM = 778


def sample_indices(workload: int, index: int, rows: int, cols: int) -> np.ndarray:
    """Seeded flat positions inside one rows x cols matrix (row-major), the
    same number in each 256 x 256 tile (at least TILE_SAMPLES, and enough for
    MIN_SAMPLES in all), uniform inside the tile; sorted."""
    rng = np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([synth.ROOT_SEED, workload, SAMPLE_STREAM, index])))
    tr, tc = -(-rows // TILE), -(-cols // TILE)
    per = max(TILE_SAMPLES, -(-MIN_SAMPLES // (tr * tc)))
    r0 = np.repeat(np.arange(tr) * TILE, tc * per)
    c0 = np.tile(np.repeat(np.arange(tc) * TILE, per), tr)
    hr = np.minimum(TILE, rows - r0)
    hc = np.minimum(TILE, cols - c0)
    r = r0 + (rng.random(r0.size) * hr).astype(np.int64)
    c = c0 + (rng.random(c0.size) * hc).astype(np.int64)
    return np.sort(r * cols + c)


def decode(x, dtype):
    return ref.decode_bf16(x) if dtype == "bf16" else np.asarray(x, dtype=np.float64)


def golden_path(workload: int) -> str:
    return os.path.join(HERE, f"workload{workload}_samples.npz")


def run_matrix(wl: synth.Workload, i: int):
    spec = wl.matrices[i]
    idx = sample_indices(wl.index, i, spec.rows, spec.cols)
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


def make(workload: int, cache_dir=None):
    wl = synth.WORKLOADS[workload]
    n = len(wl.matrices)
    cols = {k: [] for k in ("O", "dW", "buf", "rho")}
    counts = []
    t0 = time.time()
    for i in range(n):
        # optional per-matrix cache, so an interrupted run resumes where it stopped
        cpath = (os.path.join(cache_dir, f"w{workload}_s{SAMPLE_STREAM}_m{i}.npz")
                 if cache_dir else None)
        if cpath and os.path.exists(cpath):
            with np.load(cpath, allow_pickle=False) as z:
                res = {k: z[k] for k in ("O", "dW", "buf")}
                res["rho"] = float(z["rho"])
        else:
            res = run_matrix(wl, i)
            if cpath:
                np.savez(cpath, **res)
        for k in cols:
            cols[k].append(res[k])
        counts.append(len(res["O"]))
        print(f"workload {workload}: matrix {i + 1}/{n} {wl.matrices[i].rows}x{wl.matrices[i].cols} "
              f"done at {time.time() - t0:.0f}s", flush=True)
    # matrices hold different sample counts: stored concatenated, with offsets
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    np.savez_compressed(golden_path(workload), O=np.concatenate(cols["O"]),
                        dW=np.concatenate(cols["dW"]), buf=np.concatenate(cols["buf"]),
                        rho=np.array(cols["rho"]), offsets=offsets, workload=workload,
                        sample_stream=SAMPLE_STREAM)
    print(f"wrote {golden_path(workload)} in {time.time() - t0:.0f}s", flush=True)


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("workloads", nargs="*", type=int, default=[2, 4, 3, 5])
    ap.add_argument("--cache", default=None, help="directory for per-matrix results (resumable runs)")
    args = ap.parse_args()
    if args.cache:
        os.makedirs(args.cache, exist_ok=True)
    for w in args.workloads:
        make(w, args.cache)
