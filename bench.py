"""Benchmark of the batched Muon step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload 3] [--no-cpu-baseline]

One step = one muon_step call over every matrix of the workload: momentum
update, Frobenius normalisation, transpose-first cast, 5 Newton-Schulz steps
(Gram, polynomial, update products) and the parameter update, all in the HIP
library.  Inputs are the seeded synthetic workload, resident in HBM before
the timed region.  Prints one JSON line.

Default workload: a 7B-like per-device share, 8 layers of hidden 4096 and
FFN 11008 (56 matrices: 32 x 4096x4096, 16 x 11008x4096, 8 x 4096x11008),
bf16 parameters and gradients, fp32 momentum, bf16 Newton-Schulz products.

roofline: the dominant kernel by time, its algorithmic flops (dense count of
the product it computes) per launch over its mean launch duration, both from
HIP events the library records around each launch on its own stream.  The
timed region runs the library as deployed: chunks that leave compute units
idle run on the handle's second stream beside the others, so a kernel's
events there would include time the other stream holds the GPU.  The kernel
figures therefore come from a second pass of the same steps with that
concurrency off (--streams 1 times and profiles one serial region).
cpu_baseline: the fp64 CPU oracle on a bounded sample of the same workload
(one matrix of each shape bucket), extrapolated to the workload's mix.

Side measurements on workload 3 (not part of `value`):
views: the same step with every layer's q, k and v taken as zero-copy,
  head-interleaved views of one fused QKV weight (and its gradient and
  momentum), as a model adapter would hand them over;
adamw: the chained AdamW over the parameters a 7B-like model leaves to it
  (embedding and output head 2 x 32000 x 4096, 65 norm weights of 4096);
hbm_reference: the library's streaming copy over 4 GiB, the achievable HBM
  rate the bandwidth-bound kernels are compared with.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Muon-step matrices/s and NS TFLOP/s (% bf16 MFMA peak), 1×MI355X"
PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA: 256 CU x 4 SIMD x 1024 flop/clk x 2.4 GHz
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_21594_amd", "csrc", "muon_kernels.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_update_gemm_workload3.json")


def kernel_source_sha() -> str:
    with open(KERNEL_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--streams", type=int, default=2, choices=(1, 2),
                    help="library chunk concurrency in the timed region (muon_set_streams)")
    ap.add_argument("--grouping", type=int, default=1, choices=(0, 1),
                    help="grouped launches for chunks that leave CUs idle (muon_set_grouping)")
    ap.add_argument("--no-side", action="store_true",
                    help="skip the views and AdamW side measurements (counter runs)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this size (HBM counter calibration)")
    ap.add_argument("--reference-gemm", action="store_true",
                    help="instead of the step, time torch.matmul (the vendor bf16 GEMM) on the "
                         "workload's update shapes and a plain device copy, as context for the roofline")
    return ap.parse_args()


def upload(inputs, wl):
    import numpy as np
    import torch

    def dev(a, dt):
        if dt == "bf16":
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()

    W = [dev(m.W, wl.param_dtype) for m in inputs]
    G = [dev(m.g, wl.grad_dtype) for m in inputs]
    B = [dev(m.buf, "f32") for m in inputs]
    return W, G, B


def cpu_baseline(wl, inputs):
    """Times the oracle on one matrix per (short, long) shape bucket and
    extrapolates to the workload's mix of shapes."""
    import contextlib

    import numpy as np
    from oracle import muon_ref as ref
    from paper_2609_21594_amd import synth as synth_mod
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:  # pragma: no cover
        threadpool_limits = None
    # every core in the process affinity, unless the environment sets a
    # smaller BLAS/OpenMP thread count (a GPU host's per-GPU CPU share)
    affinity = len(os.sched_getaffinity(0))
    env_threads = [int(v) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS")
                   if (v := os.environ.get(k, "")).isdigit() and int(v) > 0]
    cores = min([affinity] + env_threads)
    buckets = {}
    for i, m in enumerate(wl.matrices):
        key = (min(m.rows, m.cols), max(m.rows, m.cols))
        buckets.setdefault(key, []).append(i)
    hp = ref.MuonHParams(lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay,
                         ns_steps=wl.ns_steps, nesterov=wl.nesterov)
    dec = (lambda a, dt: ref.decode_bf16(a) if dt == "bf16" else np.asarray(a, np.float64))
    total, sampled = 0.0, []
    limit = threadpool_limits(limits=cores) if threadpool_limits else contextlib.nullcontext()
    with limit:
        for key, idx in buckets.items():
            i = idx[0]
            m = inputs[i]
            t0 = time.perf_counter()
            if wl.orthogonalize_only:
                ref.orthogonalize(dec(m.g, wl.grad_dtype), wl.ns_steps)
            else:
                ref.muon_step_matrix(dec(m.W, wl.param_dtype), dec(m.g, wl.grad_dtype),
                                     np.asarray(m.buf, np.float64), hp)
            dt = time.perf_counter() - t0
            total += dt * len(idx)
            sampled.append(f"{wl.matrices[i].name} {wl.matrices[i].rows}x{wl.matrices[i].cols}: {dt:.2f}s")
    # workload 1 (one 256 x 128 fp32 matrix) on a single thread, median of 20
    wl1 = synth_mod.WORKLOADS[1]
    m1 = synth_mod.make_matrix(wl1, 0)
    hp1 = ref.MuonHParams(lr=wl1.lr, beta=wl1.beta, weight_decay=wl1.weight_decay,
                          ns_steps=wl1.ns_steps, nesterov=wl1.nesterov)
    one = threadpool_limits(limits=1) if threadpool_limits else contextlib.nullcontext()
    t1 = []
    with one:
        for _ in range(20):
            t0 = time.perf_counter()
            ref.muon_step_matrix(np.asarray(m1.W, np.float64), np.asarray(m1.g, np.float64),
                                 np.asarray(m1.buf, np.float64), hp1)
            t1.append(time.perf_counter() - t0)
    single_ms = float(np.median(t1)) * 1e3
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": len(wl.matrices) / total, "unit": "matrices/s", "cores": cores,
            "kind": "oracle", "affinity_cores": affinity, "cpu_model": cpu,
            "workload1_single_thread_ms": single_ms,
            "sample": (f"fp64 NumPy oracle, one full {'orthogonalisation' if wl.orthogonalize_only else 'Muon step'} on one matrix per shape bucket "
                       f"({'; '.join(sampled)}), extrapolated by bucket counts to all "
                       f"{len(wl.matrices)} matrices; {cores} BLAS threads ({affinity} cores in the "
                       f"process affinity{', capped by the thread count the environment sets' if cores < affinity else ''}) "
                       f"on {cpu}; workload 1 (256x128 fp32, one step) on one thread: {single_ms:.2f} ms")}


def views_step(muon, W, G, B, wl, hp, steps, warmup):
    """ms per step of workload 3 with q, k, v as head-interleaved views of a
    fused [3*4096, 4096] QKV weight per layer (32 heads of 128 rows, ordered
    q_h, k_h, v_h per head), its gradient and momentum."""
    import torch
    from paper_2609_21594_amd.binding import RowBlocks
    H, hd = 32, 128
    names = [m.name for m in wl.matrices]
    Wv, Gv, Bv, keep = [], [], [], []
    for layer in sorted({n.split(".")[0] for n in names}, key=lambda x: int(x[1:])):
        idx = [names.index(f"{layer}.{p}") for p in ("q", "k", "v")]
        fused = []
        for T in (W, G, B):
            F = torch.empty((H, 3, hd, T[idx[0]].shape[1]), dtype=T[idx[0]].dtype, device="cuda")
            for j, i in enumerate(idx):
                F[:, j] = T[i].view(H, hd, -1)
            fused.append(F)
        keep.append(fused)
        for j in range(3):
            for lst, F in zip((Wv, Gv, Bv), fused):
                lst.append(RowBlocks(F[:, j]))
        for p in ("o", "gate", "up", "down"):
            i = names.index(f"{layer}.{p}")
            Wv.append(W[i]); Gv.append(G[i]); Bv.append(B[i])
    for _ in range(warmup):
        muon.step(Wv, Gv, Bv, **hp)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        muon.step(Wv, Gv, Bv, **hp)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def adamw_bench(muon, steps, warmup):
    """The chained AdamW over a 7B-like model's AdamW parameters:
    embedding and output head (2 x 32000 x 4096) and 65 norm weights of
    4096; bf16 parameters and gradients, fp32 moments; seeded normal
    values.  Rate = algorithmic bytes (22 per element) over kernel time."""
    import torch
    sizes = [32000 * 4096] * 2 + [4096] * 65
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2609)
    P = [(0.02 * torch.randn(n, generator=gen, device="cuda")).to(torch.bfloat16) for n in sizes]
    Gr = [(1e-3 * torch.randn(n, generator=gen, device="cuda")).to(torch.bfloat16) for n in sizes]
    M = [torch.zeros(n, device="cuda") for n in sizes]
    V = [torch.zeros(n, device="cuda") for n in sizes]
    kw = dict(lr=3e-4, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.1)
    for t in range(1, warmup + 1):
        muon.adamw_step(P, Gr, M, V, t, **kw)
    torch.cuda.synchronize()
    muon.profile(True)
    muon.profile_read(reset=True)
    t0 = time.perf_counter()
    for t in range(warmup + 1, warmup + steps + 1):
        muon.adamw_step(P, Gr, M, V, t, **kw)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / steps
    st = muon.profile_read(reset=True)["adamw"]
    muon.profile(False)
    n = sum(sizes)
    gbs = st["bytes"] / (st["total_ms"] * 1e-3) / 1e9
    return {"workload": "7B-like AdamW set: 2 x 32000x4096 + 65 x 4096, bf16 params/grads, fp32 moments",
            "elements": n, "ms_per_step": wall_ms, "kernel_ms": st["total_ms"] / steps,
            "bytes_per_elem": 22, "gbs": gbs, "frac_hbm": gbs / PEAK_HBM_GBS}


def hbm_reference(muon, steps=10, mib=4096):
    """Rate of the library's reference streaming copy (muon_stream_copy) over
    `mib` MiB: the achievable HBM ceiling for the bandwidth-bound kernels."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        muon.stream_copy(dst, src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        muon.stream_copy(dst, src)   # on the current stream, which the events see
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    bytes_ = 2.0 * n * 4
    del src, dst
    torch.cuda.empty_cache()
    return {"kernel": "k_stream_copy (muon_stream_copy)", "bytes": bytes_, "ms": ms,
            "gbs": bytes_ / (ms * 1e-3) / 1e9, "frac_hbm": bytes_ / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS}


def reference_gemm(wl):
    """Vendor-library context on the same GPU: torch.matmul (hipBLASLt) for
    the update product B(s x s) @ X(s x l) of each shape bucket, batched over
    the bucket's matrices, and the rate of a plain 4 GiB device copy."""
    import torch
    shapes = sorted({(min(m.rows, m.cols), max(m.rows, m.cols)) for m in wl.matrices})
    out = {"kind": "vendor reference", "gemm": [], "copy": None}
    ev = lambda: torch.cuda.Event(enable_timing=True)
    for s_, l_ in shapes:
        n = sum(1 for m in wl.matrices if (min(m.rows, m.cols), max(m.rows, m.cols)) == (s_, l_))
        a = torch.randn(n, s_, s_, device="cuda", dtype=torch.bfloat16)
        b = torch.randn(n, s_, l_, device="cuda", dtype=torch.bfloat16)
        for _ in range(3):
            torch.bmm(a, b)
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record()
        for _ in range(10):
            torch.bmm(a, b)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 10
        tf = n * 2.0 * s_ * s_ * l_ / (ms * 1e-3) / 1e12
        out["gemm"].append({"batch": n, "m": s_, "k": s_, "n": l_, "ms": ms, "tflops": tf,
                            "pct_peak": 100 * tf / PEAK_BF16_TFLOPS})
        del a, b
    x = torch.ones(1 << 30, device="cuda")
    y = torch.empty_like(x)
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record()
    for _ in range(10):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 10
    out["copy"] = {"bytes": 2 * 4 * (1 << 30), "ms": ms, "tb_per_s": 2 * 4 * (1 << 30) / (ms * 1e-3) / 1e12}
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "this build has no multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2609_21594_amd import synth
    from paper_2609_21594_amd.binding import Muon

    wl = synth.WORKLOADS[args.workload]
    if args.reference_gemm:
        print(json.dumps(reference_gemm(wl)), flush=True)
        return
    t_gen = time.perf_counter()
    inputs = synth.make_workload(wl)
    if wl.orthogonalize_only:
        # the standalone batched NS: one ns_orthogonalize_batched call over
        # every matrix is the step
        G = [torch.from_numpy(np.ascontiguousarray(m.g).view(np.int16)).view(torch.bfloat16).cuda()
             if wl.grad_dtype == "bf16" else torch.from_numpy(np.ascontiguousarray(m.g, dtype=np.float32)).cuda()
             for m in inputs]
        outs = [torch.empty_like(t) for t in G]
        W = B = None
    else:
        W, G, B = upload(inputs, wl)
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t_gen

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    muon = Muon(0)
    muon.set_streams(args.streams)
    muon.set_grouping(bool(args.grouping))
    if wl.orthogonalize_only:
        ohp = dict(ns_steps=wl.ns_steps, ns_precision=wl.ns_precision)
        run_step = lambda: muon.orthogonalize(G, outs, **ohp)
    else:
        hp = dict(lr=wl.lr, beta=wl.beta, weight_decay=wl.weight_decay, ns_steps=wl.ns_steps,
                  nesterov=wl.nesterov, ns_precision=wl.ns_precision)
        run_step = lambda: muon.step(W, G, B, **hp)
    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()

    host_ms = []

    def timed(profile):
        if profile:
            muon.profile(True)
            muon.profile_read(reset=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        host = 0.0
        for _ in range(args.steps):
            h0 = time.perf_counter()
            run_step()
            host += time.perf_counter() - h0
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        host_ms.append(host * 1e3 / args.steps)
        st = None
        if profile:
            st = muon.profile_read(reset=True)
            muon.profile(False)
        return el, st

    # the timed region: the library as deployed
    elapsed, stats = timed(profile=args.streams == 1)
    serial_ms = None
    if stats is None:
        # kernel figures from the same steps with chunk concurrency off
        muon.set_streams(1)
        run_step()
        el1, stats = timed(profile=True)
        serial_ms = el1 * 1e3 / args.steps
        muon.set_streams(args.streams)

    ms = elapsed * 1e3 / args.steps
    n_mat = wl.n_matrices
    ns_flops = synth.workload_ns_flops(wl)
    peak = PEAK_BF16_TFLOPS if wl.ns_precision == "bf16" else PEAK_F32_TFLOPS

    kernels = {}
    for name, st in stats.items():
        if not st["launches"]:
            continue
        d = {"launches_per_step": st["launches"] / args.steps,
             "ms_per_step": st["total_ms"] / args.steps,
             "mean_launch_us": st["total_ms"] * 1e3 / st["launches"]}
        if st["flops"]:
            d["tflops"] = st["flops"] / (st["total_ms"] * 1e-3) / 1e12
            d["exec_tflops"] = st["exec_flops"] / (st["total_ms"] * 1e-3) / 1e12
        else:
            d["gbs"] = st["bytes"] / (st["total_ms"] * 1e-3) / 1e9
        kernels[name] = d
    dom = max(stats, key=lambda k: stats[k]["total_ms"])
    ds = stats[dom]
    if ds["flops"]:
        achieved = ds["flops"] / ds["launches"] / (ds["total_ms"] / ds["launches"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                "frac": achieved / peak}
    else:
        achieved = ds["bytes"] / (ds["total_ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": achieved / PEAK_HBM_GBS}
    roof["kernel"] = dom
    roof["measured_in"] = ("the timed region" if args.streams == 1 else
                           "a profiled pass of the same steps with chunk concurrency off")
    roof["mean_launch_us"] = ds["total_ms"] * 1e3 / ds["launches"]
    roof["algorithmic_per_launch"] = (ds["flops"] or ds["bytes"]) / ds["launches"]
    roof["traffic"] = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("kernel_source_sha") == kernel_source_sha() and tr.get("kernel") == dom:
            roof["traffic"] = tr.get("hbm_bytes_per_launch")

    # The Newton-Schulz contractions alone: dense flops (Eq. 1 count) and the
    # MFMA work the kernels execute (upper tiles of the symmetric products,
    # padded extents), over the summed kernel time.
    gemm_names = [k for k in ("gram_syrk", "poly_syrk", "update_gemm", "update_apply_gemm", "ns_small")
                  if k in stats and stats[k]["launches"]]
    g_ms = max(1e-12, sum(stats[k]["total_ms"] for k in gemm_names) / args.steps)
    g_exec = sum(stats[k]["exec_flops"] for k in gemm_names) / args.steps
    ns_gemm = {"ms_per_step": g_ms,
               "dense_tflops": ns_flops / (g_ms * 1e-3) / 1e12,
               "dense_pct_peak": 100.0 * ns_flops / (g_ms * 1e-3) / 1e12 / peak,
               "executed_tflops": g_exec / (g_ms * 1e-3) / 1e12,
               "executed_pct_peak": 100.0 * g_exec / (g_ms * 1e-3) / 1e12 / peak}
    out = {
        "metric": METRIC, "value": n_mat / (ms * 1e-3), "unit": "matrices/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.ns_precision, "data": "synthetic",
        "config": {"workload": wl.name, "matrices": n_mat,
                   "shapes": "32x4096x4096, 16x11008x4096, 8x4096x11008" if wl.index == 3 else
                   ", ".join(f"{m.rows}x{m.cols}" for m in wl.matrices[:8]),
                   "ns_steps": wl.ns_steps, "ns_precision": wl.ns_precision,
                   "param_dtype": wl.param_dtype, "grad_dtype": wl.grad_dtype,
                   "momentum_dtype": "f32", "parallelism": "none (one GPU)"},
        "ns_tflops": ns_flops / (ms * 1e-3) / 1e12,
        "ns_pct_peak": 100.0 * ns_flops / (ms * 1e-3) / 1e12 / peak,
        "ns_gemm": ns_gemm,
        "streams": args.streams,
        "grouping": args.grouping,
        "serial_ms_per_step": serial_ms if serial_ms is not None else ms,
        "roofline": roof,
        "kernels": kernels,
        "input_generation_s": gen_s,
        "host_ms_per_call": host_ms[0],
    }
    if wl.index == 3 and not args.no_side:
        vms = views_step(muon, W, G, B, wl, hp, args.steps, args.warmup)
        out["views"] = {"workload": "same, q/k/v as head-interleaved views of fused QKV weights",
                        "ms_per_step": vms, "vs_dense": vms / ms}
        del W, G, B
        torch.cuda.empty_cache()
        out["adamw"] = adamw_bench(muon, args.steps, args.warmup)
        ref = hbm_reference(muon)
        ref["momentum_norm_vs_copy"] = kernels["momentum_norm"]["gbs"] / ref["gbs"]
        ref["adamw_vs_copy"] = out["adamw"]["gbs"] / ref["gbs"]
        out["hbm_reference"] = ref
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, inputs)
    muon.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
