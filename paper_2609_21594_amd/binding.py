"""ctypes binding of libmuon_hip.so (argument marshalling only).

Every step of the Muon path runs in the library's HIP kernels; this module
only turns torch tensors into device pointers and sizes, passes the current
HIP stream, and raises on a non-OK status.  It fails loudly when the library
is missing: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmuon_hip.so")

MUON_OK = 0
STATUS = {0: "MUON_OK", 1: "MUON_ERR_INVALID_ARGUMENT", 2: "MUON_ERR_UNSUPPORTED",
          3: "MUON_ERR_OUT_OF_MEMORY", 4: "MUON_ERR_DEVICE"}
F32, BF16 = 0, 1
NS_BF16, NS_F32 = 0, 1
DEFAULT_CHUNK_ELEMS = 1 << 29


class MuonError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class MuonParam(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("momentum", ctypes.c_void_p), ("rows", ctypes.c_int64),
                ("cols", ctypes.c_int64), ("batch", ctypes.c_int64), ("ld", ctypes.c_int64),
                ("param_dtype", ctypes.c_int), ("grad_dtype", ctypes.c_int),
                ("row_block", ctypes.c_int64), ("block_stride", ctypes.c_int64),
                ("plane_stride", ctypes.c_int64), ("momentum_dense", ctypes.c_int32),
                ("post_scale", ctypes.c_float), ("ns_coeffs", ctypes.POINTER(ctypes.c_float)),
                ("ns_steps", ctypes.c_int32), ("scale_mode", ctypes.c_int32)]


class MuonHParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta", ctypes.c_float),
                ("weight_decay", ctypes.c_float), ("eps", ctypes.c_float),
                ("ns_steps", ctypes.c_int32), ("nesterov", ctypes.c_int32),
                ("ns_coeffs", ctypes.POINTER(ctypes.c_float)), ("ns_precision", ctypes.c_int),
                ("scale_mode", ctypes.c_int32), ("max_chunk_elems", ctypes.c_int64)]


class AdamWParam(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("exp_avg", ctypes.c_void_p), ("exp_avg_sq", ctypes.c_void_p),
                ("numel", ctypes.c_int64), ("param_dtype", ctypes.c_int),
                ("grad_dtype", ctypes.c_int)]


class AdamWHParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("reserved", ctypes.c_int32), ("step", ctypes.c_int64)]


class MuonChunkInfo(ctypes.Structure):
    _fields_ = [("s", ctypes.c_int64), ("l", ctypes.c_int64), ("s_pad", ctypes.c_int64),
                ("l_pad", ctypes.c_int64), ("first", ctypes.c_int64), ("count", ctypes.c_int64),
                ("param_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
                ("ns_steps", ctypes.c_int32), ("coeff_set", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t)]


class MuonKernelStats(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char_p), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("exec_flops", ctypes.c_double), ("bytes", ctypes.c_double)]


EXPORTS = ["muon_create", "muon_destroy", "muon_reserve", "muon_set_workspace_limit",
           "muon_workspace_bytes", "muon_step", "ns_orthogonalize_batched",
           "muon_validate_step", "muon_plan_step", "muon_status_string", "muon_last_error",
           "muon_abi_version", "muon_profile_enable", "muon_profile_read", "muon_adamw_step",
           "muon_set_streams", "ns_orthogonalize_batched_noalloc", "muon_stream_copy"]

_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2609_21594_amd.csrc.build` (no fallback exists)")
    lib = ctypes.CDLL(path)
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    lib.muon_create.argtypes = [ctypes.POINTER(vp), ctypes.c_int]
    lib.muon_destroy.argtypes = [vp]
    lib.muon_reserve.argtypes = [vp, ctypes.c_size_t]
    lib.muon_set_workspace_limit.argtypes = [vp, ctypes.c_size_t]
    lib.muon_workspace_bytes.argtypes = [vp]
    lib.muon_workspace_bytes.restype = ctypes.c_size_t
    lib.muon_step.argtypes = [vp, ctypes.POINTER(MuonParam), i64, ctypes.POINTER(MuonHParams), vp]
    for name in ("ns_orthogonalize_batched", "ns_orthogonalize_batched_noalloc"):
        getattr(lib, name).argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp),
                                       ctypes.POINTER(i64), ctypes.POINTER(i64), i64,
                                       ctypes.c_int, i32, ctypes.POINTER(ctypes.c_float),
                                       ctypes.c_float, ctypes.c_int, vp]
    lib.muon_validate_step.argtypes = [ctypes.POINTER(MuonParam), i64, ctypes.POINTER(MuonHParams),
                                       ctypes.c_char_p, ctypes.c_size_t]
    lib.muon_plan_step.argtypes = [ctypes.POINTER(MuonParam), i64, ctypes.POINTER(MuonHParams),
                                   ctypes.POINTER(MuonChunkInfo), i64, ctypes.POINTER(i64),
                                   ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(i64)]
    lib.muon_adamw_step.argtypes = [vp, ctypes.POINTER(AdamWParam), i64, ctypes.POINTER(AdamWHParams), vp]
    lib.muon_profile_enable.argtypes = [vp, ctypes.c_int]
    lib.muon_set_streams.argtypes = [vp, ctypes.c_int]
    lib.muon_set_grouping.argtypes = [vp, ctypes.c_int]
    lib.muon_stream_copy.argtypes = [vp, vp, vp, ctypes.c_size_t, vp]
    lib.muon_profile_read.argtypes = [vp, ctypes.POINTER(MuonKernelStats), ctypes.c_int,
                                      ctypes.POINTER(ctypes.c_int), ctypes.c_int]
    lib.muon_status_string.argtypes = [ctypes.c_int]
    lib.muon_status_string.restype = ctypes.c_char_p
    lib.muon_last_error.argtypes = [vp]
    lib.muon_last_error.restype = ctypes.c_char_p
    for name in ("muon_create", "muon_destroy", "muon_reserve", "muon_set_workspace_limit",
                 "muon_step", "ns_orthogonalize_batched", "muon_validate_step", "muon_plan_step",
                 "muon_profile_enable", "muon_profile_read", "muon_adamw_step", "muon_set_streams",
                 "ns_orthogonalize_batched_noalloc", "muon_stream_copy"):
        getattr(lib, name).restype = ctypes.c_int
    _lib = lib
    return lib


def _coeff_table(ns_coeffs, ns_steps):
    """Flattened K x 3 table; the library reads 3 * ns_steps values, so the
    table must have exactly ns_steps rows of three."""
    rows = [tuple(float(v) for v in r) for r in ns_coeffs]
    if any(len(r) != 3 for r in rows) or len(rows) != int(ns_steps):
        raise ValueError(f"ns_coeffs must be {int(ns_steps)} rows of (a, b, c), got {len(rows)}")
    return [v for r in rows for v in r]


def make_hparams(lr=0.02, beta=0.95, weight_decay=0.0, eps=1e-7, ns_steps=5, nesterov=True,
                 ns_coeffs: Optional[Sequence[Sequence[float]]] = None, ns_precision="bf16",
                 scale_mode=0, max_chunk_elems=0):
    """Returns (struct, keepalive) — keep the second item alive during the call."""
    coeff_arr = None
    if ns_coeffs is not None:
        flat = _coeff_table(ns_coeffs, ns_steps)
        coeff_arr = (ctypes.c_float * max(1, len(flat)))(*flat)
    hp = MuonHParams(lr, beta, weight_decay, eps, int(ns_steps), int(bool(nesterov)),
                     ctypes.cast(coeff_arr, ctypes.POINTER(ctypes.c_float)) if coeff_arr else None,
                     NS_F32 if ns_precision == "f32" else NS_BF16, int(scale_mode),
                     int(max_chunk_elems))
    return hp, coeff_arr


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


class RowBlocks:
    """A logical matrix made of the row blocks of a view: `t` is
    [nblk, rb, N] (or [E, nblk, rb, N]) with unit column stride, and its
    blocks stack into one (nblk*rb) x N matrix (per plane), e.g. the heads of
    one projection inside a fused, head-interleaved QKV weight."""

    def __init__(self, t):
        self.t = t


def _view(x):
    """(tensor, batch, rows, cols, ld, row_block, block_stride, plane_stride)
    of a logical matrix: a tensor [M, N] or [E, M, N] whose columns are
    contiguous (any row and plane strides), or RowBlocks.  Strides of
    singleton dimensions do not matter and become 0, the dense default.
    Dense tensors give all-zero strides except ld = N."""
    blocks = isinstance(x, RowBlocks)
    t = x.t if blocks else x
    if t.dim() == 0 or (t.shape[-1] > 1 and t.stride(-1) != 1):
        raise ValueError("a logical matrix needs contiguous columns")
    if blocks:
        if t.dim() == 3:
            E, nb, rb, N = 1, *tuple(t.shape)
            ps, bs, ld = 0, t.stride(0), t.stride(1)
        elif t.dim() == 4:
            E, nb, rb, N = tuple(t.shape)
            ps, bs, ld = t.stride(0), t.stride(1), t.stride(2)
        else:
            raise ValueError("RowBlocks takes [nblk, rb, N] or [E, nblk, rb, N]")
    elif t.dim() in (2, 3):
        E = 1 if t.dim() == 2 else t.shape[0]
        nb, rb, N = 1, t.shape[-2], t.shape[-1]
        ps, bs, ld = (t.stride(0) if t.dim() == 3 else 0), 0, t.stride(-2)
    else:
        raise ValueError("Muon takes matrices [M, N] or stacks [E, M, N]")
    rows = nb * rb
    # The ABI reads a zero stride as "dense default", so a stride that is
    # really zero or negative (an expanded or broadcast tensor) must never
    # reach it: rows, blocks or planes that overlap are refused here.
    if (rb > 1 and ld < N) or (nb > 1 and bs <= 0) or (E > 1 and ps <= 0):
        raise ValueError("a logical matrix's rows, blocks and planes must not overlap "
                         "(expanded or broadcast tensors are not views Muon can update)")
    if rb == 1:
        ld = N
    if nb == 1:
        rb, bs = 0, 0
    if E == 1:
        ps = 0
    return t, E, rows, N, ld, rb, bs, ps


def params_array(params, grads, moms, entry_coeffs=None, entry_scale_modes=None, entry_post_scales=None):
    """(MuonParam[], keepalive) for lists of logical matrices (see _view).
    grad takes the param's view; momentum takes it too, or is a dense
    [M, N] / [E, M, N] tensor.  entry_coeffs[i] (a K x 3 table) and
    entry_scale_modes[i] override the call's for entry i; None keeps the
    call's.  entry_post_scales[i] multiplies entry i's updated matrix (the
    post-processing stage, e.g. a QK-clip factor); None: none.  Keep the
    second item alive during the call."""
    import torch
    if not (len(params) == len(grads) == len(moms)):
        raise ValueError("params, grads and momenta must have equal length")
    n = len(params)
    entry_coeffs = entry_coeffs or [None] * n
    entry_scale_modes = entry_scale_modes or [None] * n
    entry_post_scales = entry_post_scales or [None] * n
    if len(entry_coeffs) != n or len(entry_scale_modes) != n or len(entry_post_scales) != n:
        raise ValueError("per-entry options need one item per entry")
    arr = (MuonParam * max(1, n))()
    keep = []
    for i, (W, g, m) in enumerate(zip(params, grads, moms)):
        vw, vg, vm = _view(W), _view(g), _view(m)
        if vw[1:] != vg[1:] or tuple(vw[0].shape) != tuple(vg[0].shape):
            raise ValueError(f"entry {i}: grad must have the param's shape and strides")
        if vm[0].dtype != torch.float32:
            raise TypeError(f"entry {i}: momentum must be float32")
        _, batch, rows, cols, ld, rb, bs, ps = vw
        if vm[1:] == vw[1:] and tuple(vm[0].shape) == tuple(vw[0].shape):
            mdense = 0
        elif vm[0].is_contiguous() and vm[0].numel() == batch * rows * cols and vm[3] == cols:
            mdense = 1
        else:
            raise ValueError(f"entry {i}: momentum must have the param's view or be dense")
        ctab, csteps = None, 0
        if entry_coeffs[i] is not None:
            csteps = len(entry_coeffs[i])
            flat = _coeff_table(entry_coeffs[i], csteps)
            ctab = (ctypes.c_float * max(1, len(flat)))(*flat)
            keep.append(ctab)
        smode = 0 if entry_scale_modes[i] is None else 1 + int(entry_scale_modes[i])
        post = 0.0 if entry_post_scales[i] is None else float(entry_post_scales[i])
        arr[i] = MuonParam(vw[0].data_ptr(), vg[0].data_ptr(), vm[0].data_ptr(), rows, cols, batch,
                           ld, _dtype_code(vw[0]), _dtype_code(vg[0]), rb, bs, ps, mdense, post,
                           ctypes.cast(ctab, ctypes.POINTER(ctypes.c_float)) if ctab else None,
                           csteps, smode)
    return arr, keep


def _check_device(tensors, device: int):
    """Every tensor must live on the handle's GPU: a host tensor's address
    must never reach a kernel."""
    for t in tensors:
        t = t.t if isinstance(t, RowBlocks) else t
        if t.device.type != "cuda" or t.device.index != device:
            raise ValueError(f"tensor on {t.device}, the handle runs on cuda:{device}")


def _stream_ptr(stream) -> int:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


class Muon:
    """A library handle on one device; owns the workspace."""

    def __init__(self, device: int = 0):
        self.lib = load_library()
        h = ctypes.c_void_p()
        st = self.lib.muon_create(ctypes.byref(h), int(device))
        if st != MUON_OK:
            raise MuonError(st, f"muon_create(device={device}) failed")
        self.h = h
        self.device = device

    def _check(self, st: int):
        if st != MUON_OK:
            raise MuonError(st, self.lib.muon_last_error(self.h).decode())

    def close(self):
        if getattr(self, "h", None):
            self.lib.muon_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reserve(self, nbytes: int):
        self._check(self.lib.muon_reserve(self.h, int(nbytes)))

    def set_streams(self, n: int):
        """2 (default): chunks that leave CUs idle run on a second stream; 1: off."""
        self._check(self.lib.muon_set_streams(self.h, int(n)))

    def set_grouping(self, enable: bool):
        """muon_set_grouping: chunks that leave compute units idle share one
        launch per product and step (default on)."""
        self._check(self.lib.muon_set_grouping(self.h, 1 if enable else 0))

    def set_workspace_limit(self, nbytes: int):
        self._check(self.lib.muon_set_workspace_limit(self.h, int(nbytes)))

    def profile(self, enable: bool = True):
        """Bracket every launch with HIP events on its stream."""
        self._check(self.lib.muon_profile_enable(self.h, int(bool(enable))))

    def profile_read(self, reset: bool = True):
        """{family: dict(launches, total_ms, flops, exec_flops, bytes)}; waits for the events."""
        arr = (MuonKernelStats * 16)()
        n = ctypes.c_int()
        self._check(self.lib.muon_profile_read(self.h, arr, 16, ctypes.byref(n), int(bool(reset))))
        return {arr[i].name.decode(): {f: getattr(arr[i], f) for f, _ in MuonKernelStats._fields_[1:]}
                for i in range(n.value)}

    def stream_copy(self, dst, src, stream=None):
        """dst <- src with the library's HBM reference copy (muon_stream_copy);
        same-size device tensors, contiguous."""
        _check_device([dst, src], self.device)
        nbytes = src.numel() * src.element_size()
        if dst.numel() * dst.element_size() != nbytes or not (dst.is_contiguous() and src.is_contiguous()):
            raise ValueError("stream_copy needs contiguous tensors of equal size")
        self._check(self.lib.muon_stream_copy(self.h, ctypes.c_void_p(dst.data_ptr()),
                                              ctypes.c_void_p(src.data_ptr()), nbytes,
                                              ctypes.c_void_p(_stream_ptr(stream))))

    @property
    def workspace_bytes(self) -> int:
        return int(self.lib.muon_workspace_bytes(self.h))

    def step(self, params, grads, moms, stream=None, entry_coeffs=None, entry_scale_modes=None,
             entry_post_scales=None, **hp_kw):
        """In place: momentum and params updated, grads read (muon_step).
        entry_coeffs / entry_scale_modes / entry_post_scales: optional
        per-entry overrides (see params_array)."""
        _check_device(list(params) + list(grads) + list(moms), self.device)
        arr, keep_e = params_array(params, grads, moms, entry_coeffs, entry_scale_modes, entry_post_scales)
        hp, keep = make_hparams(**hp_kw)
        self._check(self.lib.muon_step(self.h, arr, len(params), ctypes.byref(hp),
                                       ctypes.c_void_p(_stream_ptr(stream))))
        del keep, keep_e

    def adamw_step(self, params, grads, exp_avgs, exp_avg_sqs, step, lr=1e-3, betas=(0.9, 0.999),
                   eps=1e-8, weight_decay=0.0, stream=None):
        """AdamW on contiguous tensors of any shape (muon_adamw_step): params
        and both moments updated in place, grads read; `step` is t >= 1."""
        n = len(params)
        if not (len(grads) == len(exp_avgs) == len(exp_avg_sqs) == n):
            raise ValueError("params, grads and moments must have equal length")
        _check_device(list(params) + list(grads) + list(exp_avgs) + list(exp_avg_sqs), self.device)
        arr = (AdamWParam * max(1, n))()
        for i, (p, g, m, v) in enumerate(zip(params, grads, exp_avgs, exp_avg_sqs)):
            if not (p.numel() == g.numel() == m.numel() == v.numel()):
                raise ValueError(f"entry {i}: element counts differ")
            for t in (p, g, m, v):
                if not t.is_contiguous():
                    raise ValueError(f"entry {i}: tensors must be contiguous")
            if _dtype_code(m) != F32 or _dtype_code(v) != F32:
                raise TypeError(f"entry {i}: moments must be float32")
            arr[i] = AdamWParam(p.data_ptr(), g.data_ptr(), m.data_ptr(), v.data_ptr(), p.numel(),
                                _dtype_code(p), _dtype_code(g))
        hp = AdamWHParams(float(lr), float(betas[0]), float(betas[1]), float(eps), float(weight_decay),
                          0, int(step))
        self._check(self.lib.muon_adamw_step(self.h, arr, n, ctypes.byref(hp),
                                             ctypes.c_void_p(_stream_ptr(stream))))

    def orthogonalize(self, inputs, outputs, ns_steps=5, ns_coeffs=None, eps=1e-7,
                      ns_precision="bf16", stream=None, noalloc=False):
        """outputs[i] <- NS(inputs[i]) (ns_orthogonalize_batched); 2-D tensors.
        With noalloc, ns_orthogonalize_batched_noalloc: the library's fixed
        device array instead of the handle's workspace (no allocation)."""
        n = len(inputs)
        if len(outputs) != n:
            raise ValueError("inputs and outputs differ in length")
        if n == 0:
            return
        _check_device(list(inputs) + list(outputs), self.device)
        dt = _dtype_code(inputs[0])
        ins = (ctypes.c_void_p * n)()
        outs = (ctypes.c_void_p * n)()
        rows = (ctypes.c_int64 * n)()
        cols = (ctypes.c_int64 * n)()
        for i, (a, b) in enumerate(zip(inputs, outputs)):
            if a.dim() != 2 or a.shape != b.shape:
                raise ValueError(f"matrix {i}: need equal 2-D shapes")
            if _dtype_code(a) != dt or _dtype_code(b) != dt:
                raise TypeError("all inputs and outputs must share one dtype")
            if not (a.is_contiguous() and b.is_contiguous()):
                raise ValueError(f"matrix {i}: tensors must be contiguous")
            ins[i], outs[i] = a.data_ptr(), b.data_ptr()
            rows[i], cols[i] = a.shape[0], a.shape[1]
        coeff = None
        if ns_coeffs is not None:
            flat = _coeff_table(ns_coeffs, ns_steps)
            coeff = (ctypes.c_float * max(1, len(flat)))(*flat)
        fn = self.lib.ns_orthogonalize_batched_noalloc if noalloc else self.lib.ns_orthogonalize_batched
        self._check(fn(
            self.h, ins, outs, rows, cols, n, dt, int(ns_steps),
            ctypes.cast(coeff, ctypes.POINTER(ctypes.c_float)) if coeff else None,
            float(eps), NS_F32 if ns_precision == "f32" else NS_BF16,
            ctypes.c_void_p(_stream_ptr(stream))))


def validate_step(entries: Sequence[MuonParam], hp: MuonHParams):
    """Host-only check (no device): returns (status, message)."""
    lib = load_library()
    arr = (MuonParam * max(1, len(entries)))(*entries)
    msg = ctypes.create_string_buffer(256)
    st = lib.muon_validate_step(arr, len(entries), ctypes.byref(hp), msg, 256)
    return st, msg.value.decode()


def plan_step(entries: Sequence[MuonParam], hp: MuonHParams):
    """Host-only plan: (status, [chunk dicts], workspace bytes, plan order)."""
    lib = load_library()
    arr = (MuonParam * max(1, len(entries)))(*entries)
    nch = ctypes.c_int64()
    ws = ctypes.c_size_t()
    st = lib.muon_plan_step(arr, len(entries), ctypes.byref(hp), None, 0, ctypes.byref(nch),
                            ctypes.byref(ws), None)
    if st != MUON_OK:
        return st, [], 0, []
    total = sum(e.batch for e in entries)
    chunks = (MuonChunkInfo * max(1, nch.value))()
    order = (ctypes.c_int64 * max(1, total))()
    st = lib.muon_plan_step(arr, len(entries), ctypes.byref(hp), chunks, nch.value,
                            ctypes.byref(nch), ctypes.byref(ws), order)
    out = [{f: getattr(chunks[i], f) for f, _ in MuonChunkInfo._fields_} for i in range(nch.value)]
    return st, out, ws.value, list(order[:total])
