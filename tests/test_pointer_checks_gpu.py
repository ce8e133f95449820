"""The launching entry points refuse buffers a kernel could not address:
host memory (pageable or pinned) and views that run past the end of their
allocation.  Called through the C ABI with the binding's own checks
bypassed.

Every case runs on a handle whose workspace limit (1 KB) is below what any
plan needs, so that muon_step and ns_orthogonalize_batched could not launch
a kernel even if a check let the call through: such a call would fail with
MUON_ERR_OUT_OF_MEMORY instead, and the test with it.
"""
import ctypes

import numpy as np
import pytest

from tests.gpu_util import require_gpu

pytestmark = pytest.mark.gpu

INVALID, OOM = 1, 3


@pytest.fixture(scope="module")
def guarded():
    require_gpu()
    from paper_2609_21594_amd.binding import Muon
    m = Muon(0)
    m.set_workspace_limit(1024)
    yield m
    m.close()


def step_raw(m, W, G, M, rows, cols):
    from paper_2609_21594_amd import binding as B
    import torch
    arr = (B.MuonParam * 1)(B.MuonParam(W, G, M, rows, cols, 1, 0, B.BF16, B.BF16))
    hp, keep = B.make_hparams()
    st = m.lib.muon_step(m.h, arr, 1, ctypes.byref(hp),
                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return st, m.lib.muon_last_error(m.h).decode()


def test_host_buffers_are_refused(guarded):
    import torch
    rows, cols = 64, 128
    g = torch.zeros((rows, cols), dtype=torch.bfloat16, device="cuda")
    mom = torch.zeros((rows, cols), dtype=torch.float32, device="cuda")
    pageable = np.zeros(rows * cols, dtype=np.uint16)
    pinned = torch.zeros((rows, cols), dtype=torch.bfloat16).pin_memory()
    for host in (pageable.ctypes.data, pinned.data_ptr()):
        st, msg = step_raw(guarded, host, g.data_ptr(), mom.data_ptr(), rows, cols)
        assert st == INVALID and "device memory" in msg, (st, msg)
    # orthogonalize: a pinned output
    from paper_2609_21594_amd import binding as B
    ins = (ctypes.c_void_p * 1)(g.data_ptr())
    outs = (ctypes.c_void_p * 1)(pinned.data_ptr())
    r = (ctypes.c_int64 * 1)(rows)
    c = (ctypes.c_int64 * 1)(cols)
    st = guarded.lib.ns_orthogonalize_batched(guarded.h, ins, outs, r, c, 1, B.BF16, 5, None, 1e-7,
                                              B.NS_BF16, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == INVALID and "device memory" in guarded.lib.muon_last_error(guarded.h).decode()
    torch.cuda.synchronize()


def test_view_past_its_allocation_is_refused(guarded):
    # a two-row parameter whose second row starts 32 TB after its first: the
    # first lies in a device allocation, the last byte in unmapped addresses
    import torch
    from paper_2609_21594_amd import binding as B
    hip = ctypes.CDLL("libamdhip64.so")
    t = torch.empty(16 << 20, dtype=torch.uint8, device="cuda")
    g = torch.zeros((2, 4096), dtype=torch.bfloat16, device="cuda")
    mom = torch.zeros((2, 4096), dtype=torch.float32, device="cuda")
    ld = 1 << 44  # elements
    # the gradient: the next 8 KB of the same allocation, in the same layout;
    # the momentum dense
    arr = (B.MuonParam * 1)(B.MuonParam(t.data_ptr(), t.data_ptr() + 8192, mom.data_ptr(), 2, 4096, 1, ld,
                                        B.BF16, B.BF16, 0, 0, 0, 1, 0))
    hp, keep = B.make_hparams()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    st = guarded.lib.muon_step(guarded.h, arr, 1, ctypes.byref(hp), stream)
    msg = guarded.lib.muon_last_error(guarded.h).decode()
    assert st == INVALID and "past the end" in msg, (st, msg)
    # a view that ends exactly at the end of its allocation passes the checks
    # and stops at the workspace limit
    base, size = ctypes.c_void_p(), ctypes.c_size_t()
    assert hip.hipMemGetAddressRange(ctypes.byref(base), ctypes.byref(size), ctypes.c_void_p(t.data_ptr())) == 0
    end = base.value + size.value
    for a in (g, mom):  # the other buffers lie in allocations of their own
        assert not (base.value <= a.data_ptr() < end)
    arr = (B.MuonParam * 1)(B.MuonParam(end - 8192, g.data_ptr(), mom.data_ptr(), 1, 4096, 1, 0,
                                        B.BF16, B.BF16))
    st = guarded.lib.muon_step(guarded.h, arr, 1, ctypes.byref(hp), stream)
    assert st == OOM, (st, guarded.lib.muon_last_error(guarded.h).decode())
    torch.cuda.synchronize()
