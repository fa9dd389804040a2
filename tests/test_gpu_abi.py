"""The library's own checks of device arguments, on the GPU: a host address, or a device
address whose allocation ends before the bytes the call needs, is refused with
DTP_ERR_INVALID_ARG before any kernel is enqueued (so no kernel can read or write outside
what the caller owns).  Raw addresses go straight to the C ABI, past the binding's own
checks."""
import ctypes
import sys

import numpy as np
import pytest
import torch

from paper_2609_13846_amd import dtp

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


class RawAllocation:
    """A device allocation of its own (hipMalloc), so that its end is known exactly; the
    caching allocator's blocks may share a larger segment with other tensors."""

    def __init__(self, nbytes):
        torch.cuda.init()
        self.hip = ctypes.CDLL("libamdhip64.so")
        p = ctypes.c_void_p()
        assert self.hip.hipMalloc(ctypes.byref(p), ctypes.c_size_t(nbytes)) == 0
        assert self.hip.hipMemset(p, 0, ctypes.c_size_t(nbytes)) == 0
        self.base, self.size = p.value, nbytes
        # the runtime reports exactly this range, which is what the library checks against
        base, size = ctypes.c_void_p(), ctypes.c_size_t()
        assert self.hip.hipMemGetAddressRange(ctypes.byref(base), ctypes.byref(size), p) == 0
        assert (base.value, size.value) == (self.base, nbytes)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        torch.cuda.synchronize()
        assert self.hip.hipFree(ctypes.c_void_p(self.base)) == 0


def test_host_address_is_refused():
    announce("abi checks: host address")
    lib = dtp.lib()
    I, G = 64, 4
    s = torch.ones(I, device="cuda")
    B = torch.ones(G, I, device="cuda")
    host = np.zeros(I * G, np.float32)
    st = lib.dtp_down_affinity(I, G, s.data_ptr(), B.data_ptr(), host.ctypes.data, None)
    assert st == dtp.DTP_ERR_INVALID_ARG
    assert "not device memory" in lib.dtp_last_error().decode()
    assert np.all(host == 0)
    # the failed query leaves no error behind for the next call
    out = torch.zeros(I, G, device="cuda")
    dtp.dtp_down_affinity(I, G, s, B, out)
    torch.cuda.synchronize()
    assert torch.equal(out, (s[:, None] * B.t()).contiguous())


def test_allocation_too_short_is_refused():
    announce("abi checks: short allocation")
    lib = dtp.lib()
    I, G = 4096, 8
    s = torch.ones(I, device="cuda")
    B = torch.ones(G, I, device="cuda")
    with RawAllocation(1 << 20) as raw:
        near_end = raw.base + raw.size - 1024           # 1 KB left in the allocation
        st = lib.dtp_down_affinity(I, G, s.data_ptr(), B.data_ptr(), ctypes.c_void_p(near_end), None)
        assert st == dtp.DTP_ERR_INVALID_ARG
        assert "bytes left in its allocation" in lib.dtp_last_error().decode()
        # exactly enough room is accepted
        n = 1024 // (4 * G)
        st = lib.dtp_down_affinity(n, G, s.data_ptr(), B.data_ptr(), ctypes.c_void_p(near_end), None)
        assert st == dtp.DTP_OK, lib.dtp_last_error().decode()


def test_short_token_buffer_is_refused_by_the_layer():
    announce("abi checks: short token buffer")
    lib = dtp.lib()
    layer = dtp.dtp_layer_create(64, 128, 8, 4, 16, 1e-6, dtp.DTP_F32)
    try:
        w = [torch.randn(*sh, device="cuda") * 0.05 for sh in [(64, 128), (64,), (128, 64), (128, 64), (64, 128)]]
        dtp.dtp_layer_set_weights(layer, *w)
        x = torch.randn(100, 64, device="cuda")
        a = torch.randn(100, 8, 16, device="cuda")
        A = torch.zeros(4, 128, device="cuda")
        with RawAllocation(1 << 20) as raw:
            tail = raw.base + raw.size - 64 * 4 * 10    # room for 10 tokens of x, the call asks for 100
            st = lib.dtp_affinity_accumulate(ctypes.c_void_p(layer), ctypes.c_void_p(tail), a.data_ptr(),
                                             100, A.data_ptr(), None)
            assert st == dtp.DTP_ERR_INVALID_ARG
            assert "x (" in lib.dtp_last_error().decode()
        assert torch.count_nonzero(A) == 0
        dtp.dtp_affinity_accumulate(layer, x, a, 100, A)
        torch.cuda.synchronize()
        assert torch.all(A > 0)
    finally:
        dtp.dtp_layer_destroy(layer)
