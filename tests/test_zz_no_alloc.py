"""The allocation-free step, micro_sparsify_step_noalloc, against
micro_sparsify_step through the C ABI (GPU).

Both entry points get the same inputs; indices, values, the selected count,
the next threshold and the residual must be equal bit for bit.  Consecutive
calls share the device's static scratch, so the sequences below run calls of
different sizes back to back.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2310_00967_amd import _lib

pytestmark = pytest.mark.gpu

DEV = "cuda"


def note(msg):
    print(msg, flush=True)


class Pair:
    """One vector on both paths: the existing entry point on a context of its
    own (default schedule), the allocation-free one on the device's static
    scratch."""

    def __init__(self, g, res, phase=0):
        self.N = g.size
        self.ctx = _lib.micro_sparsify_init(self.N, torch.cuda.current_stream().cuda_stream)
        # grad at `phase` values past a 16-byte boundary relative to residual
        gbuf = torch.empty(self.N + 4, dtype=torch.float32, device=DEV)
        self.g = gbuf[phase:phase + self.N]
        self.g.copy_(torch.from_numpy(g))
        self.res_a = torch.from_numpy(res).to(DEV)
        self.res_b = self.res_a.clone()
        cap = max(1, self.N) + 8
        self.idx_a = torch.full((cap,), -7, dtype=torch.int32, device=DEV)
        self.val_a = torch.full((cap,), -7.0, dtype=torch.float32, device=DEV)
        self.idx_b = self.idx_a.clone()
        self.val_b = self.val_a.clone()

    def call(self, rank, world, density, theta, stream_handle):
        k_a, th_a = _lib.micro_sparsify_step(self.ctx, self.g.data_ptr(), self.res_a.data_ptr(), rank, world,
                                             density, theta, self.idx_a.data_ptr(), self.val_a.data_ptr())
        k_b, th_b = _lib.micro_sparsify_step_noalloc(self.g.data_ptr(), self.res_b.data_ptr(), self.N, rank, world,
                                                     density, theta, self.idx_b.data_ptr(),
                                                     self.val_b.data_ptr(), stream_handle)
        torch.cuda.synchronize()
        assert k_b == k_a
        assert th_b == th_a
        assert torch.equal(self.idx_b, self.idx_a)  # first k pairs and the untouched tail
        assert torch.equal(self.val_b.view(torch.int32), self.val_a.view(torch.int32))
        assert torch.equal(self.res_b.view(torch.int32), self.res_a.view(torch.int32))
        return k_b, th_b

    def close(self):
        _lib.micro_sparsify_free(self.ctx)


def make(N, seed):
    rng = np.random.default_rng(seed)
    g = rng.standard_normal(N).astype(np.float32)
    res = (rng.standard_normal(N) * 0.7).astype(np.float32)
    return g, res


@pytest.mark.parametrize("stream", ["null", "torch"])
def test_two_calls_second_smaller(stream):
    handle = None if stream == "null" else torch.cuda.current_stream().cuda_stream
    # 2,500,001-value partition (611 tiles of 4096), then a 100,002-value one:
    # the second call meets the first call's look-back words in the scratch
    for N, world, rank, seed in [(5_000_003, 2, 1, 1), (300_007, 3, 2, 2)]:
        note(f"noalloc N={N} world={world} rank={rank} stream={stream}")
        g, res = make(N, seed)
        p = Pair(g, res)
        try:
            k, _ = p.call(rank, world, 0.01, 2.3, handle)
            assert k > 0
        finally:
            p.close()


def test_error_feedback_sequence_and_scalar_loads():
    """Ten error-feedback steps on one vector (residual carried, threshold
    updated), alternating partitions of different lengths, with grad at a
    different 16-byte phase than residual (the scalar-load kernel)."""
    N, world = 1_000_003, 3
    g, res = make(N, 3)
    p = Pair(g, res, phase=1)
    try:
        theta = 2.0
        for t in range(10):
            rank = t % world
            note(f"noalloc error-feedback step {t} rank {rank}")
            _, theta = p.call(rank, world, 0.01, theta, None)
    finally:
        p.close()


def test_degenerate_sizes():
    """An empty partition (nothing launched), a one-value vector and a
    partition that selects everything."""
    for N, world, rank, theta in [(2, 5, 0, 1.0), (1, 1, 0, 1e-30), (4097, 1, 0, 1e-30), (4099, 2, 1, 1e30)]:
        note(f"noalloc degenerate N={N} world={world} rank={rank} theta={theta}")
        g, res = make(N, N)
        p = Pair(g, res)
        try:
            p.call(rank, world, 0.5, theta, None)
        finally:
            p.close()


def test_argument_errors_leave_everything_untouched():
    lib = _lib.load()
    g = torch.ones(16, dtype=torch.float32, device=DEV)
    r = torch.zeros(16, dtype=torch.float32, device=DEV)
    oi = torch.zeros(16, dtype=torch.int32, device=DEV)
    ov = torch.zeros(16, dtype=torch.float32, device=DEV)
    th = ctypes.c_double(1.0)
    k = ctypes.c_int64(-3)
    p = ctypes.c_void_p
    # overlapping grad and residual
    st = lib.micro_sparsify_step_noalloc(p(g.data_ptr()), p(g.data_ptr()), 16, 0, 1, 0.1, ctypes.byref(th),
                                         p(oi.data_ptr()), p(ov.data_ptr()), ctypes.byref(k), None, None)
    assert st == _lib.MICRO_EINVAL
    # threshold not positive
    th0 = ctypes.c_double(-1.0)
    st = lib.micro_sparsify_step_noalloc(p(g.data_ptr()), p(r.data_ptr()), 16, 0, 1, 0.1, ctypes.byref(th0),
                                         p(oi.data_ptr()), p(ov.data_ptr()), ctypes.byref(k), None, None)
    assert st == _lib.MICRO_EINVAL
    torch.cuda.synchronize()
    assert th.value == 1.0 and th0.value == -1.0 and k.value == -3
    assert not torch.any(r) and not torch.any(oi) and not torch.any(ov)
