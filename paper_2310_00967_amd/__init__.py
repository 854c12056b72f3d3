"""MiCRO's per-worker gradient sparsification step on MI355X (gfx950).

    sp = Sparsifier(n_total)                       # on torch's current device/stream
    k, theta, idx, val = sp.step(grad, residual, rank, world, density, theta)
    k, theta, cycle, idx, val = sp.ef_step(grad, residual, t, worker, world, density, theta)
    ks, thetas, sumsq, idx, val = sp.sweep(grad, residual, world, density, thetas)
    g = sp.union_gather(residual, union_idx, own_first, val)   # around the exchange
    sp.sparse_update(x, union_idx, summed, world)

`grad` and `residual` are contiguous float32 device tensors of n_total values;
`residual` is updated in place over the rank's partition only; `idx`/`val`
are views of the first k entries of preallocated output tensors.  Every step
runs in the HIP library behind include/micro_sparsify.h; PyTorch only
provides device memory and the stream.
"""
import ctypes

from . import _lib
from ._lib import (MICRO_FLAG_SEPARATE_SCAN, MICRO_FLAG_TIME_KERNEL, MICRO_RULE_FIXED_STEP,
                   MICRO_RULE_HARD_THRESHOLD, MICRO_RULE_PROPORTIONAL, MICRO_RULE_TOPK, MICRO_VARIANT_AUTO,
                   MICRO_TOPK_ROUTE_FULL, MICRO_TOPK_ROUTE_HINT_LIST, MICRO_TOPK_ROUTE_HINT_PICK,
                   MICRO_TOPK_ROUTE_LIST, MICRO_VARIANT_STAGED, MICRO_VARIANT_TICKET, MicroError, default_config, micro_cycle, micro_estimate_threshold,
                   micro_partition, micro_threshold_f32)

__all__ = ["Sparsifier", "MicroError", "default_config", "micro_partition", "micro_cycle",
           "micro_estimate_threshold", "micro_threshold_f32", "MICRO_RULE_PROPORTIONAL",
           "MICRO_RULE_FIXED_STEP", "MICRO_RULE_HARD_THRESHOLD", "MICRO_RULE_TOPK", "MICRO_VARIANT_AUTO",
           "MICRO_VARIANT_TICKET",
           "MICRO_VARIANT_STAGED",
           "MICRO_FLAG_TIME_KERNEL", "MICRO_FLAG_SEPARATE_SCAN", "MICRO_TOPK_ROUTE_FULL", "MICRO_TOPK_ROUTE_LIST",
           "MICRO_TOPK_ROUTE_HINT_LIST", "MICRO_TOPK_ROUTE_HINT_PICK"]


class Sparsifier:
    """One context of the C library bound to a torch device and stream."""

    def __init__(self, n_total, device=None, stream=None, rule=MICRO_RULE_PROPORTIONAL, beta=None,
                 lo=None, hi=None, alpha=None, variant=MICRO_VARIANT_AUTO, time_kernel=False,
                 separate_scan=False):
        import torch
        if not torch.cuda.is_available():
            raise RuntimeError("Sparsifier needs a HIP device")
        dev = torch.device(device) if device is not None else torch.device("cuda")
        if dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.n_total = int(n_total)
        cfg = default_config()
        cfg.rule = rule
        for name, v in (("beta", beta), ("lo", lo), ("hi", hi), ("alpha", alpha)):
            if v is not None:
                setattr(cfg, name, float(v))
        cfg.variant = variant
        cfg.flags = (MICRO_FLAG_TIME_KERNEL if time_kernel else 0) | (MICRO_FLAG_SEPARATE_SCAN if separate_scan else 0)
        self.config = cfg
        with torch.cuda.device(self.device):
            self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
            self._ctx = _lib.micro_sparsify_init(self.n_total, self.stream.cuda_stream, cfg)
        self._out_idx = None
        self._out_val = None
        self._lengths = {}  # (rank, world) -> partition length
        # per-call marshalling objects, made once (a context serves one
        # caller at a time): the step's in/out scalars and the stats record
        lib = _lib.load()
        self._step_fn = lib.micro_sparsify_step
        self._stats_fn = lib.micro_sparsify_last_stats
        self._theta_c = ctypes.c_double()
        self._k_c = ctypes.c_int64()
        self._theta_p = ctypes.pointer(self._theta_c)
        self._k_p = ctypes.pointer(self._k_c)
        self._stats_c = _lib.micro_step_stats()
        self._stats_p = ctypes.pointer(self._stats_c)
        self._f32, self._i32 = torch.float32, torch.int32
        self._tensor = torch.Tensor
        # the sweep's and the full pass's marshalling objects
        self._sweep_fn = lib.micro_sweep_step
        self._ef_fn = lib.micro_ef_step
        self._sweep_arrays = {}  # world -> (thetas, ks, sumsq ctypes arrays and their addresses)
        self._cycle_c = ctypes.c_int32()
        self._cycle_p = ctypes.pointer(self._cycle_c)
        self._sumsq_c = ctypes.c_double()
        self._sumsq_p = ctypes.pointer(self._sumsq_c)

    def close(self):
        if getattr(self, "_ctx", None) is not None:
            _lib.micro_sparsify_free(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def partition(self, rank, world):
        return micro_partition(self.n_total, rank, world)

    def outputs(self, capacity):
        """Preallocated (out_idx int32, out_val float32) of at least `capacity`."""
        import torch
        if self._out_idx is None or self._out_idx.numel() < capacity:
            n = max(1, int(capacity))
            self._out_idx = torch.empty(n, dtype=torch.int32, device=self.device)
            self._out_val = torch.empty(n, dtype=torch.float32, device=self.device)
        return self._out_idx, self._out_val

    def _check(self, t, name, dtype):
        import torch
        if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda \
                or t.get_device() != self.device.index or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous {dtype} tensor on {self.device}")

    def _length(self, rank, world):
        key = (rank, world)
        length = self._lengths.get(key)
        if length is None:
            length = self.partition(rank, world)[1]
            self._lengths[key] = length
        return length

    def _fits(self, t, dtype):
        return (isinstance(t, self._tensor) and t.dtype is dtype and t.is_cuda
                and t.get_device() == self.device.index and t.is_contiguous())

    def step(self, grad, residual, rank, world, density, theta, out_idx=None, out_val=None):
        """One sparsify step; returns (k, theta_next, idx[:k], val[:k]).

        idx and val are views of out_idx / out_val; without them, of this
        Sparsifier's own output buffers, which the next call overwrites: pass
        buffers of your own (or clone the views) to keep a step's selection
        while the next one runs."""
        if self._ctx is None:
            raise RuntimeError("Sparsifier is closed")
        length = self._length(rank, world)
        if out_idx is None or out_val is None:
            out_idx, out_val = self.outputs(length)
        self._check_vectors(grad, residual, out_idx, out_val)
        if out_idx.numel() < length or out_val.numel() < length:
            raise ValueError(f"output capacity below the partition length {length}")
        self._theta_c.value = float(theta)
        st = self._step_fn(self._ctx, grad.data_ptr(), residual.data_ptr(), int(rank), int(world), float(density),
                           self._theta_p, out_idx.data_ptr(), out_val.data_ptr(), self._k_p)
        if st:
            _lib.check(st, self._ctx)
        k = self._k_c.value
        return k, self._theta_c.value, out_idx[:k], out_val[:k]

    def _check_vectors(self, grad, residual, out_idx, out_val):
        f32 = self._f32
        if not (self._fits(grad, f32) and self._fits(residual, f32) and self._fits(out_idx, self._i32)
                and self._fits(out_val, f32)):
            # name the offending argument
            self._check(grad, "grad", f32)
            self._check(residual, "residual", f32)
            self._check(out_idx, "out_idx", self._i32)
            self._check(out_val, "out_val", f32)
        if grad.numel() != self.n_total or residual.numel() != self.n_total:
            raise ValueError(f"grad and residual must hold {self.n_total} values")

    def ef_step(self, grad, residual, t, worker, world, density, theta, out_idx=None, out_val=None,
                local_error=False):
        """Algorithm 1 for `worker` at iteration t over the whole vector: every
        value accumulates, the partition of the worker's cycle is searched.
        Returns (k, theta_next, cycle, idx[:k], val[:k]); with local_error,
        (k, theta_next, cycle, idx[:k], val[:k], sumsq) where sumsq is the
        squared norm of the whole new residual.  idx and val are views of the
        output buffers, as in step."""
        if self._ctx is None:
            raise RuntimeError("Sparsifier is closed")
        length = self._length(_lib.micro_cycle(t, worker, world), world)
        if out_idx is None or out_val is None:
            out_idx, out_val = self.outputs(length)
        self._check_vectors(grad, residual, out_idx, out_val)
        if out_idx.numel() < length or out_val.numel() < length:
            raise ValueError(f"output capacity below the partition length {length}")
        self._theta_c.value = float(theta)
        st = self._ef_fn(self._ctx, grad.data_ptr(), residual.data_ptr(), int(t), int(worker), int(world),
                         float(density), self._theta_p, out_idx.data_ptr(), out_val.data_ptr(), self._k_p,
                         self._cycle_p, self._sumsq_p if local_error else None)
        if st:
            _lib.check(st, self._ctx)
        k = self._k_c.value
        if local_error:
            return k, self._theta_c.value, self._cycle_c.value, out_idx[:k], out_val[:k], self._sumsq_c.value
        return k, self._theta_c.value, self._cycle_c.value, out_idx[:k], out_val[:k]

    def sweep(self, grad, residual, world, density, thetas, out_idx=None, out_val=None, want_sumsq=True):
        """Every partition of `world` searched once, each with its own
        threshold, in one launch of each kernel.  Returns (k list, thetas_next
        list, sumsq list or None, idx[:sum k], val[:sum k]); partition r's
        pairs start at sum(k[:r])."""
        if self._ctx is None:
            raise RuntimeError("Sparsifier is closed")
        world = int(world)
        if len(thetas) != world:
            raise ValueError("one threshold per partition")
        if out_idx is None or out_val is None:
            out_idx, out_val = self.outputs(self.n_total)
        self._check_vectors(grad, residual, out_idx, out_val)
        if out_idx.numel() < self.n_total or out_val.numel() < self.n_total:
            raise ValueError(f"output capacity below n_total {self.n_total}")
        arrays = self._sweep_arrays.get(world)
        if arrays is None:
            n = max(1, world)
            th, kk, sq = (ctypes.c_double * n)(), (ctypes.c_int64 * n)(), (ctypes.c_double * n)()
            arrays = (th, kk, sq, ctypes.addressof(th), ctypes.addressof(kk), ctypes.addressof(sq))
            self._sweep_arrays[world] = arrays
        th, kk, sq, th_a, kk_a, sq_a = arrays
        th[:world] = [float(x) for x in thetas]
        st = self._sweep_fn(self._ctx, grad.data_ptr(), residual.data_ptr(), world, float(density), th_a,
                            out_idx.data_ptr(), out_val.data_ptr(), kk_a, sq_a if want_sumsq else None)
        if st:
            _lib.check(st, self._ctx)
        k = kk[:world]
        total = sum(k)
        return k, th[:world], (sq[:world] if want_sumsq else None), out_idx[:total], out_val[:total]

    def union_gather(self, residual, union_idx, own_first, own_val, out=None):
        """The accumulated values at the union of the workers' selections and
        their reset in `residual`; own_val (this worker's k selected values)
        sits at union positions [own_first, own_first + k).  Enqueued on the
        context's stream.  Returns out (float32, len(union_idx))."""
        import torch
        self._check(residual, "residual", torch.float32)
        self._check(union_idx, "union_idx", torch.int32)
        self._check(own_val, "own_val", torch.float32)
        if residual.numel() != self.n_total:
            raise ValueError(f"residual must hold {self.n_total} values")
        m = union_idx.numel()
        if out is None:
            out = torch.empty(max(1, m), dtype=torch.float32, device=self.device)[:m]
        self._check(out, "out", torch.float32)
        if out.numel() < m:
            raise ValueError("out smaller than the union")
        _lib.micro_union_gather(self._ctx, residual.data_ptr(), union_idx.data_ptr(), m, own_first,
                                own_val.numel(), own_val.data_ptr(), out.data_ptr())
        return out

    def sparse_update(self, x, union_idx, sums, world):
        """x[union_idx] -= sums / world (enqueued on the context's stream)."""
        import torch
        self._check(x, "x", torch.float32)
        self._check(union_idx, "union_idx", torch.int32)
        self._check(sums, "sums", torch.float32)
        if x.numel() != self.n_total:
            raise ValueError(f"x must hold {self.n_total} values")
        if sums.numel() != union_idx.numel():
            raise ValueError("sums and union_idx lengths differ")
        _lib.micro_sparse_update(self._ctx, x.data_ptr(), union_idx.data_ptr(), sums.data_ptr(),
                                 union_idx.numel(), world)

    def last_stats(self):
        """(kernel_ms, redone_tiles, variant, fused) of the last step."""
        if self._ctx is None:
            raise RuntimeError("Sparsifier is closed")
        st = self._stats_fn(self._ctx, self._stats_p)
        if st:
            _lib.check(st, self._ctx)
        s = self._stats_c
        return s.kernel_ms, s.redone_tiles, s.variant, s.fused

    def last_topk_route(self):
        """MICRO_RULE_TOPK: how the last step found the k-th magnitude
        (MICRO_TOPK_ROUTE_*), else 0."""
        self.last_stats()
        return self._stats_c.topk_route

    def last_kernel_ms(self):
        return self.last_stats()[0]
