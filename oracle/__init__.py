"""The CPU oracle for MiCRO's per-worker sparsify step -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package.  It wraps oracle/libmicro_oracle.so (plain single-threaded C, see
micro_oracle.h) through ctypes and works on host numpy arrays.  It shares no
code with the GPU library.
"""
import ctypes
import os

import numpy as np

from .build import LIB, build_oracle

PROPORTIONAL = 0
FIXED_STEP = 1


class Rule(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("beta", ctypes.c_double),
                ("lo", ctypes.c_double), ("hi", ctypes.c_double),
                ("alpha", ctypes.c_double)]


_lib = None


def lib():
    """Loads the oracle library, building it first if it is absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build_oracle()
        L = ctypes.CDLL(LIB)
        i64p = ctypes.POINTER(ctypes.c_int64)
        L.micro_oracle_default_rule.argtypes = [ctypes.POINTER(Rule)]
        L.micro_oracle_default_rule.restype = None
        L.micro_oracle_partition.argtypes = [ctypes.c_int64, ctypes.c_int32,
                                             ctypes.c_int32, i64p, i64p]
        L.micro_oracle_partition.restype = ctypes.c_int
        L.micro_oracle_select.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_double, ctypes.c_void_p,
                                          ctypes.c_void_p]
        L.micro_oracle_select.restype = ctypes.c_int64
        L.micro_oracle_estimate.argtypes = [ctypes.POINTER(Rule), ctypes.c_double,
                                            ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_double]
        L.micro_oracle_estimate.restype = ctypes.c_double
        L.micro_oracle_step.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_double,
                                        ctypes.POINTER(Rule),
                                        ctypes.POINTER(ctypes.c_double),
                                        ctypes.c_void_p, ctypes.c_void_p, i64p]
        L.micro_oracle_step.restype = ctypes.c_int
        L.micro_oracle_cycle.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32]
        L.micro_oracle_cycle.restype = ctypes.c_int32
        L.micro_oracle_ef_step.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_double, ctypes.POINTER(Rule),
                                           ctypes.POINTER(ctypes.c_double),
                                           ctypes.c_void_p, ctypes.c_void_p, i64p,
                                           ctypes.POINTER(ctypes.c_int32)]
        L.micro_oracle_ef_step.restype = ctypes.c_int
        L.micro_oracle_accumulate.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int64, ctypes.c_void_p]
        L.micro_oracle_accumulate.restype = None
        L.micro_oracle_gather.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_int64, ctypes.c_void_p]
        L.micro_oracle_gather.restype = None
        L.micro_oracle_zero.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
        L.micro_oracle_zero.restype = None
        L.micro_oracle_update.argtypes = [ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_int32]
        L.micro_oracle_update.restype = ctypes.c_int
        L.micro_oracle_sumsq.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64]
        L.micro_oracle_sumsq.restype = ctypes.c_double
        L.micro_oracle_sweep.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int32, ctypes.c_double, ctypes.POINTER(Rule),
                                         ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_void_p]
        L.micro_oracle_sweep.restype = ctypes.c_int
        L.micro_oracle_topk_count.argtypes = [ctypes.c_double, ctypes.c_int64]
        L.micro_oracle_topk_count.restype = ctypes.c_int64
        L.micro_oracle_topk_select.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                               ctypes.c_int64, ctypes.c_double, ctypes.c_void_p,
                                               ctypes.c_void_p, i64p, ctypes.POINTER(ctypes.c_double)]
        L.micro_oracle_topk_select.restype = ctypes.c_int
        _lib = L
    return _lib


def default_rule():
    r = Rule()
    lib().micro_oracle_default_rule(ctypes.byref(r))
    return r


def make_rule(kind=PROPORTIONAL, beta=None, lo=None, hi=None, alpha=None):
    r = default_rule()
    r.kind = kind
    if beta is not None:
        r.beta = beta
    if lo is not None:
        r.lo = lo
    if hi is not None:
        r.hi = hi
    if alpha is not None:
        r.alpha = alpha
    return r


def partition(n_total, rank, world):
    """Sec. 4.1 partition bounds; returns (start, length)."""
    s, n = ctypes.c_int64(), ctypes.c_int64()
    rc = lib().micro_oracle_partition(n_total, rank, world, ctypes.byref(s),
                                      ctypes.byref(n))
    if rc != 0:
        raise ValueError("invalid partition arguments")
    return s.value, n.value


def _f32(a, name):
    if not (isinstance(a, np.ndarray) and a.dtype == np.float32
            and a.flags.c_contiguous):
        raise TypeError(f"{name} must be a C-contiguous float32 numpy array")
    return a


def select(grad, residual, start, length, theta):
    """Sec. 4.2 selection over [start, start+length); residual is updated in
    place.  Returns (idx int32[k], val float32[k])."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    if start < 0 or length < 0 or start + length > min(grad.size, residual.size):
        raise ValueError("range outside the arrays")
    out_idx = np.empty(max(length, 1), dtype=np.int32)
    out_val = np.empty(max(length, 1), dtype=np.float32)
    k = lib().micro_oracle_select(grad.ctypes.data, residual.ctypes.data, start,
                                  length, float(theta), out_idx.ctypes.data,
                                  out_val.ctypes.data)
    return out_idx[:k].copy(), out_val[:k].copy()


def estimate(density, part_len, k, theta, rule=None):
    """Sec. 4.3 threshold update; returns the next threshold (a Python float)."""
    r = rule if rule is not None else default_rule()
    return lib().micro_oracle_estimate(ctypes.byref(r), float(density),
                                       int(part_len), int(k), float(theta))


def step(grad, residual, rank, world, density, theta, rule=None, out=None):
    """One worker, one iteration.  residual (full length) is updated in place.
    Returns (idx, val, k, theta_next); idx/val are views into `out` buffers
    (allocated here when `out` is None) of length k."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    n_total = grad.size
    if residual.size != n_total:
        raise ValueError("grad and residual lengths differ")
    _, length = partition(n_total, rank, world)
    if out is None:
        out = (np.empty(max(length, 1), np.int32), np.empty(max(length, 1), np.float32))
    out_idx, out_val = out
    if out_idx.size < length or out_val.size < length:
        raise ValueError("output buffers smaller than the partition")
    r = rule if rule is not None else default_rule()
    th = ctypes.c_double(float(theta))
    k = ctypes.c_int64()
    rc = lib().micro_oracle_step(grad.ctypes.data, residual.ctypes.data, n_total,
                                 rank, world, float(density), ctypes.byref(r),
                                 ctypes.byref(th), out_idx.ctypes.data,
                                 out_val.ctypes.data, ctypes.byref(k))
    if rc != 0:
        raise ValueError("invalid oracle step arguments")
    return out_idx[:k.value], out_val[:k.value], k.value, th.value


def cycle(t, worker, world):
    """Algorithm 1's partition number of `worker` at iteration t."""
    c = lib().micro_oracle_cycle(int(t), int(worker), int(world))
    if c < 0:
        raise ValueError("invalid cycle arguments")
    return c


def ef_step(grad, residual, t, worker, world, density, theta, rule=None, out=None):
    """Algorithm 1 for one worker over the whole vector: every element
    accumulates, only the partition of the worker's cycle is searched.
    residual is updated in place.  Returns (idx, val, k, theta_next, cycle)."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    n_total = grad.size
    if residual.size != n_total:
        raise ValueError("grad and residual lengths differ")
    _, length = partition(n_total, cycle(t, worker, world), world)
    if out is None:
        out = (np.empty(max(length, 1), np.int32), np.empty(max(length, 1), np.float32))
    out_idx, out_val = out
    if out_idx.size < length or out_val.size < length:
        raise ValueError("output buffers smaller than the partition")
    r = rule if rule is not None else default_rule()
    th = ctypes.c_double(float(theta))
    k = ctypes.c_int64()
    c = ctypes.c_int32()
    rc = lib().micro_oracle_ef_step(grad.ctypes.data, residual.ctypes.data, n_total,
                                    int(t), worker, world, float(density), ctypes.byref(r),
                                    ctypes.byref(th), out_idx.ctypes.data,
                                    out_val.ctypes.data, ctypes.byref(k), ctypes.byref(c))
    if rc != 0:
        raise ValueError("invalid oracle EF step arguments")
    return out_idx[:k.value], out_val[:k.value], k.value, th.value, c.value


def _i32(a, name):
    if not (isinstance(a, np.ndarray) and a.dtype == np.int32 and a.flags.c_contiguous):
        raise TypeError(f"{name} must be a C-contiguous int32 numpy array")
    return a


def accumulate(grad, residual):
    """Algorithm 1's accumulation: returns grad + residual (binary32)."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    if grad.size != residual.size:
        raise ValueError("grad and residual lengths differ")
    acc = np.empty(grad.size, np.float32)
    lib().micro_oracle_accumulate(grad.ctypes.data, residual.ctypes.data, grad.size,
                                  acc.ctypes.data)
    return acc


def _check_idx(idx, n):
    _i32(idx, "idx")
    if idx.size and (idx.min() < 0 or idx.max() >= n):
        raise ValueError("index outside the vector")


def gather(acc, idx):
    """Algorithm 1's gathering: returns acc[idx]."""
    _f32(acc, "acc")
    _check_idx(idx, acc.size)
    out = np.empty(max(idx.size, 1), np.float32)
    lib().micro_oracle_gather(acc.ctypes.data, idx.ctypes.data, idx.size, out.ctypes.data)
    return out[:idx.size].copy()


def zero(acc, idx):
    """Algorithm 1's reset: acc[idx] = +0 in place."""
    _f32(acc, "acc")
    _check_idx(idx, acc.size)
    lib().micro_oracle_zero(acc.ctypes.data, idx.ctypes.data, idx.size)


def update(x, idx, sums, world):
    """Algorithm 1's model update: x[idx] -= sums / world in place (indices
    distinct)."""
    _f32(x, "x")
    _f32(sums, "sums")
    _check_idx(idx, x.size)
    if sums.size != idx.size:
        raise ValueError("sums and idx lengths differ")
    if lib().micro_oracle_update(x.ctypes.data, idx.ctypes.data, sums.ctypes.data,
                                 idx.size, int(world)) != 0:
        raise ValueError("world must be >= 1")


def sumsq(residual, start=0, length=None):
    """Squared L2 norm of residual[start:start+length] (binary64, index order)."""
    _f32(residual, "residual")
    if length is None:
        length = residual.size - start
    if start < 0 or length < 0 or start + length > residual.size:
        raise ValueError("range outside the array")
    return lib().micro_oracle_sumsq(residual.ctypes.data, int(start), int(length))


def sweep(grad, residual, world, density, thetas, rule=None):
    """Every partition of the vector searched once with its own threshold.
    residual is updated in place.  Returns (idx, val, k[world], thetas_next,
    sumsq[world]); idx/val are the partitions' selections concatenated in
    index order."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    n_total = grad.size
    if residual.size != n_total:
        raise ValueError("grad and residual lengths differ")
    th = np.ascontiguousarray(np.asarray(thetas, dtype=np.float64).copy())
    if th.size != world:
        raise ValueError("one threshold per partition")
    out_idx = np.empty(max(n_total, 1), np.int32)
    out_val = np.empty(max(n_total, 1), np.float32)
    k = np.zeros(max(world, 1), np.int64)
    sq = np.zeros(max(world, 1), np.float64)
    r = rule if rule is not None else default_rule()
    rc = lib().micro_oracle_sweep(grad.ctypes.data, residual.ctypes.data, n_total, int(world),
                                  float(density), ctypes.byref(r), th.ctypes.data,
                                  out_idx.ctypes.data, out_val.ctypes.data, k.ctypes.data,
                                  sq.ctypes.data)
    if rc != 0:
        raise ValueError("invalid oracle sweep arguments")
    total = int(k[:world].sum())
    return out_idx[:total], out_val[:total], k[:world].copy(), th, sq[:world].copy()


def topk_count(density, length):
    """k of the exact top-k comparator over `length` values:
    max(1, floor(density * length)), at most length (0 for length 0)."""
    return lib().micro_oracle_topk_count(float(density), int(length))


def topk_select(grad, residual, start, length, density, kth=float("nan")):
    """The exact top-k comparator over [start, start+length): the k largest
    accumulated magnitudes (equal magnitudes by lower index, NaN never), in
    index order.  residual is updated in place.  Returns (idx, val, k, kth):
    kth is the smallest selected magnitude, or the given kth when nothing is
    selected."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    if start < 0 or length < 0 or start + length > min(grad.size, residual.size):
        raise ValueError("range outside the arrays")
    out_idx = np.empty(max(length, 1), dtype=np.int32)
    out_val = np.empty(max(length, 1), dtype=np.float32)
    k = ctypes.c_int64()
    th = ctypes.c_double(float(kth))
    rc = lib().micro_oracle_topk_select(grad.ctypes.data, residual.ctypes.data, int(start), int(length),
                                        float(density), out_idx.ctypes.data, out_val.ctypes.data,
                                        ctypes.byref(k), ctypes.byref(th))
    if rc != 0:
        raise ValueError("invalid oracle top-k arguments")
    return out_idx[:k.value].copy(), out_val[:k.value].copy(), k.value, th.value


def topk_step(grad, residual, rank, world, density, theta):
    """The top-k comparator as one worker's step over its partition: returns
    (idx, val, k, theta_next), theta_next the smallest selected magnitude (theta
    unchanged when nothing is selected)."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    if residual.size != grad.size:
        raise ValueError("grad and residual lengths differ")
    start, length = partition(grad.size, rank, world)
    return topk_select(grad, residual, start, length, density, kth=theta)


def topk_ef_step(grad, residual, t, worker, world, density, theta):
    """Algorithm 1's pass with the top-k comparator in place of the threshold
    rule: every element outside the worker's partition of iteration t
    accumulates (residual = grad + residual), the partition goes through
    topk_select.  Returns (idx, val, k, theta_next, cycle)."""
    _f32(grad, "grad")
    _f32(residual, "residual")
    n_total = grad.size
    if residual.size != n_total:
        raise ValueError("grad and residual lengths differ")
    c = cycle(t, worker, world)
    start, length = partition(n_total, c, world)
    for lo, hi in ((0, start), (start + length, n_total)):
        if hi > lo:
            lib().micro_oracle_accumulate(grad.ctypes.data + 4 * lo, residual.ctypes.data + 4 * lo,
                                          hi - lo, residual.ctypes.data + 4 * lo)
    idx, val, k, th = topk_select(grad, residual, start, length, density, kth=theta)
    return idx, val, k, th, c
