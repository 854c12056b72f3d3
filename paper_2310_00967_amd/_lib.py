"""ctypes binding of the C ABI in include/micro_sparsify.h.

Argument marshalling only: every step of the sparsify path runs in the HIP
library.  The functions below carry the C names; Python callers normally use
paper_2310_00967_amd.Sparsifier.  Loading fails loudly when the library has
not been built.
"""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmicro_sparsify.so")

MICRO_OK, MICRO_EINVAL, MICRO_ECAPACITY, MICRO_ERANGE, MICRO_ENOMEM, MICRO_EHIP = range(6)
MICRO_RULE_PROPORTIONAL, MICRO_RULE_FIXED_STEP, MICRO_RULE_HARD_THRESHOLD, MICRO_RULE_TOPK = 0, 1, 2, 3
MICRO_VARIANT_AUTO, MICRO_VARIANT_TICKET, MICRO_VARIANT_STAGED = 0, 1, 2
MICRO_FLAG_TIME_KERNEL = 1
MICRO_FLAG_SEPARATE_SCAN = 2
MICRO_TOPK_ROUTE_FULL, MICRO_TOPK_ROUTE_LIST, MICRO_TOPK_ROUTE_HINT_LIST, MICRO_TOPK_ROUTE_HINT_PICK = 1, 2, 3, 4

# Every function the header declares, with (restype, argtypes).
_i64p = ctypes.POINTER(ctypes.c_int64)
_dblp = ctypes.POINTER(ctypes.c_double)
_fltp = ctypes.POINTER(ctypes.c_float)


class micro_config(ctypes.Structure):
    _fields_ = [("rule", ctypes.c_int32), ("beta", ctypes.c_double), ("lo", ctypes.c_double),
                ("hi", ctypes.c_double), ("alpha", ctypes.c_double), ("variant", ctypes.c_int32),
                ("flags", ctypes.c_int32)]


class micro_step_stats(ctypes.Structure):
    _fields_ = [("kernel_ms", ctypes.c_float), ("redone_tiles", ctypes.c_int64),
                ("variant", ctypes.c_int32), ("fused", ctypes.c_int32), ("topk_route", ctypes.c_int32)]


_cfgp = ctypes.POINTER(micro_config)

SIGNATURES = {
    "micro_config_default": (None, [_cfgp]),
    "micro_sparsify_init": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int64,
                                           ctypes.c_void_p, _cfgp]),
    "micro_sparsify_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_int32, ctypes.c_int32, ctypes.c_double, _dblp,
                                           ctypes.c_void_p, ctypes.c_void_p, _i64p]),
    "micro_sparsify_step_noalloc": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                                   ctypes.c_int32, ctypes.c_int32, ctypes.c_double, _dblp,
                                                   ctypes.c_void_p, ctypes.c_void_p, _i64p, ctypes.c_void_p,
                                                   _cfgp]),
    "micro_partition": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _i64p, _i64p]),
    "micro_sweep_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                        ctypes.c_double, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p]),
    "micro_cycle": (ctypes.c_int, [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
    "micro_ef_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                     ctypes.c_int32, ctypes.c_int32, ctypes.c_double, _dblp,
                                     ctypes.c_void_p, ctypes.c_void_p, _i64p, ctypes.POINTER(ctypes.c_int32),
                                     _dblp]),
    "micro_union_gather": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]),
    "micro_sparse_update": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_int64, ctypes.c_int32]),
    "micro_estimate_threshold": (ctypes.c_int, [_cfgp, ctypes.c_double, ctypes.c_int64,
                                                ctypes.c_int64, _dblp]),
    "micro_threshold_f32": (ctypes.c_int, [ctypes.c_double, _fltp]),
    "micro_sparsify_last_stats": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(micro_step_stats)]),
    "micro_last_error": (ctypes.c_char_p, [ctypes.c_void_p]),
    "micro_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "micro_sparsify_free": (None, [ctypes.c_void_p]),
}

_lib = None


class MicroError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


def load():
    """Loads the built HIP library (never builds it; never falls back)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build() "
                               "or python -m paper_2310_00967_amd.build")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def status_string(status):
    return load().micro_status_string(int(status)).decode()


def last_error(ctx=None):
    return load().micro_last_error(ctx).decode()


def check(status, ctx=None):
    if status != MICRO_OK:
        raise MicroError(status, last_error(ctx))


def default_config():
    c = micro_config()
    load().micro_config_default(ctypes.byref(c))
    return c


def micro_partition(n_total, rank, world):
    s, n = ctypes.c_int64(), ctypes.c_int64()
    check(load().micro_partition(int(n_total), int(rank), int(world), ctypes.byref(s), ctypes.byref(n)))
    return s.value, n.value


def micro_estimate_threshold(density, part_len, k, theta, cfg=None):
    th = ctypes.c_double(float(theta))
    check(load().micro_estimate_threshold(ctypes.byref(cfg) if cfg is not None else None,
                                          float(density), int(part_len), int(k), ctypes.byref(th)))
    return th.value


def micro_threshold_f32(theta):
    f = ctypes.c_float()
    check(load().micro_threshold_f32(float(theta), ctypes.byref(f)))
    return f.value


def micro_sparsify_init(n_total, stream_handle=None, cfg=None):
    ctx = ctypes.c_void_p()
    st = load().micro_sparsify_init(ctypes.byref(ctx), int(n_total),
                                    ctypes.c_void_p(stream_handle or 0),
                                    ctypes.byref(cfg) if cfg is not None else None)
    check(st)
    return ctx


def micro_sparsify_step(ctx, grad_ptr, residual_ptr, rank, world, density, theta,
                        out_idx_ptr, out_val_ptr):
    """Raw call with device addresses; returns (k, theta_next)."""
    th = ctypes.c_double(float(theta))
    k = ctypes.c_int64()
    st = load().micro_sparsify_step(ctx, ctypes.c_void_p(grad_ptr), ctypes.c_void_p(residual_ptr),
                                    int(rank), int(world), float(density), ctypes.byref(th),
                                    ctypes.c_void_p(out_idx_ptr), ctypes.c_void_p(out_val_ptr),
                                    ctypes.byref(k))
    check(st, ctx)
    return k.value, th.value


def micro_sparsify_step_noalloc(grad_ptr, residual_ptr, n_total, rank, world, density, theta, out_idx_ptr,
                                out_val_ptr, stream_handle=None, cfg=None):
    """Raw call of the allocation-free step with device addresses on the
    current device; returns (k, theta_next)."""
    th = ctypes.c_double(float(theta))
    k = ctypes.c_int64()
    st = load().micro_sparsify_step_noalloc(ctypes.c_void_p(grad_ptr), ctypes.c_void_p(residual_ptr),
                                            int(n_total), int(rank), int(world), float(density),
                                            ctypes.byref(th), ctypes.c_void_p(out_idx_ptr),
                                            ctypes.c_void_p(out_val_ptr), ctypes.byref(k),
                                            ctypes.c_void_p(stream_handle or 0),
                                            ctypes.byref(cfg) if cfg is not None else None)
    check(st)
    return k.value, th.value


MICRO_MAX_SWEEP = 64


def micro_sweep_step(ctx, grad_ptr, residual_ptr, world, density, thetas, out_idx_ptr, out_val_ptr,
                     want_sumsq=True):
    """Raw call with device addresses; returns (k list, thetas_next list,
    sumsq list or None)."""
    world = int(world)
    th = (ctypes.c_double * max(1, world))(*[float(x) for x in thetas])
    k = (ctypes.c_int64 * max(1, world))()
    sq = (ctypes.c_double * max(1, world))() if want_sumsq else None
    st = load().micro_sweep_step(ctx, ctypes.c_void_p(grad_ptr), ctypes.c_void_p(residual_ptr), world,
                                 float(density), ctypes.cast(th, ctypes.c_void_p),
                                 ctypes.c_void_p(out_idx_ptr), ctypes.c_void_p(out_val_ptr),
                                 ctypes.cast(k, ctypes.c_void_p),
                                 ctypes.cast(sq, ctypes.c_void_p) if sq is not None else None)
    check(st, ctx)
    return list(k[:world]), list(th[:world]), (list(sq[:world]) if sq is not None else None)


def micro_cycle(t, worker, world):
    c = ctypes.c_int32()
    check(load().micro_cycle(int(t), int(worker), int(world), ctypes.byref(c)))
    return c.value


def micro_ef_step(ctx, grad_ptr, residual_ptr, t, worker, world, density, theta, out_idx_ptr, out_val_ptr,
                  want_sumsq=False):
    """Raw call with device addresses; returns (k, theta_next, cycle, sumsq
    or None)."""
    th = ctypes.c_double(float(theta))
    k = ctypes.c_int64()
    c = ctypes.c_int32()
    sq = ctypes.c_double(-1.0)
    st = load().micro_ef_step(ctx, ctypes.c_void_p(grad_ptr), ctypes.c_void_p(residual_ptr), int(t),
                              int(worker), int(world), float(density), ctypes.byref(th),
                              ctypes.c_void_p(out_idx_ptr), ctypes.c_void_p(out_val_ptr), ctypes.byref(k),
                              ctypes.byref(c), ctypes.byref(sq) if want_sumsq else None)
    check(st, ctx)
    return k.value, th.value, c.value, (sq.value if want_sumsq else None)


def micro_union_gather(ctx, residual_ptr, union_ptr, m, own_first, own_count, own_val_ptr, out_ptr):
    check(load().micro_union_gather(ctx, ctypes.c_void_p(residual_ptr), ctypes.c_void_p(union_ptr), int(m),
                                    int(own_first), int(own_count), ctypes.c_void_p(own_val_ptr),
                                    ctypes.c_void_p(out_ptr)), ctx)


def micro_sparse_update(ctx, x_ptr, union_ptr, sums_ptr, m, world):
    check(load().micro_sparse_update(ctx, ctypes.c_void_p(x_ptr), ctypes.c_void_p(union_ptr),
                                     ctypes.c_void_p(sums_ptr), int(m), int(world)), ctx)


def micro_sparsify_last_stats(ctx):
    st = micro_step_stats()
    check(load().micro_sparsify_last_stats(ctx, ctypes.byref(st)), ctx)
    return st


def micro_sparsify_free(ctx):
    load().micro_sparsify_free(ctx)
