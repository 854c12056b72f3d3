"""Runs the HIP path and the CPU oracle side by side on identical inputs.

Test infrastructure (not collected by pytest).  The oracle follows its own
trajectory on a host mirror of the residual; after every call the GPU's
indices, values, selected count, next threshold and the residual are compared
with the oracle's bit for bit.
"""
import concurrent.futures as cf
import sys

import numpy as np
import torch

import oracle
import paper_2310_00967_amd as micro
from paper_2310_00967_amd import synth

_POOL = cf.ThreadPoolExecutor(max_workers=8)
_CHUNK = 1 << 24


def first_mismatch(a, b):
    """Index of the first bitwise difference between two equal-length 4-byte
    arrays (chunked over threads), or -1."""
    a = a.view(np.uint32)
    b = b.view(np.uint32)
    if a.shape != b.shape:
        return 0
    n = a.size
    starts = list(range(0, n, _CHUNK))

    def chunk(s):
        e = min(n, s + _CHUNK)
        if np.array_equal(a[s:e], b[s:e]):
            return -1
        return s + int(np.flatnonzero(a[s:e] != b[s:e])[0])

    for r in _POOL.map(chunk, starts):
        if r >= 0:
            return r
    return -1


def note(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class ParityRun:
    """Keeps the device buffers, the host mirror and the per-rank thresholds
    of one workload and checks each step."""

    def __init__(self, w, density, device="cuda", rule_kind=oracle.PROPORTIONAL,
                 variant=micro.MICRO_VARIANT_AUTO, separate_scan=False, expect_schedule=None):
        # expect_schedule: the schedule every call must report having run
        # (MICRO_VARIANT_TICKET or MICRO_VARIANT_STAGED), or None
        self.expect_schedule = expect_schedule
        self.w = w
        self.d = density
        self.N = w.n_total
        self.dev = torch.device(device)
        # rule_kind: oracle.PROPORTIONAL, oracle.FIXED_STEP or "hard" (the
        # library's hard-threshold rule against the oracle's zero fixed step)
        lib_rule = {oracle.PROPORTIONAL: micro.MICRO_RULE_PROPORTIONAL, oracle.FIXED_STEP: micro.MICRO_RULE_FIXED_STEP,
                    "hard": micro.MICRO_RULE_HARD_THRESHOLD}[rule_kind]
        self.sp = micro.Sparsifier(self.N, device=self.dev, rule=lib_rule, variant=variant,
                                   separate_scan=separate_scan)
        self.rule = (oracle.make_rule(oracle.FIXED_STEP, alpha=0.0) if rule_kind == "hard"
                     else oracle.make_rule(rule_kind))
        self.res_dev = torch.zeros(self.N, dtype=torch.float32, device=self.dev)
        self.g_dev = torch.empty(self.N, dtype=torch.float32, device=self.dev)
        pin = torch.cuda.is_available()
        self.g_host = torch.empty(self.N, dtype=torch.float32, pin_memory=pin)
        self.res_gpu_host = torch.empty(self.N, dtype=torch.float32, pin_memory=pin)
        self.res_mirror = np.zeros(self.N, np.float32)
        self.bounds = {r: oracle.partition(self.N, r, w.world) for r in w.ranks}
        maxlen = max(ln for _, ln in self.bounds.values())
        self.o_idx = np.empty(max(1, maxlen), np.int32)
        self.o_val = np.empty(max(1, maxlen), np.float32)
        self.thetas = None
        self.errors = []

    def load_gradient(self, t):
        synth.gradient(self.w, t, self.dev, out=self.g_dev)

    def init_thresholds(self):
        self.thetas = {}
        for r, (s, ln) in self.bounds.items():
            self.thetas[r] = synth.initial_theta(self.w, self.g_dev, s, s + ln, self.d)
        self.thetas0 = dict(self.thetas)

    def check_rank(self, t, r):
        s, ln = self.bounds[r]
        w = self.w
        th = self.thetas[r]
        # same g bytes for the oracle
        self.g_host[s:s + ln].copy_(self.g_dev[s:s + ln])
        g_np = self.g_host.numpy()
        k_gpu, th_gpu, idx_gpu, val_gpu = self.sp.step(self.g_dev, self.res_dev, r, w.world, self.d, th)
        idx_gpu = idx_gpu.cpu().numpy()
        val_gpu = val_gpu.cpu().numpy()
        self.res_gpu_host[s:s + ln].copy_(self.res_dev[s:s + ln])
        o_idx, o_val, k_or, th_or = oracle.step(g_np, self.res_mirror, r, w.world, self.d, th,
                                                rule=self.rule, out=(self.o_idx, self.o_val))
        where = f"{w.name} d={self.d} step {t} rank {r}"
        if self.expect_schedule is not None:
            ran = self.sp.last_stats()[2]
            assert ran == self.expect_schedule, f"{where}: schedule {ran}, expected {self.expect_schedule}"
        assert k_gpu == k_or, f"{where}: k gpu {k_gpu} oracle {k_or}"
        assert th_gpu == th_or, f"{where}: theta gpu {th_gpu!r} oracle {th_or!r}"
        assert np.array_equal(idx_gpu, o_idx), f"{where}: indices differ"
        assert first_mismatch(val_gpu, o_val) < 0, f"{where}: values differ"
        mm = first_mismatch(self.res_gpu_host.numpy()[s:s + ln], self.res_mirror[s:s + ln])
        assert mm < 0, f"{where}: residual differs at {s + mm}"
        self.thetas[r] = th_or
        self.errors.append(abs(k_or / ln - self.d) / self.d if ln else 0.0)
        return k_or

    def run(self, steps, verbose=True):
        for t in range(steps):
            self.load_gradient(t)
            if t == 0:
                self.init_thresholds()
            for r in self.w.ranks:
                self.check_rank(t, r)
            if verbose and (t % 10 == 0 or t == steps - 1):
                note(f"  {self.w.name} d={self.d}: step {t} ok")
        # the residual outside the swept partitions never changes
        covered = np.zeros(self.N, bool)
        for s, ln in self.bounds.values():
            covered[s:s + ln] = True
        if not covered.all():
            outside = self.res_dev.cpu().numpy()[~covered]
            assert not np.any(outside.view(np.uint32)), "residual outside the partitions was written"

    def close(self):
        self.sp.close()
