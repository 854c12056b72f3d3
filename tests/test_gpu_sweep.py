"""The sweep of every partition in one set of launches (GPU): bit-exact
pairs, counts, thresholds and residual against the oracle's sweep, and the
partitions' local-error squared norms within the bound that any binary64
summation order of nonnegative terms satisfies."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2310_00967_amd as micro
from paper_2310_00967_amd import _lib, synth

from gpu_harness import first_mismatch, note

pytestmark = pytest.mark.gpu

DEV = "cuda"
U = 2.0 ** -53


def sumsq_tolerance(n, ref):
    """Both sides are within gamma_{n-1} * exact of the exact sum."""
    g = max(n - 1, 0) * U
    return 2.0 * g / (1.0 - 2.0 * g) * abs(ref) * 1.01


def check_sweep(g, res, world, density, thetas, phase_shift=0, sp=None, where=""):
    """One sweep on both sides from host arrays; returns the new thresholds."""
    N = g.size
    own = sp is None
    if own:
        sp = micro.Sparsifier(N, device=DEV)
    gbuf = torch.empty(N + 4, dtype=torch.float32, device=DEV)
    g_dev = gbuf[phase_shift:phase_shift + N]
    g_dev.copy_(torch.from_numpy(g))
    r_dev = torch.from_numpy(res).to(DEV)
    out_idx = torch.full((max(1, N) + 8,), -5, dtype=torch.int32, device=DEV)
    out_val = torch.full((max(1, N) + 8,), -5.0, dtype=torch.float32, device=DEV)
    k, th, sq, idx, val = sp.sweep(g_dev, r_dev, world, density, thetas, out_idx, out_val)
    r_or = res.copy()
    o_idx, o_val, k_or, th_or, sq_or = oracle.sweep(g, r_or, world, density, thetas)
    assert k == list(k_or), where
    assert th == list(th_or), where
    assert np.array_equal(idx.cpu().numpy(), o_idx), where
    v = val.cpu().numpy()
    assert first_mismatch(np.ascontiguousarray(v), np.ascontiguousarray(o_val)) < 0, where
    assert first_mismatch(r_dev.cpu().numpy(), r_or) < 0, where
    assert bool((out_idx[sum(k):] == -5).all()), where
    for r in range(world):
        _, ln = oracle.partition(N, r, world)
        if np.isnan(sq_or[r]):
            assert np.isnan(sq[r]), where
        else:
            assert abs(sq[r] - sq_or[r]) <= sumsq_tolerance(ln, sq_or[r]), (where, r, sq[r], sq_or[r])
    if own:
        sp.close()
    return th


@pytest.mark.parametrize("name,density,steps", [
    ("toy", 0.01, 20),
    ("resnet18", 0.01, 100),
    ("resnet50", 0.001, 20),
    ("bert_large", 0.01, 5),
])
def test_sweep_workload_parity(name, density, steps):
    """All partitions of the workload each step, from the calibrated
    thresholds, on one residual carried across steps."""
    w = synth.get(name)
    N = w.n_total
    note(f"sweep parity {name} world {w.world} steps {steps}")
    sp = micro.Sparsifier(N, device=DEV)
    g_dev = torch.empty(N, dtype=torch.float32, device=DEV)
    res_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    g_host = torch.empty(N, dtype=torch.float32, pin_memory=True)
    r_host = torch.empty(N, dtype=torch.float32, pin_memory=True)
    mirror = np.zeros(N, np.float32)
    thetas = None
    try:
        for t in range(steps):
            synth.gradient(w, t, DEV, out=g_dev)
            if thetas is None:
                thetas = []
                for r in range(w.world):
                    s, ln = oracle.partition(N, r, w.world)
                    thetas.append(synth.initial_theta(w, g_dev, s, s + ln, density))
            g_host.copy_(g_dev)
            k, th, sq, idx, val = sp.sweep(g_dev, res_dev, w.world, density, thetas)
            o_idx, o_val, k_or, th_or, sq_or = oracle.sweep(g_host.numpy(), mirror, w.world, density, thetas)
            where = f"{name} step {t}"
            assert k == list(k_or) and th == list(th_or), where
            assert np.array_equal(idx.cpu().numpy(), o_idx), where
            assert first_mismatch(val.cpu().numpy(), o_val) < 0, where
            r_host.copy_(res_dev)
            assert first_mismatch(r_host.numpy(), mirror) < 0, where
            for r in range(w.world):
                _, ln = oracle.partition(N, r, w.world)
                assert abs(sq[r] - sq_or[r]) <= sumsq_tolerance(ln, sq_or[r]), (where, r)
            thetas = list(th_or)
    finally:
        sp.close()


@pytest.mark.parametrize("phase_shift", [0, 2])
@pytest.mark.parametrize("N,world", [(1, 1), (5, 8), (1023, 3), (4099, 64), (70_001, 7),
                                     (1_100_003, 16), (3_000_017, 64)])
def test_sweep_ragged_sizes_worlds_and_phases(N, world, phase_shift):
    rng = np.random.default_rng(N + world + phase_shift)
    g = (rng.standard_normal(N) * np.exp(rng.uniform(-1.5, 1.5, N))).astype(np.float32)
    res = (rng.standard_normal(N) * 0.4).astype(np.float32)
    thetas = list(np.exp(rng.uniform(0.0, 1.2, world)))
    check_sweep(g, res, world, 0.02, thetas, phase_shift, where=f"N={N} world={world}")


@pytest.mark.parametrize("seed", range(24))
def test_sweep_fuzz(seed):
    """Random vector lengths up to 3M, worlds up to 64 (segments of every
    size, empty ones included), thresholds per partition spread over two
    decades (from near-empty to dense selections), densities and phases."""
    rng = np.random.default_rng(5000 + seed)
    N = int(rng.integers(1, 3_000_000))
    world = int(rng.integers(1, 65))
    g = (rng.standard_normal(N) * np.exp(rng.uniform(-1.5, 1.5, N))).astype(np.float32)
    res = (rng.standard_normal(N) * rng.uniform(0.0, 1.0)).astype(np.float32)
    thetas = list(np.exp(rng.uniform(-1.5, 3.0, world)))
    density = float(rng.choice([0.001, 0.01, 0.1]))
    phase = int(rng.integers(0, 4))
    note(f"sweep fuzz seed {seed}: N={N} world={world} d={density} phase {phase}")
    check_sweep(g, res, world, density, thetas, phase, where=f"seed {seed} N={N} world={world}")


def test_sweep_dense_partitions_and_specials():
    """Some partitions select almost everything (tiles redone by the move
    kernel inside several segments), one holds NaN (its norm is NaN), one
    infinities."""
    N, world = 2_500_000, 5
    rng = np.random.default_rng(5)
    g = rng.standard_normal(N).astype(np.float32)
    res = np.zeros(N, np.float32)
    g[1_000_100] = np.nan
    g[2_300_000] = np.inf
    thetas = [1e-3, 3.0, 1e-30, 2.0, 0.5]
    check_sweep(g, res, world, 0.01, thetas, where="dense")


@pytest.mark.parametrize("N,world,fused_default", [(1_100_003, 16, 1), (40_000_019, 3, 1), (23_000_001, 9, 1),
                                                   (70_000_003, 5, 0)])
def test_sweep_fused_and_separate_launches_agree(N, world, fused_default):
    """A sweep of up to 64 scan chunks runs its stream and scan passes as one
    launch by default (each segment laid out like a single partition's fused
    launch, stats fused = 1), a larger one apart, and MICRO_FLAG_SEPARATE_SCAN
    always apart.  Both give the oracle's pairs, counts, thresholds and
    residual, and its norms within the bound; the sizes give segments of one
    to fourteen chunks, so scan workgroups are interleaved among a segment's
    tiles, and a dense region overflows tiles."""
    rng = np.random.default_rng(N % 997 + world)
    g = (rng.standard_normal(N) * np.exp(rng.uniform(-1.0, 1.0, N))).astype(np.float32)
    g[N // 2:N // 2 + 200_000] *= 40.0
    res = (rng.standard_normal(N) * 0.3).astype(np.float32)
    thetas = list(np.exp(rng.uniform(0.5, 1.2, world)))
    for separate in (False, True):
        note(f"sweep fused/separate N={N} world={world} separate={separate}")
        sp = micro.Sparsifier(N, device=DEV, separate_scan=separate)
        check_sweep(g, res, world, 0.01, thetas, sp=sp, where=f"N={N} world={world} separate={separate}")
        _, redone, variant, fused = sp.last_stats()
        assert fused == (0 if separate else fused_default) and redone > 0
        sp.close()


def test_sweep_equals_separate_steps():
    N, world = 4_000_037, 12
    rng = np.random.default_rng(9)
    g = torch.from_numpy(rng.standard_normal(N).astype(np.float32)).to(DEV)
    res0 = torch.from_numpy((rng.standard_normal(N) * 0.5).astype(np.float32)).to(DEV)
    thetas = [1.5 + 0.1 * r for r in range(world)]
    sp = micro.Sparsifier(N, device=DEV)
    r1 = res0.clone()
    k, th, sq, idx, val = sp.sweep(g, r1, world, 0.01, thetas)
    idx, val = idx.clone(), val.clone()
    r2 = res0.clone()
    pos = 0
    for r in range(world):
        kr, thr, ir, vr = sp.step(g, r2, r, world, 0.01, thetas[r])
        assert (kr, thr) == (k[r], th[r])
        assert torch.equal(ir, idx[pos:pos + kr]) and torch.equal(vr.view(torch.int32), val[pos:pos + kr].view(torch.int32))
        pos += kr
    assert torch.equal(r1.view(torch.int32), r2.view(torch.int32))
    sp.close()


def test_sweep_validation():
    N = 1000
    sp = micro.Sparsifier(N, device=DEV)
    lib = _lib.load()
    g = torch.randn(N, device=DEV)
    r = torch.randn(N, device=DEV)
    r0 = r.clone()
    oi = torch.full((N,), -1, dtype=torch.int32, device=DEV)
    ov = torch.full((N,), -1.0, device=DEV)

    def call(world, thetas, res=r.data_ptr(), idx=oi.data_ptr()):
        th = (ctypes.c_double * max(1, len(thetas)))(*thetas)
        k = (ctypes.c_int64 * 70)(*([-7] * 70))
        return lib.micro_sweep_step(sp._ctx, ctypes.c_void_p(g.data_ptr()), ctypes.c_void_p(res), world, 0.1,
                                    ctypes.cast(th, ctypes.c_void_p), ctypes.c_void_p(idx),
                                    ctypes.c_void_p(ov.data_ptr()), ctypes.cast(k, ctypes.c_void_p), None), k

    for world, thetas, kw in [(0, [1.0], {}), (65, [1.0] * 65, {}), (2, [1.0, 0.0], {}),
                              (2, [1.0, float("inf")], {}), (2, [1.0, 1.0], dict(res=g.data_ptr() + 400)),
                              (2, [1.0, 1.0], dict(idx=r.data_ptr()))]:
        st, k = call(world, thetas, **kw)
        assert st == _lib.MICRO_EINVAL, (world, thetas, kw)
        assert k[0] == -7
    torch.cuda.synchronize()
    assert torch.equal(r, r0) and bool((oi == -1).all())
    sp.close()
    tk = micro.Sparsifier(N, device=DEV, variant=micro.MICRO_VARIANT_TICKET)
    with pytest.raises(micro.MicroError):
        tk.sweep(g, r, 2, 0.1, [1.0, 1.0])
    tk.close()
