"""Bit-exact parity of the HIP path with the CPU oracle (GPU).

Every call goes through the C ABI (include/micro_sparsify.h) via the ctypes
binding.  Indices, values, the selected count, the next threshold and the
residual must equal the oracle's bit for bit; the tolerance is zero.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2310_00967_amd as micro
from paper_2310_00967_amd import synth

from gpu_harness import ParityRun, first_mismatch, note

pytestmark = pytest.mark.gpu

DEV = "cuda"
STAGED, TICKET = micro.MICRO_VARIANT_STAGED, micro.MICRO_VARIANT_TICKET
# the staged schedule with its scan pass launched on its own
# (MICRO_FLAG_SEPARATE_SCAN); plain STAGED fuses it into the streaming launch
SEPARATE = -STAGED
VARIANTS = pytest.mark.parametrize("variant", [STAGED, SEPARATE, TICKET], ids=["staged", "separate", "ticket"])


def make_sparsifier(n, variant, **kw):
    if variant == SEPARATE:
        return micro.Sparsifier(n, device=DEV, variant=STAGED, separate_scan=True, **kw)
    return micro.Sparsifier(n, device=DEV, variant=variant, **kw)


@pytest.mark.parametrize("name,density,steps,variant", [
    ("toy", 0.01, 20, STAGED),
    ("toy", 0.01, 20, TICKET),
    ("resnet18", 0.01, 100, STAGED),
    ("resnet50", 0.001, 100, STAGED),
    ("resnet50", 0.001, 30, SEPARATE),
    ("bert_large", 0.01, 50, STAGED),
    ("bert_large", 0.01, 20, SEPARATE),
    ("bert_large", 0.01, 10, TICKET),
])
def test_workload_parity(name, density, steps, variant):
    note(f"parity {name} d={density} steps={steps} variant={variant}")
    run = ParityRun(synth.get(name), density, DEV, variant=abs(variant), separate_scan=variant == SEPARATE)
    try:
        run.run(steps)
    finally:
        run.close()


@pytest.mark.parametrize("name,density,steps,schedule", [
    ("resnet18", 0.01, 100, TICKET),     # 730,594-value partitions: one pass
    ("resnet50", 0.001, 100, STAGED),    # 3,194,629 values: the staged schedule
])
def test_workload_parity_default_schedule(name, density, steps, schedule):
    """The workload under the library's default (AUTO) schedule, the one the
    benchmark and any caller with a default configuration run, every rank at
    every step, with the schedule each call took checked."""
    note(f"parity {name} d={density} steps={steps} AUTO (expects {schedule})")
    run = ParityRun(synth.get(name), density, DEV, variant=micro.MICRO_VARIANT_AUTO, expect_schedule=schedule)
    try:
        run.run(steps)
    finally:
        run.close()


@pytest.mark.parametrize("density", [0.001, 0.01])
def test_gpt_parity(density):
    """The 1.3B-value GPT gradient as one partition (world 1), 20 steps."""
    note(f"parity gpt_1p3b d={density}")
    run = ParityRun(synth.get("gpt_1p3b"), density, DEV)
    try:
        run.run(20)
    finally:
        run.close()


# ---------------------------------------------------------------------------
# edge cases and ragged sizes (small inputs, oracle finishes instantly)
# ---------------------------------------------------------------------------

def gpu_vs_oracle(g, res, rank, world, density, theta, phase_shift=0, variant=STAGED):
    """One call on both sides; g/res are host float32 arrays.  phase_shift != 0
    places grad at a different 16-byte phase than residual (scalar-load kernels)."""
    N = g.size
    sp = make_sparsifier(N, variant)
    gbuf = torch.empty(N + 4, dtype=torch.float32, device=DEV)
    g_dev = gbuf[phase_shift:phase_shift + N]
    g_dev.copy_(torch.from_numpy(g))
    r_dev = torch.from_numpy(res).to(DEV)
    s, ln = oracle.partition(N, rank, world)
    sentinel = -12345
    out_idx = torch.full((max(1, ln) + 8,), sentinel, dtype=torch.int32, device=DEV)
    out_val = torch.full((max(1, ln) + 8,), float(sentinel), dtype=torch.float32, device=DEV)
    k, th, idx, val = sp.step(g_dev, r_dev, rank, world, density, theta, out_idx, out_val)
    r_or = res.copy()
    o_idx, o_val, k_or, th_or = oracle.step(g, r_or, rank, world, density, theta)
    assert k == k_or
    assert th == th_or
    assert np.array_equal(idx.cpu().numpy(), o_idx)
    v = val.cpu().numpy()
    nan_ok = np.isnan(v) & np.isnan(o_val)
    assert np.array_equal(v.view(np.uint32)[~nan_ok], o_val.view(np.uint32)[~nan_ok])
    rg = r_dev.cpu().numpy()
    nan_ok = np.isnan(rg) & np.isnan(r_or)
    assert np.array_equal(rg.view(np.uint32)[~nan_ok], r_or.view(np.uint32)[~nan_ok])
    # nothing written past k
    assert np.all(out_idx.cpu().numpy()[k:] == sentinel)
    assert np.all(out_val.cpu().numpy()[k:] == float(sentinel))
    sp.close()
    return k


@pytest.mark.parametrize("N,world,rank", [
    (1, 1, 0), (3, 1, 0), (4095, 1, 0), (4096, 1, 0), (4097, 1, 0), (4099, 3, 1),
    (12289, 3, 2), (40000, 7, 6), (100003, 16, 5), (262144 + 5, 4, 3), (1000, 2000, 1999),
])
@pytest.mark.parametrize("phase_shift", [0, 1])
@pytest.mark.parametrize("regime", ["sparse", "all", "none"])
@VARIANTS
def test_ragged_and_degenerate(N, world, rank, phase_shift, regime, variant):
    rng = np.random.default_rng(N + world + rank)
    g = rng.standard_normal(N).astype(np.float32)
    res = (rng.standard_normal(N) * 0.7).astype(np.float32)
    theta = {"sparse": 2.4, "all": 1e-30, "none": 1e30}[regime]
    k = gpu_vs_oracle(g, res, rank, world, 0.01, theta, phase_shift, variant)
    _, ln = oracle.partition(N, rank, world)
    if regime == "all":
        assert k == ln
    if regime == "none":
        assert k == 0


@pytest.mark.parametrize("seed", range(12))
@VARIANTS
def test_fuzz_sizes_and_starts(seed, variant):
    """Random N, world and rank: every start phase modulo 4, ragged tails,
    selection fractions from 0% to 100%."""
    rng = np.random.default_rng(1000 + seed)
    N = int(rng.integers(1, 3_000_000))
    world = int(rng.integers(1, 17))
    rank = int(rng.integers(0, world))
    g = (rng.standard_normal(N) * rng.uniform(0.1, 3)).astype(np.float32)
    res = (rng.standard_normal(N) * rng.uniform(0.0, 2)).astype(np.float32)
    theta = float(np.exp(rng.uniform(-4, 2.5)))
    gpu_vs_oracle(g, res, rank, world, float(rng.choice([0.001, 0.01, 0.1])), theta,
                  phase_shift=int(rng.integers(0, 4)), variant=variant)


@VARIANTS
def test_ieee_specials_and_threshold_boundaries(variant):
    f = np.float32
    tiny = f(2.0) ** -149
    base = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, tiny, 1.0, -1.0, tiny, 3.0], dtype=np.float32)
    g = np.tile(base, 1000)
    res = np.tile(np.array([0.0, 0.0, 0.0, -0.0, 0.0, tiny, 0.0, 0.0, -tiny, np.nan], np.float32), 1000)
    gpu_vs_oracle(g, res, 0, 1, 0.5, float(f(2.0) ** -148), variant=variant)
    gpu_vs_oracle(g, res, 0, 1, 0.5, float(f(2.0) ** -148), phase_shift=3, variant=variant)
    # thresholds at, and between, binary32 magnitudes
    rng = np.random.default_rng(5)
    g = rng.standard_normal(50_000).astype(np.float32)
    res = np.zeros_like(g)
    a = float(np.sort(np.abs(g))[-500])
    for theta in [a, np.nextafter(a, np.inf), np.nextafter(a, 0.0),
                  float(np.nextafter(np.float32(a), np.float32(np.inf))), a * (1 + 1e-12)]:
        gpu_vs_oracle(g, res, 0, 1, 0.01, float(theta), variant=variant)
    # threshold above FLT_MAX: only infinities are selected
    g[::97] = np.inf
    k = gpu_vs_oracle(g, res, 0, 1, 0.01, 1e39, variant=variant)
    assert k == g[::97].size


@VARIANTS
def test_subnormals_are_not_flushed(variant):
    tiny = np.float32(2.0) ** -149
    N = 70_000
    g = np.full(N, tiny, np.float32)
    res = np.full(N, tiny, np.float32)
    k = gpu_vs_oracle(g, res, 0, 1, 0.5, float(np.float32(2.0) ** -148), variant=variant)
    assert k == N


@pytest.mark.parametrize("phase_shift", [0, 2])
def test_dense_tiles_redone_by_move_kernel_mixed_with_staged_ones(phase_shift):
    """Tiles with more selected values than their staging slot holds (256 of
    1024) are listed by the scan kernel and redone by the move kernel's
    wavefronts straight into the output; they interleave with staged tiles
    and with each other, including at the ragged ends and across scan chunks
    (a million values each); theta = 1e-30 flags every tile."""
    rng = np.random.default_rng(77)
    N = 3 * 1_048_576 + 1234
    g = rng.standard_normal(N).astype(np.float32)
    res = np.zeros(N, np.float32)
    # dense bands (most values selected) of varied lengths and offsets
    for lo, ln in [(0, 700), (5000, 4096), (70_000, 1), (1_000_001, 300_000),
                   (2_097_000, 5000), (N - 3000, 3000)]:
        g[lo:lo + ln] *= 40.0
    for world, rank in [(1, 0), (3, 1), (7, 6)]:
        for theta in [3.0, 0.3, 1e-30]:
            gpu_vs_oracle(g, res, rank, world, 0.01, theta, phase_shift, STAGED)
    sp = micro.Sparsifier(N, device=DEV, variant=STAGED)
    g_dev = torch.from_numpy(g).to(DEV)
    r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    sp.step(g_dev, r_dev, 0, 1, 0.01, 3.0)
    _, redone, variant, _ = sp.last_stats()
    assert variant == STAGED and redone > 300
    sp.close()


@VARIANTS
def test_deterministic_under_repetition(variant):
    """The look-back must give the same bits every time (20 repetitions)."""
    N = 4_000_037
    rng = np.random.default_rng(9)
    g = torch.from_numpy(rng.standard_normal(N).astype(np.float32)).to(DEV)
    res0 = torch.from_numpy((rng.standard_normal(N) * 0.5).astype(np.float32)).to(DEV)
    sp = make_sparsifier(N, variant)
    ref = None
    for _ in range(20):
        res = res0.clone()
        k, th, idx, val = sp.step(g, res, 1, 3, 0.01, 2.0)
        cur = (k, th, idx.cpu().numpy().copy(), val.cpu().numpy().copy(), res.cpu().numpy())
        if ref is None:
            ref = cur
        else:
            assert cur[0] == ref[0] and cur[1] == ref[1]
            assert np.array_equal(cur[2], ref[2])
            assert first_mismatch(cur[3], ref[3]) < 0
            assert first_mismatch(cur[4], ref[4]) < 0
    sp.close()


def test_every_rank_of_a_world_and_disjointness():
    """Sweeping every rank with one threshold reproduces the unpartitioned
    filter (partition invariance) with pairwise disjoint outputs."""
    N = 1_000_003
    rng = np.random.default_rng(21)
    g = rng.standard_normal(N).astype(np.float32)
    res = np.zeros(N, np.float32)
    g_dev = torch.from_numpy(g).to(DEV)
    r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    sp = micro.Sparsifier(N, device=DEV)
    idx_all = []
    for r in range(16):
        k, th, idx, val = sp.step(g_dev, r_dev, r, 16, 0.01, 2.5)
        idx_all.append(idx.cpu().numpy().copy())
    whole_idx, _ = oracle.select(g, res, 0, N, 2.5)
    cat = np.concatenate(idx_all)
    assert np.array_equal(cat, whole_idx)
    assert np.unique(cat).size == cat.size
    assert first_mismatch(r_dev.cpu().numpy(), res) < 0
    sp.close()


def test_checkpoint_resume_matches_straight_run():
    w = synth.get("toy")
    N = w.n_total
    gs = [synth.gradient(w, t, DEV) for t in range(6)]

    def run(sp, res, th, ts):
        out = []
        for t in ts:
            k, th, idx, val = sp.step(gs[t], res, 0, w.world, 0.01, th)
            out.append((k, th, idx.cpu().numpy().copy(), val.cpu().numpy().copy()))
        return out, th

    sp = micro.Sparsifier(N, device=DEV)
    res_a = torch.zeros(N, device=DEV)
    straight, _ = run(sp, res_a, 2.33, range(6))
    res_b = torch.zeros(N, device=DEV)
    first, th_b = run(sp, res_b, 2.33, range(3))
    saved = res_b.cpu().clone()
    sp.close()
    sp2 = micro.Sparsifier(N, device=DEV)      # a fresh context resumes
    res_c = saved.to(DEV)
    resumed, _ = run(sp2, res_c, th_b, range(3, 6))
    for a, b in zip(straight, first + resumed):
        assert a[0] == b[0] and a[1] == b[1]
        assert np.array_equal(a[2], b[2]) and np.array_equal(a[3].view(np.uint32), b[3].view(np.uint32))
    assert first_mismatch(res_a.cpu().numpy(), res_c.cpu().numpy()) < 0
    sp2.close()


def test_fixed_step_rule_matches_oracle():
    w = synth.get("toy")
    run = ParityRun(w, 0.01, DEV, rule_kind=oracle.FIXED_STEP)
    try:
        run.run(6, verbose=False)
    finally:
        run.close()


@pytest.mark.parametrize("name,density,steps", [("toy", 0.01, 20), ("resnet50", 0.001, 20)])
def test_hard_threshold_comparator_matches_oracle_and_drifts(name, density, steps):
    """The hard-threshold comparator (MICRO_RULE_HARD_THRESHOLD, Sec. 1 and
    Sec. 5.2): bit for bit the oracle's steps with a fixed threshold, and
    under error feedback its actual density climbs well above the target,
    where the adaptive rule's stays near it."""
    note(f"hard threshold {name} d={density}")
    w = synth.get(name)
    run = ParityRun(w, density, DEV, rule_kind="hard")
    try:
        run.run(steps, verbose=False)
        assert run.thetas == run.thetas0  # the library's threshold never moved
        hard = np.mean(run.errors[-5:])
    finally:
        run.close()
    run = ParityRun(w, density, DEV)
    try:
        run.run(steps, verbose=False)
        adaptive = np.mean(run.errors[-5:])
    finally:
        run.close()
    # the oracle measures 10.5 / 0.17 (toy) and 1.49 / 0.09 (ResNet-50) over
    # the last five steps
    assert hard > 1.0          # the actual density above twice the target
    assert adaptive < hard / 4


def test_fused_and_separate_scans_on_one_context():
    """STAGED steps run the streaming and scan passes as one launch (stats
    fused = 1) unless MICRO_FLAG_SEPARATE_SCAN asks for two (fused = 0); both
    give the oracle's bits.  A multi-chunk partition with a dense region (its
    tiles overflow their staging slots) is stepped many times on one context,
    with sweeps (always separate launches) in between: the epoch-tagged
    flagged-tile counter is never cleared between launches, so a stale count
    would misplace pairs or redo the wrong tiles."""
    N = 9_000_011  # about nine scan chunks
    rng = np.random.default_rng(77)
    for sep in (False, True):
        note(f"fused/separate N={N} separate={sep}")
        sp = make_sparsifier(N, SEPARATE if sep else STAGED)
        r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
        r_host = np.zeros(N, np.float32)
        theta, thetas, redone = 2.0, [2.0, 2.0, 2.0], 0
        for t in range(8):
            g = rng.standard_normal(N).astype(np.float32)
            if t % 3 != 2:
                g[6_000_000:6_400_000] *= 40.0  # dense: every tile there overflows
            g_dev = torch.from_numpy(g).to(DEV)
            if t % 4 == 3:
                k, th, _, idx, val = sp.sweep(g_dev, r_dev, 3, 0.01, thetas)
                o_idx, o_val, k_or, th_or, _ = oracle.sweep(g, r_host, 3, 0.01, thetas)
                assert (k, th) == (list(k_or), list(th_or)), t
                thetas = th
            else:
                k, th, idx, val = sp.step(g_dev, r_dev, 1, 2, 0.01, theta)
                o_idx, o_val, k_or, th_or = oracle.step(g, r_host, 1, 2, 0.01, theta)
                assert (k, th) == (k_or, th_or), t
                _, redo, variant, fused = sp.last_stats()
                assert variant == STAGED and fused == (0 if sep else 1), t
                redone += redo
                theta = th
            assert np.array_equal(idx.cpu().numpy(), o_idx), t
            assert first_mismatch(val.cpu().numpy(), o_val) < 0, t
            assert first_mismatch(r_dev.cpu().numpy(), r_host) < 0, t
        assert redone > 0
        sp.close()


@pytest.mark.parametrize("N", [
    2 << 20,                     # 2,048 tiles, 2 chunks: every scan workgroup after the tiles
    3 << 20,                     # 3 chunks: chunk 0's scan workgroup among the tiles
    (3 << 20) + 1,               # one more tile, a one-tile last chunk
    (7 << 20) + 17 * 1024 + 5,   # ragged last tile, five interleaved chunks
    (256 << 20) + 1,             # 257 chunks
])
def test_fused_launch_interleaves_scan_workgroups(N):
    """The fused stream-and-scan launch places the scan workgroup of chunk c
    after the tiles of chunk c + 2 and the last chunks' after all tiles; it
    takes every partition (stats fused = 1).  Sizes around the boundaries of
    that layout give the oracle's bits."""
    note(f"fused layout N={N}")
    rng = np.random.default_rng(N % 1000)
    g = rng.standard_normal(N, dtype=np.float32)
    g[N // 3:N // 3 + 300_000] *= 30.0  # a dense region: its tiles overflow their staging slots
    res = np.zeros(N, np.float32)
    sp = micro.Sparsifier(N, device=DEV, variant=STAGED)
    g_dev = torch.from_numpy(g).to(DEV)
    r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    k, th, idx, val = sp.step(g_dev, r_dev, 0, 1, 0.01, 2.6)
    assert sp.last_stats()[3] == 1, N
    assert sp.last_stats()[1] > 0, N  # tiles redone by the move kernel
    o_idx, o_val, k_or, th_or = oracle.step(g, res, 0, 1, 0.01, 2.6)
    assert (k, th) == (k_or, th_or), N
    assert np.array_equal(idx.cpu().numpy(), o_idx), N
    assert first_mismatch(val.cpu().numpy(), o_val) < 0, N
    assert first_mismatch(r_dev.cpu().numpy(), res) < 0, N
    sp.close()
    del g_dev, r_dev
    torch.cuda.empty_cache()


def test_auto_schedule_picks_by_partition_length():
    """AUTO runs the one-pass ticket schedule up to 2^20 values and the staged
    schedule above, with the same bits either way (lengths on both sides of
    the boundary, compared with the oracle)."""
    rng = np.random.default_rng(20)
    for N, want in [(1 << 20, TICKET), ((1 << 20) + 1, STAGED), (262_144, TICKET), (3_000_000, STAGED)]:
        g = rng.standard_normal(N).astype(np.float32)
        res = (rng.standard_normal(N) * 0.5).astype(np.float32)
        sp = micro.Sparsifier(N, device=DEV, time_kernel=True)
        g_dev = torch.from_numpy(g).to(DEV)
        r_dev = torch.from_numpy(res).to(DEV)
        k, th, idx, val = sp.step(g_dev, r_dev, 0, 1, 0.01, 2.4)
        assert sp.last_stats()[2] == want, N
        r_or = res.copy()
        o_idx, o_val, k_or, th_or = oracle.step(g, r_or, 0, 1, 0.01, 2.4)
        assert (k, th) == (k_or, th_or)
        assert np.array_equal(idx.cpu().numpy(), o_idx)
        assert first_mismatch(val.cpu().numpy(), o_val) < 0
        assert first_mismatch(r_dev.cpu().numpy(), r_or) < 0
        sp.close()


def test_count_swings_on_one_context():
    """The move grid is sized from the density and the previous launch; k
    jumping between almost nothing and everything on one context (a grid far
    too small, then far too large) keeps the bits."""
    N = 5_000_011
    rng = np.random.default_rng(33)
    g = rng.standard_normal(N).astype(np.float32)
    sp = micro.Sparsifier(N, device=DEV, variant=STAGED)
    g_dev = torch.from_numpy(g).to(DEV)
    res = np.zeros(N, np.float32)
    r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    for theta in [5.5, 1e-30, 4.0, 1e-30, 0.3, 6.0, 1e-30]:
        k, th, idx, val = sp.step(g_dev, r_dev, 0, 1, 0.001, theta)
        o_idx, o_val, k_or, th_or = oracle.step(g, res, 0, 1, 0.001, theta)
        assert (k, th) == (k_or, th_or), theta
        assert np.array_equal(idx.cpu().numpy(), o_idx), theta
        assert first_mismatch(val.cpu().numpy(), o_val) < 0, theta
        assert first_mismatch(r_dev.cpu().numpy(), res) < 0, theta
    sp.close()


def test_move_piece_size_does_not_change_the_result():
    """The density steers only the threshold update and the move kernel's
    piece size (512, 1024 or 4096 items by the expected sequence length; on
    256 compute units d = 0.001, 0.1 and 1 give the three sizes for this
    partition).  At the same threshold all must select, place and reset the
    same bits, and match the oracle."""
    N = 3_000_017
    rng = np.random.default_rng(71)
    g = rng.standard_normal(N).astype(np.float32)
    res0 = (rng.standard_normal(N) * 0.5).astype(np.float32)
    sp = micro.Sparsifier(N, device=DEV, variant=STAGED)
    g_dev = torch.from_numpy(g).to(DEV)
    for theta in [2.5, 1.0]:
        outs = []
        for density in [0.001, 0.1, 1.0]:
            r_dev = torch.from_numpy(res0).to(DEV)
            k, th, idx, val = sp.step(g_dev, r_dev, 0, 1, density, theta)
            res = res0.copy()
            o_idx, o_val, k_or, th_or = oracle.step(g, res, 0, 1, density, theta)
            assert (k, th) == (k_or, th_or), (theta, density)
            outs.append((idx.cpu().numpy(), val.cpu().numpy(), r_dev.cpu().numpy()))
            assert np.array_equal(outs[-1][0], o_idx), (theta, density)
            assert first_mismatch(outs[-1][1], o_val) < 0, (theta, density)
        for other in outs[1:]:
            assert np.array_equal(outs[0][0], other[0]), theta
            assert first_mismatch(outs[0][1], other[1]) < 0, theta
            assert first_mismatch(outs[0][2], other[2]) < 0, theta
        assert first_mismatch(outs[0][2], res) < 0, theta
    sp.close()


def test_largest_vector_the_index_type_allows():
    """n_total = 2^31 - 1, the largest vector int32 indices address: one
    partition-wide step (staged) and one full error-feedback pass of world 2,
    bit for bit against the oracle.  About 40 GB of device memory."""
    N = 2**31 - 1
    note(f"largest vector N={N}")
    gen = torch.Generator(device=DEV).manual_seed(2024)
    g_dev = torch.randn(N, generator=gen, device=DEV, dtype=torch.float32)
    r_dev = (torch.randn(N, generator=gen, device=DEV, dtype=torch.float32) * 0.5)
    g = g_dev.cpu().numpy()
    res = r_dev.cpu().numpy()
    sp = micro.Sparsifier(N, device=DEV)
    k, th, idx, val = sp.step(g_dev, r_dev, 0, 1, 0.001, 3.3)
    assert sp.last_stats()[2] == STAGED
    o_idx, o_val, k_or, th_or = oracle.step(g, res, 0, 1, 0.001, 3.3)
    assert (k, th) == (k_or, th_or)
    assert np.array_equal(idx.cpu().numpy(), o_idx)
    assert int(o_idx[-1]) > 2**31 - 2**20  # indices near the top of the range were selected
    assert first_mismatch(val.cpu().numpy(), o_val) < 0
    assert first_mismatch(r_dev.cpu().numpy(), res) < 0
    del idx, val, o_idx, o_val
    note("largest vector: full pass, world 2")
    k, th, c, idx, val = sp.ef_step(g_dev, r_dev, 1, 0, 2, 0.001, 3.3)
    o_idx, o_val, k_or, th_or, c_or = oracle.ef_step(g, res, 1, 0, 2, 0.001, 3.3)
    assert (k, th, c) == (k_or, th_or, c_or) and c == 1
    assert np.array_equal(idx.cpu().numpy(), o_idx)
    assert first_mismatch(val.cpu().numpy(), o_val) < 0
    assert first_mismatch(r_dev.cpu().numpy(), res) < 0
    sp.close()


def test_two_contexts_on_two_streams():
    """Contexts own their scratch and stream: two contexts, each on its own
    torch stream (default priority), stepping interleaved on different
    workloads and schedules, each match the oracle."""
    rng = np.random.default_rng(44)
    cases = []
    for N, variant, world, rank in [(2_500_003, STAGED, 3, 1), (300_001, TICKET, 2, 0)]:
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            sp = micro.Sparsifier(N, device=DEV, variant=variant, stream=s)
            r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
        cases.append(dict(N=N, sp=sp, stream=s, world=world, rank=rank, r_dev=r_dev,
                          res=np.zeros(N, np.float32), theta=2.0, rng=rng))
    for t in range(6):
        for c in cases:
            g = (c["rng"].standard_normal(c["N"])).astype(np.float32)
            with torch.cuda.stream(c["stream"]):
                g_dev = torch.from_numpy(g).to(DEV, non_blocking=False)
                k, th, idx, val = c["sp"].step(g_dev, c["r_dev"], c["rank"], c["world"], 0.01, c["theta"])
                idx_h, val_h, r_h = idx.cpu().numpy(), val.cpu().numpy(), c["r_dev"].cpu().numpy()
            o_idx, o_val, k_or, th_or = oracle.step(g, c["res"], c["rank"], c["world"], 0.01, c["theta"])
            assert (k, th) == (k_or, th_or)
            assert np.array_equal(idx_h, o_idx)
            assert first_mismatch(val_h, o_val) < 0
            assert first_mismatch(r_h, c["res"]) < 0
            c["theta"] = th
    for c in cases:
        c["sp"].close()
