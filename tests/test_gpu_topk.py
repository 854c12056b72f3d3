"""The exact top-k comparator (MICRO_RULE_TOPK) against the CPU oracle (GPU).

Every call goes through the C ABI via the ctypes binding.  Indices, values,
the selected count, the returned k-th magnitude and the residual must equal
the oracle's (oracle.topk_step / oracle.topk_ef_step) bit for bit, whatever
the incoming theta: none (NaN: the radix select's passes over the partition
first), the exact k-th magnitude (the step at 7/8 of it lists at least k
values: the passes over that list), one far above it (the step lists fewer
than k: the list returns to the residual and the passes and the pick run
over it) or far below it (a long list).  At the GPT-1.3B size, where the
oracle's sort would take minutes, the result is checked against the
properties that define the top k: the count, strictly increasing indices
inside the partition, the values and residual equal to the accumulation,
every selected magnitude at least every other one, and equal magnitudes
taken by lower index.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2310_00967_amd as micro
from paper_2310_00967_amd import synth

from gpu_harness import note

pytestmark = pytest.mark.gpu

DEV = "cuda"
AUTO, STAGED, TICKET = micro.MICRO_VARIANT_AUTO, micro.MICRO_VARIANT_STAGED, micro.MICRO_VARIANT_TICKET
SEPARATE = -STAGED
VARIANTS = pytest.mark.parametrize("variant", [STAGED, SEPARATE, TICKET], ids=["staged", "separate", "ticket"])


def make(n, variant=AUTO, **kw):
    if variant == SEPARATE:
        return micro.Sparsifier(n, device=DEV, rule=micro.MICRO_RULE_TOPK, variant=STAGED, separate_scan=True, **kw)
    return micro.Sparsifier(n, device=DEV, rule=micro.MICRO_RULE_TOPK, variant=variant, **kw)


def same_bits(a, b):
    """Bitwise equality of two float32 arrays, any NaN matching any NaN."""
    a = np.ascontiguousarray(a, np.float32)
    b = np.ascontiguousarray(b, np.float32)
    both = np.isnan(a) & np.isnan(b)
    return a.shape == b.shape and np.array_equal(a.view(np.uint32)[~both], b.view(np.uint32)[~both])


HINT_ROUTES = (micro.MICRO_TOPK_ROUTE_HINT_LIST, micro.MICRO_TOPK_ROUTE_HINT_PICK)
HINTS = pytest.mark.parametrize("hint", ["none", "exact", "high", "low"])


def hint_bound(theta):
    """The step's first threshold under a hint: the largest binary32 at or
    below 7/8 of theta."""
    b = float(theta) * 0.875
    f = np.float32(b)
    if float(f) > b:
        f = np.nextafter(f, np.float32(0))
    return f


def topk_k(density, ln):
    return oracle.topk_count(density, ln)


def theta_for(hint, kth):
    """The incoming theta for a hint kind, given the oracle's k-th magnitude."""
    if not isinstance(hint, str):
        return float(hint)
    if hint == "none" or not (0.0 < kth < math.inf):
        return math.nan
    return {"exact": kth, "high": 8.0 * kth, "low": kth / 1024.0}[hint]


def topk_vs_oracle(g, res, rank, world, density, variant=AUTO, phase_shift=0, sp=None, hint="none"):
    """One call on both sides; g/res are host float32 arrays.  `hint` picks
    the incoming theta (theta_for) or is the theta itself."""
    N = g.size
    own = sp is None
    if own:
        sp = make(N, variant)
    r_or = res.copy()
    o_idx, o_val, k_or, th_or = oracle.topk_step(g, r_or, rank, world, density, 1.0)
    theta = theta_for(hint, th_or if k_or else math.nan)
    if k_or == 0:
        th_or = theta  # nothing selected: theta comes back unchanged
    gbuf = torch.empty(N + 4, dtype=torch.float32, device=DEV)
    g_dev = gbuf[phase_shift:phase_shift + N]
    g_dev.copy_(torch.from_numpy(g))
    r_dev = torch.from_numpy(res).to(DEV)
    s, ln = oracle.partition(N, rank, world)
    sentinel = -12345
    out_idx = torch.full((max(1, ln) + 8,), sentinel, dtype=torch.int32, device=DEV)
    out_val = torch.full((max(1, ln) + 8,), float(sentinel), dtype=torch.float32, device=DEV)
    k, th, idx, val = sp.step(g_dev, r_dev, rank, world, density, theta, out_idx, out_val)
    route = sp.last_topk_route()
    where = f"N={N} rank {rank}/{world} d={density} variant {variant} shift {phase_shift} hint {hint} route {route}"
    assert k == k_or, f"{where}: k {k} oracle {k_or}"
    assert th == th_or or (math.isnan(th) and math.isnan(th_or)), f"{where}: kth {th!r} oracle {th_or!r}"
    assert np.array_equal(idx.cpu().numpy(), o_idx), f"{where}: indices differ"
    assert same_bits(val.cpu().numpy(), o_val), f"{where}: values differ"
    assert same_bits(r_dev.cpu().numpy(), r_or), f"{where}: residual differs"
    # Without a hint the step lists at most every value from the floor of
    # the k-th magnitude's first radix bin (its top 11 magnitude bits) up;
    # with one, every value from the hint's bound up; where that list falls
    # short, the values from the bin's floor up are extracted (or the top k
    # picked).  Past that nothing is written.
    acc = (g[s:s + ln] + res[s:s + ln]).astype(np.float32)
    keys = acc.view(np.uint32) & np.uint32(0x7FFFFFFF)
    finite = keys <= np.uint32(0x7F800000)
    bin_floor = np.uint32(np.float32(th_or).view(np.uint32) & np.uint32(0x7FF00000)) if k_or else None
    usable = (variant != TICKET and ln >= 8 and topk_k(density, ln) <= ln // 8 and 0 < theta < math.inf
              and float(theta) * 0.875 <= float(np.finfo(np.float32).max) and hint_bound(theta) > 0)
    assert (route in HINT_ROUTES) == usable, where
    if route in HINT_ROUTES:
        low = np.uint32(hint_bound(theta).view(np.uint32))
        reach = max(int(np.sum((keys >= low) & finite)), k_or)
        if route == micro.MICRO_TOPK_ROUTE_HINT_PICK and k_or:
            reach = max(reach, int(np.sum((keys >= bin_floor) & finite)))
        if route == micro.MICRO_TOPK_ROUTE_HINT_LIST:
            assert int(np.sum((keys >= low) & finite)) >= k_or, where
    else:
        reach = int(np.sum((keys >= bin_floor) & finite)) if k_or else 0
    if hint == "high" and route in HINT_ROUTES:
        assert route == micro.MICRO_TOPK_ROUTE_HINT_PICK, where
    assert np.all(out_idx.cpu().numpy()[reach:] == sentinel), f"{where}: written past the selection"
    if own:
        sp.close()
    return k


def gen(rng, n, kind):
    if kind == "normal":
        return rng.standard_normal(n).astype(np.float32), (0.5 * rng.standard_normal(n)).astype(np.float32)
    if kind == "quantised":  # few magnitudes: many values share the k-th
        return (np.round(rng.standard_normal(n) * 4) / 4).astype(np.float32), np.zeros(n, np.float32)
    if kind == "laplace":
        return rng.laplace(0, 1e-3, n).astype(np.float32), rng.laplace(0, 1e-3, n).astype(np.float32)
    raise ValueError(kind)


@pytest.mark.parametrize("N,world,rank", [
    (1, 1, 0), (3, 1, 0), (1023, 1, 0), (1024, 1, 0), (1025, 1, 0), (4099, 3, 1),
    (12289, 3, 2), (100003, 16, 5), (262144 + 5, 4, 3), (1000, 2000, 1999),
])
@pytest.mark.parametrize("density", [1e-4, 0.01, 0.5, 1.0])
@VARIANTS
@HINTS
def test_ragged_sizes_and_densities(N, world, rank, density, variant, hint):
    rng = np.random.default_rng(N * 3 + rank + int(density * 1e4))
    g, res = gen(rng, N, "normal")
    topk_vs_oracle(g, res, rank, world, density, variant, hint=hint)


@pytest.mark.parametrize("N", [5000, 1 << 20, (1 << 20) + 3, 3_000_017])
@pytest.mark.parametrize("density", [0.01, 0.3])
@pytest.mark.parametrize("kind", ["quantised", "laplace"])
@pytest.mark.parametrize("phase_shift", [0, 1])
@pytest.mark.parametrize("hint", ["none", "exact", "high"])
def test_equal_magnitudes_and_phases(N, density, kind, phase_shift, hint):
    """Quantised values put thousands of values at the k-th magnitude, so the
    trim pass runs over long lists; phase 1 takes the scalar-load passes (and
    a residual of another 16-byte phase than the gradient's for the pick's
    passes)."""
    note(f"top-k ties N={N} d={density} {kind} shift {phase_shift} hint {hint}")
    rng = np.random.default_rng(N + int(density * 100) + len(kind))
    g, res = gen(rng, N, kind)
    topk_vs_oracle(g, res, 0, 1, density, AUTO, phase_shift, hint=hint)


@VARIANTS
def test_all_values_equal(variant):
    """Every value ties: the k lowest indices, the rest returned to the residual."""
    for N, d in [(10, 0.3), (4097, 0.01), (2_000_003, 0.25), (2_000_003, 0.01)]:
        g = np.full(N, -0.5, np.float32)
        res = np.zeros(N, np.float32)
        for hint in ["none", "exact", "high", "low"]:
            k = topk_vs_oracle(g, res, 0, 1, d, variant, hint=hint)
            assert k == oracle.topk_count(d, N)


@VARIANTS
def test_special_values(variant):
    f = np.float32
    tiny = f(2.0) ** -149
    base = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, tiny, 1.0, -1.0, tiny, 3.0], dtype=np.float32)
    g = np.tile(base, 1000)
    res = np.tile(np.array([0.0, 0.0, 0.0, -0.0, 0.0, tiny, 0.0, 0.0, -tiny, np.nan], np.float32), 1000)
    for d in [1e-4, 0.05, 0.2, 0.35, 0.7, 1.0]:  # infinities only, then magnitude 3 ... up to every non-NaN value
        for hint in ["none", "exact", "high", "low", 1e-45, 3e38, -1.0, 0.0, math.inf]:
            topk_vs_oracle(g, res, 0, 1, d, variant, hint=hint)
    # more NaN than the selection leaves: fewer than k selected
    g2 = g.copy()
    g2[::3] = np.nan
    topk_vs_oracle(g2, res, 0, 1, 1.0, variant)
    # every value NaN: nothing selected, theta unchanged, residual = acc
    g3 = np.full(5000, np.nan, np.float32)
    for d, theta in [(0.5, 7.25), (0.01, 7.25), (0.01, 1e-30)]:
        k = topk_vs_oracle(g3, np.zeros(5000, np.float32), 0, 1, d, variant, hint=theta)
        assert k == 0
    # zeros only: the k-th magnitude is 0, the lowest indices win
    for hint in ["none", 1.0]:
        k = topk_vs_oracle(np.zeros(3000, np.float32), np.zeros(3000, np.float32), 0, 1, 0.1, variant, hint=hint)
        assert k == 300


def test_one_context_many_calls():
    """The radix-select counters and state are left clean by every call: a
    context alternating sizes, partitions, densities, hints and the
    nothing-selected case stays exact."""
    N = 300_007
    sp = make(N)
    rng = np.random.default_rng(99)
    for t in range(48):
        kind = ["normal", "quantised", "laplace"][t % 3]
        g, res = gen(rng, N, kind)
        world = [1, 3, 8][t % 3]
        rank = t % world
        d = [0.001, 0.02, 0.5, 1.0, 0.01][t % 5]
        if t % 7 == 6:
            g[:] = np.nan
        topk_vs_oracle(g, res, rank, world, d, sp=sp, hint=["exact", "none", "high", "low"][t % 4])
    sp.close()


@pytest.mark.parametrize("hint", ["exact", "high", "low"])
def test_hint_routes_are_taken(hint):
    """A 2M-value partition at d = 0.01 (k = 20,000): with the exact k-th
    magnitude as the hint the step at 7/8 of it lists at least k values and the
    passes run over that list; with 8 times it the step lists fewer than k
    and the pick runs over the residual; with 1/1024 of it the step lists
    about half the partition, more than the staging pairs hold, and the pick
    runs too."""
    N = 2_000_003
    rng = np.random.default_rng(7)
    g, res = gen(rng, N, "normal")
    sp = make(N)
    topk_vs_oracle(g, res, 0, 1, 0.01, sp=sp, hint=hint)
    want = {"exact": micro.MICRO_TOPK_ROUTE_HINT_LIST, "high": micro.MICRO_TOPK_ROUTE_HINT_PICK,
            "low": micro.MICRO_TOPK_ROUTE_HINT_PICK}[hint]
    assert sp.last_topk_route() == want
    topk_vs_oracle(g, res, 0, 1, 0.01, sp=sp, hint="none")
    assert sp.last_topk_route() == micro.MICRO_TOPK_ROUTE_LIST
    sp.close()


@pytest.mark.parametrize("seed", range(64))
def test_fuzz_sizes_densities_and_hints(seed):
    """Random partition sizes and ranks, densities from 1e-4 to 0.3, value
    kinds, schedules, grad phases and hints (the kinds above or any positive
    number), each case bit for bit against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    N = int(rng.integers(1, 3_000_000))
    world = int(rng.choice([1, 2, 3, 8, 16]))
    rank = int(rng.integers(0, world))
    density = float(10 ** rng.uniform(-4, np.log10(0.3)))
    kind = str(rng.choice(["normal", "quantised", "laplace"]))
    variant = int(rng.choice([AUTO, STAGED, SEPARATE, TICKET]))
    hint = rng.choice(["none", "exact", "high", "low", "random"])
    if hint == "random":
        hint = float(10 ** rng.uniform(-6, 2))
    g, res = gen(rng, N, kind)
    if rng.random() < 0.2:  # a sprinkle of special values
        pos = rng.integers(0, N, size=max(1, N // 1000))
        g[pos] = rng.choice(np.array([np.nan, np.inf, -np.inf, 0.0, -0.0], np.float32), size=pos.size)
    note(f"top-k fuzz seed {seed}: N={N} rank {rank}/{world} d={density:.3g} {kind} variant {variant} hint {hint}")
    topk_vs_oracle(g, res, rank, world, density, variant, phase_shift=int(rng.integers(0, 4)), hint=hint)


@pytest.mark.parametrize("variant", [AUTO, STAGED, SEPARATE], ids=["auto", "staged", "separate"])
def test_hint_list_of_exactly_k_below_the_hint(variant):
    """k values of 9.0 among small ones and a hint of 10: the step lists from
    8.75 up, exactly the k values, all of them below the hint, so the staged
    step left acc in their residual; with nothing to drop, the trim still has
    to set their residual to +0."""
    N = (1 << 20) + 5003
    rng = np.random.default_rng(77)
    g = (0.1 * rng.standard_normal(N)).astype(np.float32)
    k = oracle.topk_count(0.01, N)
    g[rng.choice(N, size=k, replace=False)] = np.float32(9.0)
    res = np.zeros(N, np.float32)
    sp = make(N, variant)
    topk_vs_oracle(g, res, 0, 1, 0.01, variant, sp=sp, hint=10.0)
    assert sp.last_topk_route() == micro.MICRO_TOPK_ROUTE_HINT_LIST
    sp.close()


@pytest.mark.parametrize("seed", range(40))
def test_hint_bounds_adversarial(seed):
    """Magnitudes just below, at and just above the step's two bounds for a
    hint of 1 (7/8, where it lists from, and 1, where it zeroes from), with
    random multiplicities and signs; k falls on, next to or between the
    groups, so the k-th magnitude meets either bound, the list holds exactly
    k values or far more, and ties at the k-th magnitude straddle the
    bounds."""
    rng = np.random.default_rng(9000 + seed)
    f = np.float32
    b, z = f(0.875), f(1.0)
    mags = np.array([f(0.5), np.nextafter(b, f(0)), b, f(0.9), np.nextafter(z, f(0)), z,
                     np.nextafter(z, f(2)), f(1.5), f(3.0)], np.float32)
    counts = rng.integers(1, 3000, size=mags.size)
    counts[0] += 200_000  # the bulk below both bounds (k stays within an eighth of the partition)
    if seed % 7 == 6:
        counts[rng.integers(1, mags.size - 1)] = 0
    vals = np.repeat(mags, counts)
    vals *= np.where(rng.random(vals.size) < 0.5, f(-1), f(1))
    rng.shuffle(vals)
    N = vals.size
    # k on the boundary of group `edge` (counting from the largest
    # magnitudes: k takes the groups above it whole), one below or above it,
    # or anywhere
    tops = np.cumsum(counts[::-1])[:-1]
    edge, choice = seed % tops.size, (seed // tops.size) % 4
    k = int(tops[edge]) + (0, -1, 1, 0)[choice]
    if choice == 3:
        k = int(rng.integers(1, N // 8 + 1))
    k = max(1, min(N // 8, k))
    density = (k + 0.5) / N
    assert oracle.topk_count(density, N) == k
    g = vals.astype(np.float32)
    res = np.zeros(N, np.float32)
    variant = [STAGED, SEPARATE, AUTO][seed % 3]
    note(f"top-k bounds seed {seed}: N={N} k={k} counts {counts.tolist()} variant {variant}")
    topk_vs_oracle(g, res, 0, 1, density, variant, hint=1.0)


@VARIANTS
@HINTS
def test_hint_with_dense_tiles(variant, hint):
    """A block of 100,000 large values in a 1M-value partition, k = 40,000:
    at the hint's bound most values of the block are listed, so its tiles
    overflow their staging slots and the move kernel redoes them, with the
    residual set to +0 only from the hint up."""
    N = 1_000_003
    rng = np.random.default_rng(31)
    g = (0.01 * rng.standard_normal(N)).astype(np.float32)
    g[200_000:300_000] = rng.uniform(1.0, 2.0, 100_000).astype(np.float32) * np.where(
        rng.random(100_000) < 0.5, -1, 1).astype(np.float32)
    res = (0.001 * rng.standard_normal(N)).astype(np.float32)
    sp = make(N, variant)
    topk_vs_oracle(g, res, 0, 1, 40_000 / N, variant, sp=sp, hint=hint)
    if variant != TICKET:
        _, redone, _, _ = sp.last_stats()
        if hint in ("exact", "low"):
            assert redone > 0
    sp.close()


@pytest.mark.parametrize("N,world", [(100_003, 4), (3_000_017, 8)])
def test_ef_steps_passing_theta_on(N, world):
    """Algorithm 1's pass with the top-k comparator over several iterations,
    each call given the k-th magnitude the last one returned (the hint), on
    both sides."""
    rng = np.random.default_rng(N + 1)
    sp = make(N)
    g_dev = torch.empty(N, dtype=torch.float32, device=DEV)
    r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    r_host = np.zeros(N, np.float32)
    theta = 1.0
    routes = []
    for t in range(6):
        g = (rng.laplace(0, 1e-3, N) * (1.0 + 0.5 * t)).astype(np.float32)
        g_dev.copy_(torch.from_numpy(g))
        k, th, c, idx, val = sp.ef_step(g_dev, r_dev, t, 2, world, 0.01, theta)
        routes.append(sp.last_topk_route())
        o_idx, o_val, k_or, th_or, c_or = oracle.topk_ef_step(g, r_host, t, 2, world, 0.01, theta)
        assert (k, th, c) == (k_or, th_or, c_or)
        assert np.array_equal(idx.cpu().numpy(), o_idx)
        assert same_bits(val.cpu().numpy(), o_val)
        assert same_bits(r_dev.cpu().numpy(), r_host)
        theta = th_or
    # 1.0 is far above the k-th magnitude at first: the pick; then the last
    # k-th magnitude is a hint the step's list covers
    assert routes[0] == micro.MICRO_TOPK_ROUTE_HINT_PICK
    assert micro.MICRO_TOPK_ROUTE_HINT_LIST in routes[1:]
    sp.close()


@pytest.mark.parametrize("N,world", [(100_003, 4), (3_000_017, 8)])
def test_ef_step_with_local_error(N, world):
    rng = np.random.default_rng(N)
    sp = make(N)
    g_dev = torch.empty(N, dtype=torch.float32, device=DEV)
    r_dev = torch.zeros(N, dtype=torch.float32, device=DEV)
    r_host = np.zeros(N, np.float32)
    theta = 1.0
    for t in range(3):
        g = (np.round(rng.standard_normal(N) * 8) / 8).astype(np.float32)  # ties at the k-th magnitude
        g_dev.copy_(torch.from_numpy(g))
        k, th, c, idx, val, sq = sp.ef_step(g_dev, r_dev, t, 1, world, 0.01, theta, local_error=True)
        o_idx, o_val, k_or, th_or, c_or = oracle.topk_ef_step(g, r_host, t, 1, world, 0.01, theta)
        assert (k, th, c) == (k_or, th_or, c_or)
        assert np.array_equal(idx.cpu().numpy(), o_idx)
        assert same_bits(val.cpu().numpy(), o_val)
        assert same_bits(r_dev.cpu().numpy(), r_host)
        exact = math.fsum(float(x) * float(x) for x in r_host.astype(np.float64))
        ties = int(np.sum(np.abs(r_host) == np.float32(th_or)))
        assert abs(sq - exact) <= (N + ties) * 2.0 ** -53 * exact
        theta = th_or
    sp.close()


def test_sweep_rejects_topk():
    sp = make(1000)
    g = torch.zeros(1000, dtype=torch.float32, device=DEV)
    r = torch.zeros(1000, dtype=torch.float32, device=DEV)
    with pytest.raises(micro.MicroError) as e:
        sp.sweep(g, r, 2, 0.1, [1.0, 1.0])
    assert e.value.status == 1
    sp.close()


def test_bert_large_rank3_full_partition():
    """BERT-large rank 3 of 8 (41,892,736 values) at d = 0.01, the whole
    partition against the oracle, two steps of error feedback."""
    w = synth.get("bert_large")
    sp = make(w.n_total)
    g_dev = torch.empty(w.n_total, dtype=torch.float32, device=DEV)
    r_dev = torch.zeros(w.n_total, dtype=torch.float32, device=DEV)
    s, ln = oracle.partition(w.n_total, 3, w.world)
    r_host = np.zeros(ln, np.float32)
    theta = 1.0
    for t in range(2):
        synth.gradient(w, t, DEV, out=g_dev)
        g_host = g_dev[s:s + ln].cpu().numpy()
        note(f"top-k bert_large rank 3 step {t}")
        k, th, idx, val = sp.step(g_dev, r_dev, 3, w.world, 0.01, theta)
        o_idx, o_val, k_or, th_or = oracle.topk_select(g_host, r_host, 0, ln, 0.01, kth=theta)
        assert k == k_or == oracle.topk_count(0.01, ln) and th == th_or
        assert np.array_equal(idx.cpu().numpy(), o_idx + s)
        assert same_bits(val.cpu().numpy(), o_val)
        assert same_bits(r_dev[s:s + ln].cpu().numpy(), r_host)
        theta = th
    sp.close()


def check_topk_properties(g, before, after, s, ln, idx, val, k, th, density):
    """The top k of [s, s + ln), checked from its definition with torch."""
    acc = g[s:s + ln] + before[s:s + ln]
    valid = ~torch.isnan(acc)
    want = min(oracle.topk_count(density, ln), int(valid.sum()))
    assert k == want
    loc = idx.long() - s
    assert int(loc[0]) >= 0 and int(loc[-1]) < ln
    assert bool((loc[1:] > loc[:-1]).all())
    assert torch.equal(val.view(torch.int32), acc[loc].view(torch.int32))
    sel = torch.zeros(ln, dtype=torch.bool, device=acc.device)
    sel[loc] = True
    part_after = after[s:s + ln]
    assert bool((part_after[sel].view(torch.int32) == 0).all())
    assert torch.equal(part_after[~sel].view(torch.int32), acc[~sel].view(torch.int32))
    assert torch.equal(after[:s].view(torch.int32), before[:s].view(torch.int32))
    assert torch.equal(after[s + ln:].view(torch.int32), before[s + ln:].view(torch.int32))
    mag = acc.abs()
    kth = mag[loc].min()
    assert th == float(kth)
    others = ~sel & valid
    if bool(others.any()):
        assert float(mag[others].max()) <= float(kth)
        tied_out = torch.nonzero(others & (mag == kth))
        if tied_out.numel():
            assert int(torch.nonzero(sel & (mag == kth)).max()) < int(tied_out.min())


@pytest.mark.parametrize("density", [0.01, 0.001])
def test_gpt_1p3b_full_size_properties(density):
    w = synth.get("gpt_1p3b")
    sp = make(w.n_total)
    g = torch.empty(w.n_total, dtype=torch.float32, device=DEV)
    res = torch.zeros(w.n_total, dtype=torch.float32, device=DEV)
    theta = 1.0
    for t in range(2):
        synth.gradient(w, t, DEV, out=g)
        before = res.clone()
        note(f"top-k gpt_1p3b d={density} step {t}")
        k, th, idx, val = sp.step(g, res, 0, 1, density, theta)
        check_topk_properties(g, before, res, 0, w.n_total, idx, val, k, th, density)
        theta = th
        del before
    sp.close()
    torch.cuda.empty_cache()


def test_largest_vector_the_index_type_allows():
    """n_total = 2^31 - 1, the largest vector int32 indices address: one
    partition-wide top-k step at d = 0.001, checked against the definition
    (at this size many values share the k-th magnitude, so the trim runs
    over a long list).  About 50 GB of device memory."""
    N = 2**31 - 1
    note(f"top-k largest vector N={N}")
    gen = torch.Generator(device=DEV).manual_seed(2025)
    g = torch.randn(N, generator=gen, device=DEV, dtype=torch.float32)
    res = torch.randn(N, generator=gen, device=DEV, dtype=torch.float32) * 0.5
    before = res.clone()
    sp = make(N)
    k, th, idx, val = sp.step(g, res, 0, 1, 0.001, 1.0)
    check_topk_properties(g, before, res, 0, N, idx, val, k, th, 0.001)
    assert int(idx[-1]) > 2**31 - 2**20  # indices near the top of the range were selected
    sp.close()
    del g, res, before, idx, val
    torch.cuda.empty_cache()


def test_build_up_of_the_comparators_and_its_absence_under_micro():
    """bench.build_up on the toy workload (4 workers): MiCRO's exclusive
    partitions make the union of the workers' selections exactly their sum;
    the top-k workers' selections overlap but stay distinct, so their union
    lies between one worker's density and n times it."""
    import bench
    w = synth.get("toy")
    d = w.densities[0]
    b = bench.build_up(w, d, 3)
    n = b["workers"]
    assert n == w.world
    for t in range(3):
        assert abs(b["union_density"]["micro"][t] - b["worker_density"]["micro"][t]) < 1e-12
        k_frac = oracle.topk_count(d, w.n_total) / w.n_total
        assert abs(b["worker_density"]["topk"][t] - k_frac) < 1e-12
        assert k_frac < b["union_density"]["topk"][t] <= n * k_frac + 1e-12
        assert b["union_density"]["hard_threshold"][t] <= n * b["worker_density"]["hard_threshold"][t] + 1e-12
