"""Pins of the oracle's full error-feedback pass, cyclic partition assignment
and union gather / reset / update (Algorithm 1, Sec. 2, Sec. 4.1, Sec. 4.4).

The oracle is checked against things other than itself: numpy's evaluation of
the definitions, the already-pinned partition-only step and partition
function, properties the paper states (exclusive partitions, rotation over n
iterations, nothing lost by error feedback) and special cases.
"""
import numpy as np
import pytest

import oracle


# ---------------------------------------------------------------------------
# cyclic assignment (Algorithm 1; Sec. 4.1)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("world", [1, 2, 3, 4, 7, 8, 16])
def test_cycle_is_a_rotation(world):
    """At t = 0 every worker searches its own partition; every iteration
    moves every worker one partition on (mod n)."""
    for worker in range(world):
        assert oracle.cycle(0, worker, world) == worker
        for t in range(3 * world + 2):
            assert oracle.cycle(t + 1, worker, world) == (oracle.cycle(t, worker, world) + 1) % world


@pytest.mark.parametrize("world", [1, 2, 5, 8, 16])
def test_cycle_partitions_exclusive_and_covering(world):
    """Sec. 4.1: at each iteration the workers hold pairwise different
    partitions; over n consecutive iterations each worker visits all of them."""
    for t0 in [0, 1, 5, 1000, 2**40 + 3]:
        at_t = sorted(oracle.cycle(t0, i, world) for i in range(world))
        assert at_t == list(range(world))
        for worker in range(world):
            seen = sorted(oracle.cycle(t0 + u, worker, world) for u in range(world))
            assert seen == list(range(world))


def test_cycle_rejects_bad_arguments():
    for args in [(-1, 0, 2), (0, 2, 2), (0, -1, 2), (0, 0, 0)]:
        with pytest.raises(ValueError):
            oracle.cycle(*args)


# ---------------------------------------------------------------------------
# full error-feedback pass
# ---------------------------------------------------------------------------

def numpy_ef(g, res, t, worker, world, theta):
    """numpy's evaluation of the pass: acc over the whole vector, selection
    in the cycle's partition only."""
    n = g.size
    c = oracle.cycle(t, worker, world)
    s, ln = oracle.partition(n, c, world)
    acc = g + res
    inside = np.zeros(n, bool)
    inside[s:s + ln] = True
    sel = inside & (np.abs(acc).astype(np.float64) >= theta)
    new_res = np.where(sel, np.float32(0.0), acc).astype(np.float32)
    idx = np.flatnonzero(sel).astype(np.int32)
    return idx, acc[idx], new_res, c, ln


def random_case(rng, n, heavy=False):
    g = rng.standard_normal(n).astype(np.float32)
    if heavy:
        g *= np.exp(rng.uniform(-4, 4, n)).astype(np.float32)
    res = (rng.standard_normal(n) * 0.7).astype(np.float32)
    return g, res


@pytest.mark.parametrize("n,world", [(0, 1), (1, 1), (17, 4), (1000, 3), (65_537, 8), (100_003, 16)])
def test_ef_step_matches_numpy_definition(n, world):
    rng = np.random.default_rng(n + world)
    for t in [0, 1, world + 2]:
        for worker in sorted({0, world - 1, world // 2}):
            for theta in [0.5, 1.7, 3.0]:
                g, res = random_case(rng, n, heavy=(t == 1))
                idx_np, val_np, res_np, c_np, ln = numpy_ef(g, res, t, worker, world, theta)
                r = res.copy()
                idx, val, k, th, c = oracle.ef_step(g, r, t, worker, world, 0.01, theta)
                assert c == c_np
                assert k == idx_np.size
                assert np.array_equal(idx, idx_np)
                assert np.array_equal(val.view(np.uint32), val_np.view(np.uint32))
                assert np.array_equal(r.view(np.uint32), res_np.view(np.uint32))
                assert th == oracle.estimate(0.01, ln, k, theta)


@pytest.mark.parametrize("world", [1, 2, 5])
def test_ef_step_is_partition_step_plus_accumulation(world):
    """Inside the cycle's partition the pass is the partition-only step;
    outside it is the plain accumulation; with one worker it is the step."""
    rng = np.random.default_rng(11 + world)
    n = 50_011
    g, res = random_case(rng, n)
    for t in range(2 * world):
        worker = (3 * t) % world
        r_ef = res.copy()
        idx, val, k, th, c = oracle.ef_step(g, r_ef, t, worker, world, 0.02, 1.9)
        r_step = res.copy()
        idx2, val2, k2, th2 = oracle.step(g, r_step, c, world, 0.02, 1.9)
        s, ln = oracle.partition(n, c, world)
        assert (k, th) == (k2, th2)
        assert np.array_equal(idx, idx2) and np.array_equal(val.view(np.uint32), val2.view(np.uint32))
        acc = oracle.accumulate(g, res)
        outside = np.ones(n, bool)
        outside[s:s + ln] = False
        assert np.array_equal(r_ef[outside].view(np.uint32), acc[outside].view(np.uint32))
        assert np.array_equal(r_ef[s:s + ln].view(np.uint32), r_step[s:s + ln].view(np.uint32))
        if world == 1:
            assert np.array_equal(r_ef.view(np.uint32), r_step.view(np.uint32))


@pytest.mark.parametrize("world", [2, 3, 8])
def test_ef_step_workers_partition_the_hard_threshold_selection(world):
    """Sec. 1 / Sec. 4.2: filtering is invariant to partitioning, so at one
    iteration the n workers (each on its own copy of the same vectors) select
    disjoint sets whose union is the selection over the whole vector."""
    rng = np.random.default_rng(5 * world)
    n = 30_001
    g, res = random_case(rng, n, heavy=True)
    theta = 2.2
    acc = g + res
    whole = np.flatnonzero(np.abs(acc).astype(np.float64) >= theta)
    t = 7
    parts = []
    for worker in range(world):
        idx, _, _, _, c = oracle.ef_step(g, res.copy(), t, worker, world, 0.01, theta)
        parts.append(idx)
    allidx = np.concatenate(parts)
    assert allidx.size == np.unique(allidx).size
    assert np.array_equal(np.sort(allidx), whole)


def test_ef_step_searches_every_partition_in_n_iterations():
    """Sec. 4.1: a worker with a threshold below every magnitude selects, over
    n consecutive iterations, every index exactly once."""
    world, n = 4, 10_003
    rng = np.random.default_rng(3)
    g = (rng.standard_normal(n) + 10.0).astype(np.float32)  # all |acc| > 1
    res = np.zeros(n, np.float32)
    got = []
    for t in range(world):
        idx, _, _, _, _ = oracle.ef_step(g, res, t, 2, world, 0.5, 1e-3)
        got.append(idx)
    allidx = np.concatenate(got)
    assert np.array_equal(np.sort(allidx), np.arange(n))


def test_ef_step_special_cases():
    rng = np.random.default_rng(8)
    n, world = 9_999, 3
    g, res = random_case(rng, n)
    acc = g + res
    # threshold above every finite binary32: a pure accumulation
    r = res.copy()
    idx, val, k, _, c = oracle.ef_step(g, r, 4, 1, world, 0.1, 1e39)
    assert k == 0 and np.array_equal(r.view(np.uint32), acc.view(np.uint32))
    # threshold below every magnitude: the partition is copied out, reset to
    # zero there, accumulated elsewhere
    r = res.copy()
    idx, val, k, _, c = oracle.ef_step(g, r, 4, 1, world, 0.1, 1e-30)
    s, ln = oracle.partition(n, c, world)
    assert k == ln and np.array_equal(idx, np.arange(s, s + ln))
    assert np.array_equal(val.view(np.uint32), acc[s:s + ln].view(np.uint32))
    assert not np.any(r[s:s + ln].view(np.uint32))
    assert np.array_equal(np.delete(r, np.s_[s:s + ln]).view(np.uint32),
                          np.delete(acc, np.s_[s:s + ln]).view(np.uint32))


def test_ef_step_rejects_bad_arguments_without_writing():
    g = np.ones(10, np.float32)
    r = np.full(10, 0.25, np.float32)
    for args in [(-1, 0, 2, 0.1, 1.0), (0, 2, 2, 0.1, 1.0), (0, 0, 2, 0.0, 1.0),
                 (0, 0, 2, 0.1, 0.0), (0, 0, 2, 0.1, float("inf")), (0, 0, 0, 0.1, 1.0)]:
        with pytest.raises(ValueError):
            oracle.ef_step(g, r, *args)
        assert np.all(r == np.float32(0.25))


# ---------------------------------------------------------------------------
# gather, reset and model update at the union of selected indices
# ---------------------------------------------------------------------------

def test_gather_zero_update_match_numpy():
    rng = np.random.default_rng(21)
    n = 20_000
    acc = rng.standard_normal(n).astype(np.float32)
    idx = np.sort(rng.choice(n, 777, replace=False)).astype(np.int32)
    assert np.array_equal(oracle.gather(acc, idx).view(np.uint32), acc[idx].view(np.uint32))
    a = acc.copy()
    oracle.zero(a, idx)
    b = acc.copy()
    b[idx] = 0.0
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    for world in [1, 3, 8]:
        x = rng.standard_normal(n).astype(np.float32)
        sums = (rng.standard_normal(idx.size) * 3).astype(np.float32)
        y = x.copy()
        oracle.update(y, idx, sums, world)
        z = x.copy()
        z[idx] = x[idx] - sums / np.float32(world)
        assert np.array_equal(y.view(np.uint32), z.view(np.uint32))


def test_update_special_cases():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(100).astype(np.float32)
    idx = np.arange(0, 100, 3, dtype=np.int32)
    v = rng.standard_normal(idx.size).astype(np.float32)
    y = x.copy()
    oracle.update(y, idx, np.zeros(idx.size, np.float32), 5)
    assert np.array_equal(y.view(np.uint32), x.view(np.uint32))
    y = x.copy()
    oracle.update(y, idx, (v * np.float32(4)).astype(np.float32), 4)  # exact average
    assert np.array_equal(y[idx], x[idx] - v)
    with pytest.raises(ValueError):
        oracle.update(x.copy(), idx, v, 0)


@pytest.mark.parametrize("world", [2, 4])
def test_algorithm1_loses_nothing(world):
    """Sec. 2: error feedback keeps every unselected gradient.  Simulating
    Algorithm 1 for n workers with values whose binary32 arithmetic is exact
    (small multiples of 1/8, n a power of two), after T iterations every
    element satisfies  sum_i e_i + n * (x_0 - x_T) = sum_t sum_i G_i,t
    exactly, the workers' selections never overlap, and their union is what
    each worker gathers and resets."""
    rng = np.random.default_rng(world)
    n, T = 4_099, 6
    x0 = (rng.integers(-64, 64, n) / 8).astype(np.float32)
    x = x0.copy()
    res = [np.zeros(n, np.float32) for _ in range(world)]
    total = np.zeros(n, np.float64)
    theta = [2.0] * world
    for t in range(T):
        grads = [(rng.integers(-16, 17, n) / 8).astype(np.float32) for _ in range(world)]
        for gi in grads:
            total += gi
        accs = [oracle.accumulate(grads[i], res[i]) for i in range(world)]
        picked = []
        for i in range(world):
            idx, val, k, theta[i], c = oracle.ef_step(grads[i], res[i], t, i, world, 0.05, theta[i])
            assert np.array_equal(val, accs[i][idx])
            picked.append(idx)
        union = np.sort(np.concatenate(picked)).astype(np.int32)
        assert union.size == np.unique(union).size
        summed = np.zeros(union.size, np.float32)
        for i in range(world):
            gi = oracle.gather(accs[i], union)
            summed = (summed + gi).astype(np.float32)
            oracle.zero(accs[i], union)
            # the pass already reset the worker's own selection and carried the rest
            r = res[i].copy()
            oracle.zero(r, union)
            assert np.array_equal(r, accs[i])
            res[i] = accs[i]
        oracle.update(x, union, summed, world)
    lhs = sum(r.astype(np.float64) for r in res) + world * (x0.astype(np.float64) - x.astype(np.float64))
    assert np.array_equal(lhs, total)


# ---------------------------------------------------------------------------
# local error norm (Sec. 2, Eq. 1) and the sweep of every partition
# ---------------------------------------------------------------------------

U = 2.0 ** -53  # unit roundoff of binary64


def order_bound(n, exact):
    """Error bound of any binary64 summation order for n nonnegative terms."""
    g = (n - 1) * U
    return g / (1 - g) * exact if n > 1 else 0.0


def test_sumsq_within_the_summation_bound_of_the_exact_sum():
    import math
    rng = np.random.default_rng(31)
    for n in [1, 2, 17, 1000, 100_003]:
        r = (rng.standard_normal(n) * np.exp(rng.uniform(-20, 20, n))).astype(np.float32)
        exact = math.fsum(float(v) * float(v) for v in r.astype(np.float64))  # squares exact in binary64
        got = oracle.sumsq(r)
        assert abs(got - exact) <= order_bound(n, exact)
        s, ln = min(3, n), max(0, n - 7)
        ex2 = math.fsum(float(v) ** 2 for v in r[s:s + ln].astype(np.float64))
        assert abs(oracle.sumsq(r, s, ln) - ex2) <= order_bound(ln, ex2)


def test_sumsq_special_cases():
    assert oracle.sumsq(np.zeros(1000, np.float32)) == 0.0
    assert oracle.sumsq(np.zeros(0, np.float32)) == 0.0
    x = np.float32(3.0000002)
    assert oracle.sumsq(np.array([x], np.float32)) == float(x) * float(x)  # exact square
    tiny = np.float32(2.0) ** -149
    assert oracle.sumsq(np.array([tiny, -tiny], np.float32)) == 2.0 * 2.0 ** -298
    ints = np.arange(-500, 501, dtype=np.float32)
    assert oracle.sumsq(ints) == 2 * sum(i * i for i in range(501))
    assert np.isnan(oracle.sumsq(np.array([1.0, np.nan], np.float32)))
    assert oracle.sumsq(np.array([1.0, -np.inf], np.float32)) == np.inf
    # binary32 squares that overflow binary32 stay finite in binary64
    big = np.float32(3e38)
    assert oracle.sumsq(np.array([big], np.float32)) == float(big) ** 2


@pytest.mark.parametrize("n,world", [(0, 3), (5, 8), (1000, 1), (65_537, 4), (200_003, 16)])
def test_sweep_matches_numpy_per_partition_filter(n, world):
    rng = np.random.default_rng(n + 7 * world)
    g = (rng.standard_normal(n) * np.exp(rng.uniform(-2, 2, n))).astype(np.float32)
    res0 = (rng.standard_normal(n) * 0.3).astype(np.float32)
    thetas = np.exp(rng.uniform(-1, 1.5, world))
    res = res0.copy()
    idx, val, k, th, sq = oracle.sweep(g, res, world, 0.02, thetas)
    acc = g + res0
    want_idx, want_k = [], []
    new_res = acc.copy()
    for r in range(world):
        s, ln = oracle.partition(n, r, world)
        sel = np.flatnonzero(np.abs(acc[s:s + ln]).astype(np.float64) >= thetas[r]) + s
        want_idx.append(sel)
        want_k.append(sel.size)
        new_res[sel] = 0.0
        assert th[r] == oracle.estimate(0.02, ln, sel.size, thetas[r])
        exact_sq = float(np.sum(new_res[s:s + ln].astype(np.float64) ** 2))
        assert abs(sq[r] - exact_sq) <= 2 * order_bound(ln, exact_sq)
    want_idx = np.concatenate(want_idx) if want_idx else np.zeros(0, np.int64)
    assert np.array_equal(idx, want_idx) and np.array_equal(k, want_k)
    assert np.array_equal(val.view(np.uint32), acc[want_idx].view(np.uint32))
    assert np.array_equal(res.view(np.uint32), new_res.view(np.uint32))


def test_sweep_does_not_depend_on_partition_order():
    """Partitions are disjoint: taking the steps in reverse order gives the
    same residual, pairs and thresholds."""
    n, world = 77_777, 6
    rng = np.random.default_rng(12)
    g = rng.standard_normal(n).astype(np.float32)
    res0 = (rng.standard_normal(n) * 0.5).astype(np.float32)
    thetas = [1.0 + 0.2 * r for r in range(world)]
    res = res0.copy()
    idx, val, k, th, sq = oracle.sweep(g, res, world, 0.05, thetas)
    res2 = res0.copy()
    parts = {}
    for r in reversed(range(world)):
        parts[r] = oracle.step(g, res2, r, world, 0.05, thetas[r])
    assert np.array_equal(res.view(np.uint32), res2.view(np.uint32))
    assert np.array_equal(idx, np.concatenate([parts[r][0] for r in range(world)]))
    assert [parts[r][2] for r in range(world)] == list(k)
    assert [parts[r][3] for r in range(world)] == list(th)


def test_sweep_rejects_bad_arguments():
    g = np.ones(10, np.float32)
    r = np.zeros(10, np.float32)
    for world, d, th in [(0, 0.1, []), (2, 0.0, [1, 1]), (2, 0.1, [1, 0]), (2, 0.1, [1, np.inf])]:
        with pytest.raises(ValueError):
            oracle.sweep(g, r, world, d, th)
    assert not np.any(r)
