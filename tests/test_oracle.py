"""Pins the CPU oracle to things other than itself (CPU only).

* the plain definition of the filter evaluated by numpy (binary32 add with
  round-to-nearest-even and no fused multiply-add, magnitude widened to
  binary64, ">=", flatnonzero) on random vectors;
* brute force on tiny vectors with the threshold at, just above and just below
  each accumulated magnitude (binary64 and binary32 neighbours);
* IEEE special values, subnormals, the all/none-selected reductions;
* the invariants of Sec. 2 / Sec. 4.1 / Sec. 4.2 (error-feedback conservation,
  exhaustive selection, indices inside the partition and increasing, partition
  tiling, partition invariance of the filter, disjointness of the ranks);
* exact scale equivariance under powers of two.
"""
import numpy as np
import pytest

import oracle


def numpy_filter(g, res, start, length, theta):
    """The plain definition, evaluated by numpy on copies."""
    acc = (g[start:start + length] + res[start:start + length]).astype(np.float32)
    mask = np.abs(acc).astype(np.float64) >= theta
    idx = (np.flatnonzero(mask) + start).astype(np.int32)
    val = acc[mask]
    new_res = res.copy()
    new_res[start:start + length] = np.where(mask, np.float32(0.0), acc)
    return idx, val, new_res


def bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


def assert_bits_equal(a, b):
    assert a.shape == b.shape
    assert np.array_equal(bits(a), bits(b))


@pytest.mark.parametrize("length", [0, 1, 2, 3, 5, 63, 64, 65, 1000, 4099, 100003])
@pytest.mark.parametrize("regime", ["sparse", "dense", "all", "none"])
def test_select_matches_numpy_definition(length, regime):
    rng = np.random.default_rng(length * 7 + len(regime))
    n = length + 11
    g = rng.standard_normal(n).astype(np.float32)
    res = (rng.standard_normal(n) * 0.5).astype(np.float32)
    theta = {"sparse": 2.5, "dense": 0.3, "all": 1e-30, "none": 1e30}[regime]
    start = 5
    want_idx, want_val, want_res = numpy_filter(g, res, start, length, theta)
    got_res = res.copy()
    idx, val = oracle.select(g, got_res, start, length, theta)
    assert np.array_equal(idx, want_idx)
    assert_bits_equal(val, want_val)
    assert_bits_equal(got_res, want_res)
    if regime == "all":
        assert idx.size == length
    if regime == "none":
        assert idx.size == 0


def test_threshold_boundaries_brute_force():
    rng = np.random.default_rng(1)
    g = (rng.standard_normal(24) * 3).astype(np.float32)
    res = (rng.standard_normal(24)).astype(np.float32)
    acc = (g + res).astype(np.float32)
    for j in range(acc.size):
        a = float(abs(acc[j]))
        cands = {
            a: True,                                  # equality selects (">=")
            np.nextafter(a, np.inf): False,           # next binary64 above
            np.nextafter(a, 0.0): True,               # next binary64 below
            float(np.nextafter(np.float32(a), np.float32(np.inf))): False,
            float(np.nextafter(np.float32(a), np.float32(0))): True,
        }
        for theta, selected in cands.items():
            r = res.copy()
            idx, val = oracle.select(g, r, 0, g.size, theta)
            assert (j in set(idx.tolist())) == selected, (j, a, theta)
            # brute force over every element: selected iff |acc| >= theta
            want = [i for i in range(acc.size) if float(abs(acc[i])) >= theta]
            assert idx.tolist() == want


def test_special_values():
    f = np.float32
    tiny = f(np.float32(2.0) ** -149)  # smallest subnormal
    g = np.array([np.nan, np.inf, -np.inf, -0.0, 0.0, tiny, 1.0, -1.0, tiny, 3.0], dtype=np.float32)
    res = np.array([0.0, 0.0, 0.0, -0.0, 0.0, tiny, 0.0, 0.0, -tiny, np.nan], dtype=np.float32)
    theta = float(f(2.0) ** -148)  # exactly tiny + tiny
    r = res.copy()
    idx, val = oracle.select(g, r, 0, g.size, theta)
    # NaN never selected and carried; +-inf selected; -0 and +0 not selected;
    # the subnormal sum 2^-148 is kept exactly (no flush to zero) and selected;
    # tiny + (-tiny) = +0 is not selected.
    assert idx.tolist() == [1, 2, 5, 6, 7]
    assert np.isposinf(val[0]) and np.isneginf(val[1])
    assert val[2] == f(2.0) ** -148
    assert np.isnan(r[0]) and np.isnan(r[9])
    assert bits(r[[1, 2, 5, 6, 7]]).tolist() == [0, 0, 0, 0, 0]  # +0.0 written
    assert bits(r[3:4]).tolist() == [0x80000000]  # -0 + -0 = -0 carried
    assert bits(r[8:9]).tolist() == [0]           # tiny - tiny = +0 carried


def test_zero_length_partition_is_a_no_op():
    g = np.ones(3, np.float32)
    res = np.full(3, 0.25, np.float32)
    # world > N leaves some ranks with an empty partition
    empty = [r for r in range(5) if oracle.partition(3, r, 5)[1] == 0]
    assert empty
    for r in empty:
        rr = res.copy()
        idx, val, k, th = oracle.step(g, rr, r, 5, 0.5, 0.7)
        assert k == 0 and th == 0.7
        assert_bits_equal(rr, res)


@pytest.mark.parametrize("n_total,world", [(0, 1), (1, 1), (10, 3), (11_689_512, 16),
                                           (1_048_576, 4), (335_141_888, 8), (7, 16),
                                           (2**31 - 1, 7), (1_315_723_264, 1)])
def test_partitions_tile_exactly(n_total, world):
    """Sec. 4.1: n contiguous ranges that tile [0, N), lengths within one of
    each other, and all equal when n divides N."""
    pos = 0
    lens = []
    for r in range(world):
        s, ln = oracle.partition(n_total, r, world)
        assert s == pos and ln >= 0
        pos += ln
        lens.append(ln)
    assert pos == n_total
    assert max(lens) - min(lens) <= 1
    if n_total % world == 0:
        assert len(set(lens)) == 1
    assert sum(lens) == n_total


def test_partition_rejects_bad_arguments():
    for args in [(10, -1, 4), (10, 4, 4), (10, 0, 0), (-1, 0, 1)]:
        with pytest.raises(ValueError):
            oracle.partition(*args)


def test_invariants_on_one_step():
    rng = np.random.default_rng(7)
    N, world = 10007, 5
    g = rng.standard_normal(N).astype(np.float32)
    res0 = (rng.standard_normal(N) * 2).astype(np.float32)
    theta = 2.1
    acc = (g + res0).astype(np.float32)
    seen = set()
    total = 0
    cat_idx, cat_val = [], []
    for r in range(world):
        s, ln = oracle.partition(N, r, world)
        res = res0.copy()
        idx, val = oracle.select(g, res, s, ln, theta)
        # I1 conservation, per element
        sel = np.zeros(N, bool)
        sel[idx] = True
        part = np.zeros(N, bool)
        part[s:s + ln] = True
        assert_bits_equal(val, acc[idx])
        assert np.all(bits(res[sel]) == 0)
        assert_bits_equal(res[part & ~sel], acc[part & ~sel])
        assert_bits_equal(res[~part], res0[~part])  # outside the partition untouched
        # I2 exhaustive: k equals the count of |acc| >= theta in the partition
        assert idx.size == int(np.count_nonzero(np.abs(acc[s:s + ln]).astype(np.float64) >= theta))
        # I3 inside the partition and strictly increasing
        assert np.all((idx >= s) & (idx < s + ln))
        assert np.all(np.diff(idx) > 0)
        # I6 disjoint across ranks
        assert not (seen & set(idx.tolist()))
        seen |= set(idx.tolist())
        total += idx.size
        cat_idx.append(idx)
        cat_val.append(val)
    assert len(seen) == total
    # I4 partition invariance: the concatenation equals the unpartitioned filter
    res = res0.copy()
    full_idx, full_val = oracle.select(g, res, 0, N, theta)
    assert np.array_equal(np.concatenate(cat_idx), full_idx)
    assert_bits_equal(np.concatenate(cat_val), full_val)


@pytest.mark.parametrize("shift", [-20, -3, 5, 17])
def test_power_of_two_scale_equivariance(shift):
    rng = np.random.default_rng(11)
    g = rng.standard_normal(5000).astype(np.float32)
    res = rng.standard_normal(5000).astype(np.float32)
    theta = 1.7
    c = np.float32(2.0) ** shift
    r1, r2 = res.copy(), (res * c).astype(np.float32)
    i1, v1 = oracle.select(g, r1, 0, 5000, theta)
    i2, v2 = oracle.select((g * c).astype(np.float32), r2, 0, 5000, theta * float(c))
    assert np.array_equal(i1, i2)
    assert_bits_equal((v1 * c).astype(np.float32), v2)
    assert_bits_equal((r1 * c).astype(np.float32), r2)


def test_step_rejects_bad_arguments():
    g = np.zeros(8, np.float32)
    for kw in [dict(rank=0, world=0, density=0.1, theta=1.0),
               dict(rank=2, world=2, density=0.1, theta=1.0),
               dict(rank=0, world=1, density=0.0, theta=1.0),
               dict(rank=0, world=1, density=1.5, theta=1.0),
               dict(rank=0, world=1, density=float("nan"), theta=1.0),
               dict(rank=0, world=1, density=0.1, theta=0.0),
               dict(rank=0, world=1, density=0.1, theta=float("inf")),
               dict(rank=0, world=1, density=0.1, theta=float("nan"))]:
        r = np.zeros(8, np.float32)
        with pytest.raises(ValueError):
            oracle.step(g, r, **kw)
