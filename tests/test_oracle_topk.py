"""Pins the oracle's exact top-k comparator to things other than itself (CPU only).

* the definition evaluated by numpy: binary32 accumulation, NaN removed, a
  stable argsort of the negated magnitudes (so equal magnitudes keep index
  order), the first k taken and emitted in index order;
* the count k = max(1, floor(d * P)) against Python integer arithmetic;
* planted ties, NaN, infinities, signed zeros and subnormals;
* the already pinned threshold rule: without ties at the k-th magnitude, the
  top-k selection is the threshold selection at that magnitude;
* the order invariant (every selected magnitude >= every other non-NaN one)
  and exact conservation (acc = new residual + selected values);
* the hand-worked example in tests/golden/topk_worked_example.txt.
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "topk_worked_example.txt")


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)


def numpy_topk(g, res, start, length, density):
    acc = (g[start:start + length] + res[start:start + length]).astype(np.float32)
    k = 0 if length == 0 else min(length, max(1, math.floor(density * length)))
    valid = np.flatnonzero(~np.isnan(acc))
    order = valid[np.argsort(-np.abs(acc[valid]).astype(np.float64), kind="stable")]
    take = order[:min(k, valid.size)]
    mask = np.zeros(length, bool)
    mask[take] = True
    new_res = res.copy()
    new_res[start:start + length] = np.where(mask, np.float32(0.0), acc)
    kth = float(np.abs(acc[take[-1]])) if take.size else None
    return (np.flatnonzero(mask) + start).astype(np.int32), acc[mask], new_res, kth


def data(rng, n, kind):
    if kind == "normal":
        return rng.standard_normal(n).astype(np.float32), (0.5 * rng.standard_normal(n)).astype(np.float32)
    if kind == "quantised":  # few distinct magnitudes: ties everywhere
        return (np.round(rng.standard_normal(n) * 4) / 4).astype(np.float32), np.zeros(n, np.float32)
    if kind == "laplace":
        return rng.laplace(0, 1e-3, n).astype(np.float32), rng.laplace(0, 1e-3, n).astype(np.float32)
    raise ValueError(kind)


@pytest.mark.parametrize("length", [0, 1, 2, 3, 64, 65, 1000, 4099, 100003])
@pytest.mark.parametrize("density", [1e-4, 0.01, 0.3, 1.0])
@pytest.mark.parametrize("kind", ["normal", "quantised", "laplace"])
def test_topk_matches_numpy_definition(length, density, kind):
    rng = np.random.default_rng(length * 31 + int(density * 1e4) + len(kind))
    g, res = data(rng, length + 9, kind)
    start = 4
    want_idx, want_val, want_res, want_kth = numpy_topk(g, res, start, length, density)
    got_res = res.copy()
    idx, val, k, kth = oracle.topk_select(g, got_res, start, length, density, kth=-1.0)
    assert k == want_idx.size
    assert np.array_equal(idx, want_idx)
    assert np.array_equal(bits(val), bits(want_val))
    assert np.array_equal(bits(got_res), bits(want_res))
    assert kth == (want_kth if want_kth is not None else -1.0)


@pytest.mark.parametrize("length", [1, 2, 3, 7, 10, 99, 1000, 12345, 2 ** 31 - 1])
@pytest.mark.parametrize("density", [1e-9, 1e-4, 0.001, 0.01, 0.1, 0.3, 0.5, 0.999, 1.0])
def test_topk_count(length, density):
    assert oracle.topk_count(density, length) == min(length, max(1, math.floor(density * length)))


def test_topk_count_edges():
    assert oracle.topk_count(0.5, 0) == 0
    assert oracle.topk_count(0.3, 10) == 3       # 0.3 * 10 rounds to 3.0000000000000004 in binary64
    assert oracle.topk_count(0.1, 30) == 3
    assert oracle.topk_count(1.0, 5) == 5


def test_equal_magnitudes_go_to_the_lower_index():
    n = 1000
    g = np.where(np.arange(n) % 2 == 0, 1.0, -1.0).astype(np.float32)
    res = np.zeros(n, np.float32)
    idx, val, k, kth = oracle.topk_select(g, res, 0, n, 0.013)
    assert k == 13
    assert np.array_equal(idx, np.arange(13, dtype=np.int32))
    assert kth == 1.0
    # one value larger than the rest, placed last: it ranks first, the ties fill the rest
    g2 = g.copy()
    g2[-1] = 2.0
    idx2, _, k2, _ = oracle.topk_select(g2, np.zeros(n, np.float32), 0, n, 0.013)
    assert np.array_equal(idx2, np.concatenate([np.arange(12), [n - 1]]).astype(np.int32))


def test_nan_never_infinities_first_signed_zeros_tie():
    g = np.array([np.nan, 1.0, -np.inf, 0.0, -0.0, 1e-45, np.inf, np.nan, -1.0, 0.0], np.float32)
    res = np.zeros(g.size, np.float32)
    res[4] = -0.0
    # k = 10 but two are NaN: everything else is selected
    r = res.copy()
    idx, val, k, kth = oracle.topk_select(g, r, 0, g.size, 1.0)
    assert k == 8 and list(idx) == [1, 2, 3, 4, 5, 6, 8, 9]
    assert np.isnan(r[0]) and np.isnan(r[7])
    assert kth == 0.0
    # k = 3: the two infinities (lower index first), then the first of the two magnitude-1 values
    r = res.copy()
    idx, val, k, kth = oracle.topk_select(g, r, 0, g.size, 0.3)
    assert list(idx) == [1, 2, 6] and math.isinf(kth) is False and kth == 1.0
    # k = 5: then the other magnitude-1 value (j = 8) and the subnormal
    r = res.copy()
    idx, val, k, kth = oracle.topk_select(g, r, 0, g.size, 0.5)
    assert list(idx) == [1, 2, 5, 6, 8]
    assert kth == float(np.float32(1e-45))
    # the -0 + -0 = -0 at j = 4 stays -0 in the residual when not selected
    assert bits(r)[4] == 0x80000000


def test_all_nan_selects_nothing():
    g = np.full(7, np.nan, np.float32)
    r = np.zeros(7, np.float32)
    idx, val, k, kth = oracle.topk_select(g, r, 0, 7, 0.5, kth=3.5)
    assert k == 0 and kth == 3.5 and np.isnan(r).all()


@pytest.mark.parametrize("seed", range(6))
def test_without_ties_topk_is_the_threshold_rule_at_its_kth_magnitude(seed):
    rng = np.random.default_rng(1000 + seed)
    n = 50000
    g = rng.standard_normal(n).astype(np.float32)
    res = (0.1 * rng.standard_normal(n)).astype(np.float32)
    start, length = 1234, 40000
    r1, r2 = res.copy(), res.copy()
    idx, val, k, kth = oracle.topk_select(g, r1, start, length, 0.01)
    acc = (g + res).astype(np.float32)[start:start + length]
    assert np.sum(np.abs(acc) == np.float32(kth)) == 1  # no tie at the k-th magnitude
    tidx, tval = oracle.select(g, r2, start, length, kth)
    assert np.array_equal(idx, tidx) and np.array_equal(bits(val), bits(tval))
    assert np.array_equal(bits(r1), bits(r2))


@pytest.mark.parametrize("kind", ["normal", "quantised", "laplace"])
def test_order_invariant_and_conservation(kind):
    rng = np.random.default_rng(7)
    n = 20000
    g, res = data(rng, n, kind)
    r = res.copy()
    idx, val, k, kth = oracle.topk_select(g, r, 0, n, 0.05)
    acc = (g + res).astype(np.float32)
    assert k == oracle.topk_count(0.05, n)
    sel = np.zeros(n, bool)
    sel[idx] = True
    assert np.all(np.diff(idx) > 0)
    assert np.abs(acc[sel]).min() >= np.abs(acc[~sel]).max()
    assert np.abs(acc[sel]).min() == np.float32(kth)
    # equal magnitudes: no unselected one has a lower index than a selected one
    tied_out = np.flatnonzero(~sel & (np.abs(acc) == np.float32(kth)))
    tied_in = np.flatnonzero(sel & (np.abs(acc) == np.float32(kth)))
    if tied_out.size:
        assert tied_in.max() < tied_out.min()
    back = r.copy()
    back[idx] = val
    assert np.array_equal(bits(back), bits(acc))


def test_ef_step_is_accumulation_outside_plus_topk_inside():
    rng = np.random.default_rng(11)
    n, world = 30011, 5
    g, res = data(rng, n, "normal")
    for t in range(3):
        r1, r2 = res.copy(), res.copy()
        idx, val, k, th, c = oracle.topk_ef_step(g, r1, t, 2, world, 0.01, 1.0)
        start, length = oracle.partition(n, c, world)
        acc = (g + res).astype(np.float32)
        r2[:start] = acc[:start]
        r2[start + length:] = acc[start + length:]
        want_idx, want_val, want_res, want_kth = numpy_topk(g, r2, start, length, 0.01)
        assert c == (t + 2) % world
        assert np.array_equal(idx, want_idx) and np.array_equal(bits(val), bits(want_val))
        assert np.array_equal(bits(r1), bits(want_res)) and th == want_kth


def test_invalid_arguments():
    g = np.zeros(4, np.float32)
    with pytest.raises(ValueError):
        oracle.topk_select(g, g.copy(), 0, 4, 0.0)
    with pytest.raises(ValueError):
        oracle.topk_select(g, g.copy(), 0, 4, 1.5)
    with pytest.raises(ValueError):
        oracle.topk_select(g, g.copy(), 2, 4, 0.5)


def load_golden():
    out = {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, val = line.split(":", 1)
        out[key.strip()] = val.split()
    return out


def test_golden_worked_example():
    f = load_golden()
    for case in ("a", "b"):
        get = lambda key: f[f"{case}_{key}"]
        n, world, rank = int(get("n_total")[0]), int(get("world")[0]), int(get("rank")[0])
        d = float(get("density")[0])
        g = np.array([float(x) for x in get("grad")], np.float32)
        res = np.array([float(x) for x in get("residual")], np.float32)
        assert g.size == n and res.size == n
        r = res.copy()
        idx, val, k, th = oracle.topk_step(g, r, rank, world, d, 9.0)
        assert k == int(get("k")[0])
        assert list(idx) == [int(x) for x in get("idx")]
        assert np.array_equal(bits(val), bits(np.array([float(x) for x in get("val")], np.float32)))
        assert th == float(get("kth")[0])
        assert np.array_equal(bits(r), bits(np.array([float(x) for x in get("residual_step")], np.float32)))
        if f"{case}_residual_ef" in f:
            r = res.copy()
            idx, val, k, th, c = oracle.topk_ef_step(g, r, 0, rank, world, d, 9.0)
            assert c == rank and list(idx) == [int(x) for x in get("idx")]
            assert np.array_equal(bits(r), bits(np.array([float(x) for x in get("residual_ef")], np.float32)))
