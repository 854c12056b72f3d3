"""The seeded synthetic inputs (CPU): model layouts, determinism and the
initial-threshold calibration."""
import math

import numpy as np
import pytest
import torch

from paper_2310_00967_amd import synth

# parameter counts of the published architectures the layouts follow
EXPECTED = {"toy": (1, 1_048_576), "resnet18": (62, 11_689_512), "resnet50": (161, 25_557_032),
            "bert_large": (391, 335_141_888), "gpt_1p3b": (292, 1_315_723_264)}


@pytest.mark.parametrize("name", sorted(EXPECTED))
def test_layouts(name):
    w = synth.get(name)
    tensors, n = EXPECTED[name]
    assert len(w.shapes) == tensors
    assert w.n_total == n == synth.N_TOTAL[name]


def test_gradients_are_seeded_per_step():
    w = synth.get("resnet18", shrink=64)
    a0, a0b, a1 = synth.gradient(w, 0), synth.gradient(w, 0), synth.gradient(w, 1)
    assert torch.equal(a0, a0b)
    assert not torch.equal(a0, a1)
    assert a0.dtype == torch.float32 and a0.numel() == w.n_total


def test_frozen_tensors_are_zero():
    w = synth.get("bert_large", shrink=512)
    g = synth.gradient(w, 3)
    _, frozen = synth.tensor_scales(w)
    assert frozen.sum() == 4
    off = 0
    for size, fz in zip(w.sizes, frozen):
        seg = g[off:off + size]
        assert bool((seg == 0).all()) == bool(fz) or size == 1
        off += size


@pytest.mark.parametrize("n", [1, 2, 7, 1000, 65_537])
@pytest.mark.parametrize("density", [0.001, 0.01, 0.3, 1.0])
def test_calibration_is_the_kth_largest_magnitude(n, density):
    rng = np.random.default_rng(n)
    g = torch.from_numpy((rng.standard_normal(n) * rng.uniform(1e-6, 10)).astype(np.float32))
    start, end = n // 5, n
    th = synth.calibrate_theta0(g, start, end, density)
    P = end - start
    K = max(1, int(math.floor(density * P)))
    want = float(np.sort(np.abs(g.numpy()[start:end]))[::-1][K - 1])
    assert th == want
