"""Seeded synthetic gradients shaped like the paper's models.

This module is the only code shared by the GPU path's tests and benchmark and
the CPU oracle's tests.  It holds none of the sparsifier's arithmetic: it only
lays out model-shaped flattened gradient vectors and draws their values.

The paper trains ResNet-18, GoogLeNet and SENet-18 on CIFAR-10/100 (Sec. 5.1,
Table 2); no dataset or trained model is available here, so seeded synthetic
gradients with the parameter layouts of ResNet-18, ResNet-50, BERT-large and a
1.3B-parameter GPT stand in for them:

* toy        -- 1,048,576 i.i.d. N(0, 1) values; world 4, rank 0; d = 0.01;
                initial threshold 2.33; 20 steps.
* resnet18   -- 62 tensors (torchvision ResNet-18 parameter order), 11,689,512
                values, N(0, s_j) with s_j log-uniform in [1e-4, 1e-1]; world 16,
                every rank swept each step; d = 0.01; 100 steps.
* resnet50   -- 161 tensors, 25,557,032 values, Laplace(0, b_j) with b_j
                log-uniform in [1e-5, 1e-2]; world 8, rank 0; d = 0.001; 100 steps.
* bert_large -- 391 tensors (BERT-large with pooler), 335,141,888 values,
                s_j * t_3 (Student t, 3 degrees of freedom) with s_j
                log-uniform in [1e-5, 1e-2]; 1% of the tensors (4) are all zero
                (frozen); world 8, rank 3; d = 0.01; 50 steps.
* gpt_1p3b   -- 292 tensors (24 layers, hidden 2048, FFN 8192, 50257 x 2048 tied
                embedding, 2048 learned positions), 1,315,723,264 values,
                N(0, s_j) with s_j log-uniform in [1e-6, 1e-2]; world 1;
                d = 0.001 and d = 0.01; 20 steps each.

Values of step t come from a generator seeded with SEED + t on the device the
gradient is drawn on; per-tensor scales and the frozen-tensor choice come once
from numpy's PCG64 seeded with SEED.  The initial threshold of every workload
but the toy is calibrated as the K-th largest magnitude of the step-0 gradient
inside the partition, K = max(1, floor(d * P)).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np
import torch

SEED = 231000967
CHUNK = 1 << 26  # values drawn per generator call (fixed, so draws are reproducible)


# --------------------------------------------------------------------------
# parameter layouts (registration order of the published architectures)
# --------------------------------------------------------------------------

def resnet18_shapes():
    shapes = [(64, 3, 7, 7), (64,), (64,)]
    inplanes = 64
    for planes, stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        for b in range(2):
            cin = inplanes if b == 0 else planes
            shapes += [(planes, cin, 3, 3), (planes,), (planes,),
                       (planes, planes, 3, 3), (planes,), (planes,)]
            if b == 0 and (stride != 1 or inplanes != planes):
                shapes += [(planes, inplanes, 1, 1), (planes,), (planes,)]
        inplanes = planes
    shapes += [(1000, 512), (1000,)]
    return shapes


def resnet50_shapes():
    shapes = [(64, 3, 7, 7), (64,), (64,)]
    inplanes = 64
    for planes, blocks in ((64, 3), (128, 4), (256, 6), (512, 3)):
        for b in range(blocks):
            cin = inplanes if b == 0 else planes * 4
            shapes += [(planes, cin, 1, 1), (planes,), (planes,),
                       (planes, planes, 3, 3), (planes,), (planes,),
                       (planes * 4, planes, 1, 1), (planes * 4,), (planes * 4,)]
            if b == 0:
                shapes += [(planes * 4, inplanes, 1, 1), (planes * 4,), (planes * 4,)]
        inplanes = planes * 4
    shapes += [(1000, 2048), (1000,)]
    return shapes


def bert_large_shapes(vocab=30522, hidden=1024, ffn=4096, layers=24, positions=512):
    shapes = [(vocab, hidden), (positions, hidden), (2, hidden), (hidden,), (hidden,)]
    for _ in range(layers):
        for _qkv_out in range(4):  # query, key, value, attention output
            shapes += [(hidden, hidden), (hidden,)]
        shapes += [(hidden,), (hidden,)]          # attention LayerNorm
        shapes += [(ffn, hidden), (ffn,)]         # intermediate
        shapes += [(hidden, ffn), (hidden,)]      # output
        shapes += [(hidden,), (hidden,)]          # output LayerNorm
    shapes += [(hidden, hidden), (hidden,)]       # pooler
    return shapes


def gpt_shapes(vocab=50257, hidden=2048, ffn=8192, layers=24, positions=2048):
    shapes = [(vocab, hidden), (positions, hidden)]
    for _ in range(layers):
        shapes += [(hidden,), (hidden,),                     # ln_1
                   (hidden, 3 * hidden), (3 * hidden,),      # fused qkv
                   (hidden, hidden), (hidden,),              # attention projection
                   (hidden,), (hidden,),                     # ln_2
                   (hidden, ffn), (ffn,),                    # MLP in
                   (ffn, hidden), (hidden,)]                 # MLP out
    shapes += [(hidden,), (hidden,)]                         # final LayerNorm
    return shapes


# --------------------------------------------------------------------------
# workloads
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shapes: tuple
    dist: str                  # "normal", "laplace", "student_t3"
    scale_range: tuple         # (lo, hi) of the log-uniform per-tensor scale; None = unit
    world: int
    ranks: tuple               # ranks run each step, in this order
    densities: tuple
    steps: int
    theta0: float | None       # None = calibrated from the step-0 gradient
    frozen_frac: float = 0.0

    @property
    def sizes(self):
        return [int(np.prod(s)) for s in self.shapes]

    @property
    def n_total(self):
        return sum(self.sizes)


def _workloads():
    return {
        "toy": Workload("toy", ((1 << 20,),), "normal", None, 4, (0,), (0.01,), 20, 2.33),
        "resnet18": Workload("resnet18", tuple(resnet18_shapes()), "normal", (1e-4, 1e-1),
                             16, tuple(range(16)), (0.01,), 100, None),
        "resnet50": Workload("resnet50", tuple(resnet50_shapes()), "laplace", (1e-5, 1e-2),
                             8, (0,), (0.001,), 100, None),
        "bert_large": Workload("bert_large", tuple(bert_large_shapes()), "student_t3",
                               (1e-5, 1e-2), 8, (3,), (0.01,), 50, None, frozen_frac=0.01),
        "gpt_1p3b": Workload("gpt_1p3b", tuple(gpt_shapes()), "normal", (1e-6, 1e-2),
                             1, (0,), (0.001, 0.01), 20, None),
    }


WORKLOADS = _workloads()

N_TOTAL = {"toy": 1_048_576, "resnet18": 11_689_512, "resnet50": 25_557_032,
           "bert_large": 335_141_888, "gpt_1p3b": 1_315_723_264}


def get(name, shrink=1):
    """Returns the named workload; shrink > 1 divides every tensor's size by
    `shrink` (keeping at least one value per tensor) for small CPU runs."""
    w = WORKLOADS[name]
    if shrink == 1:
        return w
    shapes = tuple((max(1, int(np.prod(s)) // shrink),) for s in w.shapes)
    return dataclasses.replace(w, shapes=shapes)


def tensor_scales(w):
    """Per-tensor scale and frozen flags, drawn once from SEED on the CPU."""
    rng = np.random.Generator(np.random.PCG64(SEED))
    m = len(w.shapes)
    if w.scale_range is None:
        scales = np.ones(m)
    else:
        lo, hi = w.scale_range
        scales = np.exp(rng.uniform(math.log(lo), math.log(hi), size=m))
    frozen = np.zeros(m, dtype=bool)
    n_frozen = int(round(w.frozen_frac * m))
    if n_frozen:
        frozen[rng.choice(m, size=n_frozen, replace=False)] = True
    return scales, frozen


def _draw(dist, n, gen, device):
    """n unit-scale values of the workload's distribution, in fixed-size chunks."""
    out = torch.empty(n, dtype=torch.float32, device=device)
    for off in range(0, n, CHUNK):
        m = min(CHUNK, n - off)
        seg = out[off:off + m]
        if dist == "normal":
            seg.normal_(generator=gen)
        elif dist == "laplace":
            e2 = torch.empty(m, dtype=torch.float32, device=device)
            seg.exponential_(generator=gen)
            e2.exponential_(generator=gen)
            seg.sub_(e2)
        elif dist == "student_t3":
            seg.normal_(generator=gen)
            chi = torch.zeros(m, dtype=torch.float32, device=device)
            z = torch.empty(m, dtype=torch.float32, device=device)
            for _ in range(3):
                z.normal_(generator=gen)
                chi.addcmul_(z, z)
            seg.div_(torch.sqrt(chi.div_(3.0)))
        else:
            raise ValueError(dist)
    return out


def gradient(w, t, device="cpu", out=None):
    """The flattened fp32 gradient of step t (seed SEED + t) on `device`."""
    device = torch.device(device)
    gen = torch.Generator(device=device)
    gen.manual_seed(SEED + int(t))
    g = _draw(w.dist, w.n_total, gen, device)
    scales, frozen = tensor_scales(w)
    off = 0
    for size, s, fz in zip(w.sizes, scales, frozen):
        seg = g[off:off + size]
        if fz:
            seg.zero_()
        elif s != 1.0:
            seg.mul_(float(s))
        off += size
    if out is not None:
        out.copy_(g)
        return out
    return g


def calibrate_theta0(g, start, end, density):
    """Initial threshold: the K-th largest magnitude in g[start:end),
    K = max(1, floor(density * P)), as a Python float (exact widening).

    Found by bisection over the bit patterns of non-negative binary32 values,
    which order like the integers: the largest x with #{|g| >= x} >= K is the
    K-th largest magnitude.  31 counting passes on the tensor's device."""
    P = end - start
    if P <= 0:
        return 1.0
    K = max(1, int(math.floor(density * P)))
    mag = g[start:end].abs()
    lo, hi = 0, 0x7F800000  # +0 .. +inf
    probe = torch.empty(1, dtype=torch.int32)
    while lo < hi:
        mid = (lo + hi + 1) // 2
        probe[0] = mid
        x = float(probe.view(torch.float32)[0])
        if int((mag >= x).sum()) >= K:
            lo = mid
        else:
            hi = mid - 1
    probe[0] = lo
    return float(probe.view(torch.float32)[0])


def initial_theta(w, g0, start, end, density):
    """The workload's initial threshold for the range [start, end) (the caller
    supplies the partition bounds)."""
    if w.theta0 is not None:
        return float(w.theta0)
    th = calibrate_theta0(g0, start, end, density)
    return th if th > 0.0 else 1e-30
