"""The hand-worked example of Algorithm 1 (tests/golden/): the oracle on the
CPU and the HIP library on the GPU must both reproduce it exactly."""
import numpy as np
import pytest

import oracle
from golden_fixture import load

G = load()


def rule():
    return oracle.make_rule(oracle.PROPORTIONAL, beta=G["beta"], lo=G["lo"], hi=G["hi"])


def test_oracle_reproduces_the_worked_example():
    res = np.zeros(G["n_total"], np.float32)
    theta = G["theta0"]
    for t in range(3):
        idx, val, k, theta, c = oracle.ef_step(G[f"grad_{t}"], res, t, G["worker"], G["world"], G["density"],
                                               theta, rule=rule())
        assert c == G[f"cycle_{t}"]
        assert np.array_equal(idx, G[f"idx_{t}"]) and np.array_equal(val, G[f"val_{t}"])
        assert np.array_equal(res, G[f"residual_{t}"])
        assert theta == G[f"theta_{t + 1}"]
        assert oracle.sumsq(res) == G[f"sumsq_{t}"]


def test_oracle_reproduces_the_worked_exchange():
    acc = oracle.accumulate(G["grad_0"], np.zeros(G["n_total"], np.float32))
    got = oracle.gather(acc, G["union"])
    assert np.array_equal(got, G["union_gathered"])
    oracle.zero(acc, G["union"])
    # acc was also reset at the worker's own selection, as the pass does
    assert np.array_equal(acc, G["union_residual"])
    x = G["union_x0"].copy()
    oracle.update(x, G["union"], G["union_sums"], G["world"])
    assert np.array_equal(x, G["union_x1"])


@pytest.mark.gpu
def test_library_reproduces_the_worked_example():
    import torch
    import paper_2310_00967_amd as micro
    N = G["n_total"]
    sp = micro.Sparsifier(N, device="cuda", beta=G["beta"], lo=G["lo"], hi=G["hi"])
    res = torch.zeros(N, dtype=torch.float32, device="cuda")
    theta = G["theta0"]
    for t in range(3):
        g = torch.from_numpy(G[f"grad_{t}"]).to("cuda")
        k, theta, c, idx, val, sq = sp.ef_step(g, res, t, G["worker"], G["world"], G["density"], theta,
                                               local_error=True)
        assert c == G[f"cycle_{t}"]
        assert np.array_equal(idx.cpu().numpy(), G[f"idx_{t}"])
        assert np.array_equal(val.cpu().numpy(), G[f"val_{t}"])
        assert np.array_equal(res.cpu().numpy(), G[f"residual_{t}"])
        assert theta == G[f"theta_{t + 1}"]
        assert sq == G[f"sumsq_{t}"]
    # the exchange after the pass of t = 0
    res = torch.zeros(N, dtype=torch.float32, device="cuda")
    g0 = torch.from_numpy(G["grad_0"]).to("cuda")
    k, th, c, idx, val = sp.ef_step(g0, res, 0, G["worker"], G["world"], G["density"], G["theta0"])
    union = torch.from_numpy(G["union"]).to("cuda")
    out = sp.union_gather(res, union, G["union_own_first"], val.clone())
    x = torch.from_numpy(G["union_x0"]).to("cuda")
    sums = torch.from_numpy(G["union_sums"]).to("cuda")
    sp.sparse_update(x, union, sums, G["world"])
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), G["union_gathered"])
    assert np.array_equal(res.cpu().numpy(), G["union_residual"])
    assert np.array_equal(x.cpu().numpy(), G["union_x1"])
    sp.close()
