"""Replicas behind a global router on the GPU (paper: global dispatch
policies, cluster scale): every replica instance exactly equal to the CPU
oracle, and the cluster percentiles of tas_percentiles_grouped (pooled over
the R adjacent replica instances) equal to the oracle's pooled nearest-rank
values; with group 1 it equals tas_percentiles."""
import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.mark.parametrize("cfg,R,dispatch", [(1, 4, "rr"), (1, 8, "random"), (2, 4, "random"),
                                            (4, 8, "rr")])
def test_cluster_parity(torch, cfg, R, dispatch):
    from paper_2606_18431_amd import tas

    w = W.make_cluster(cfg, n_clusters=2, replicas=R, dispatch=dispatch, n_req=1500)
    print(f"[gpu] cluster cfg {cfg} R={R} {dispatch}: {w.n_inst} instances", flush=True)
    sim = tas.Simulation(w)
    sim.step()
    g = sim.results()
    gp = sim.group_percentiles(R)
    g1 = sim.group_percentiles(1)
    sim.close()
    o = oracle.run(w)
    assert g["rc"] == 0 and o["rc"] == 0
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct"):
        assert np.array_equal(g[key], o[key]), key
    assert np.array_equal(g1, g["pct"])
    assert np.array_equal(gp, oracle.group_percentiles(o, R))
