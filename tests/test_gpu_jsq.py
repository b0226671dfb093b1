"""Parity of the join-shortest-queue cluster (paper: composability with global
dispatch policies) on the GPU with the CPU oracle, through the C ABI: one
workgroup per cluster, one wavefront per replica, the router between them.
Exact: the replica of every request, every latency, the per-replica counters
and the cluster's totals and percentiles. Cases: the hand-worked schedules,
2 to 16 replicas under the base and extended policies, the smallest on-chip
list (spills, refills and the retry pass inside replicas)."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "jsq_hand.json")))["cases"]


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def gpu_run(w, **kw):
    from paper_2606_18431_amd import tas

    print(f"[gpu] {w.name} jsq replicas={w.meta.get('replicas')} inst={w.n_inst} "
          f"n_req={w.n_req} {kw}", flush=True)
    sim = tas.Simulation(w, **kw)
    sim.step()
    out = sim.results()
    sim.close()
    return out


def totals(rc):
    """Instance counters from per-replica ones: sums, the latest clock and the
    largest KV peak."""
    out = rc.sum(axis=1)
    out[:, 5] = rc[:, :, 5].max(axis=1)
    out[:, 6] = rc[:, :, 6].max(axis=1)
    return out


def assert_parity(g, o):
    assert np.array_equal(g["status"], o["status"]), (g["status"], o["status"])
    assert np.all(g["status"] == 0)
    for key in ("assign", "ttft", "ttlt", "tbtmax", "pct"):
        if not np.array_equal(g[key], o[key]):
            bad = np.argwhere(g[key] != o[key])[0]
            raise AssertionError(f"{key} differs first at {tuple(bad)}: gpu {g[key][tuple(bad)]} "
                                 f"oracle {o[key][tuple(bad)]}")
    assert np.array_equal(g["rcounters"], o["counters"])
    assert np.array_equal(g["counters"], totals(o["counters"]))
    # per-replica adaptive gamma, bit for bit, and its grid-cell changes
    assert np.array_equal(g["rgamma"].view(np.int64), o["gamma"].view(np.int64))
    assert np.array_equal(g["rswitches"], o["switches"])


@pytest.mark.parametrize("c", GOLDEN, ids=[c["name"] for c in GOLDEN])
def test_jsq_hand_worked_on_gpu(torch, c):
    w = W.Workload(c["name"], np.asarray([c["arrival"]], np.int64),
                   np.asarray([c["prompt"]], np.int32), np.asarray([c["decode"]], np.int32),
                   W.Engine(), np.stack([W.setting(0, c["policy"])]),
                   meta=dict(replicas=c["replicas"], dispatch="jsq"))
    g = gpu_run(w)
    assert g["rc"] == 0
    assert g["assign"][0].tolist() == c["assign"]
    assert g["ttlt"][0].tolist() == c["ttlt"]
    assert g["tbtmax"][0].tolist() == c["tbtmax"]
    assert g["rcounters"][0].tolist() == c["counters"]


SETS = [dict(policy=W.FCFS), dict(policy=W.SRPT), dict(policy=W.BOOST, gamma=1e-3, **W.UNIBOOST),
        dict(policy=W.BOOST, gamma=1e-2, **W.VANILLA), dict(policy=W.SARATHI),
        dict(policy=W.DIST, gamma=1e-3), dict(policy=W.BOOST, gamma=1e-3, signal=1, **W.UNIBOOST),
        dict(policy=W.LAS)]


@pytest.mark.parametrize("cfg,R,n", [(1, 2, 500), (2, 4, 300), (3, 8, 150), (1, 16, 60),
                                     (2, 3, 400)])
def test_parity_jsq(torch, cfg, R, n):
    w = W.make_cluster(cfg, n_clusters=2 if R <= 4 else 1, replicas=R, dispatch="jsq", n_req=n,
                       settings=SETS)
    o = oracle.jsq(w, R)
    g = gpu_run(w)
    assert_parity(g, o)


@pytest.mark.parametrize("cfg,R", [(2, 4), (3, 2)])
def test_parity_jsq_smallest_list(torch, cfg, R):
    w = W.make_cluster(cfg, n_clusters=1, replicas=R, dispatch="jsq", n_req=400, settings=SETS)
    o = oracle.jsq(w, R)
    g = gpu_run(w, list_cap=w.engine.max_seqs + 64)
    assert_parity(g, o)


def test_jsq_large_sweep_law(torch):
    """The large-sweep engine (256 sequences, 16384-token budget) with 8
    replicas: the 512-thread build at its largest list."""
    w = W.make_cluster(4, n_clusters=1, replicas=8, dispatch="jsq", n_req=150, settings=SETS[:4])
    o = oracle.jsq(w, 8)
    g = gpu_run(w)
    assert_parity(g, o)


def test_parity_jsq_cache_signal(torch):
    """The cache-aware signal behind the router: each replica reads the hits
    of the global requests it received."""
    R = 4
    w = W.make_cluster(2, n_clusters=2, replicas=R, dispatch="jsq", n_req=300,
                       settings=[dict(policy=W.BOOST, gamma=1e-3, signal=2, **W.UNIBOOST),
                                 dict(policy=W.BOOST, gamma=1e-2, signal=2, **W.VANILLA)])
    w.cached = np.stack([W.cached_tokens([7, c], w.prompt[c]) for c in range(w.n_traces)])
    o = oracle.jsq(w, R)
    g = gpu_run(w)
    assert_parity(g, o)


@pytest.mark.parametrize("cfg,R", [(2, 4), (3, 2)])
def test_parity_jsq_adaptive_gamma(torch, cfg, R):
    """Adaptive gamma behind the router: every replica runs its own estimate
    from its own completions (small windows, so gamma crosses many cells)."""
    ada = dict(W.ADA, window=40, min_samples=20, beta=0.2)
    w = W.make_cluster(cfg, n_clusters=1, replicas=R, dispatch="jsq", n_req=300,
                       settings=[dict(policy=W.BOOST, gamma=1e-3, ada=ada, **W.UNIBOOST),
                                 dict(policy=W.BOOST, gamma=1e-2, ada=ada, **W.VANILLA),
                                 dict(policy=W.FCFS)])
    o = oracle.jsq(w, R)
    g = gpu_run(w)
    assert_parity(g, o)
    assert np.all(o["switches"][:2] > 0)
