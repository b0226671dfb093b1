"""Pins of the oracle's join-shortest-queue cluster (paper: composability
with global dispatch policies). Checked against a hand-worked schedule, the
single-replica special case, an independent replay of every routing decision
from the outputs, and the per-replica schedules recomputed as plain
instances."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "jsq_hand.json")))["cases"]


def one_trace(arrival, prompt, decode, settings, engine=None):
    return W.Workload("jsq", np.asarray([arrival], np.int64), np.asarray([prompt], np.int32),
                      np.asarray([decode], np.int32), engine or W.Engine(), np.stack(settings))


@pytest.mark.parametrize("c", GOLDEN, ids=[c["name"] for c in GOLDEN])
def test_jsq_hand_worked(c):
    w = one_trace(c["arrival"], c["prompt"], c["decode"], [W.setting(0, c["policy"])])
    o = oracle.jsq(w, c["replicas"])
    assert o["rc"] == 0
    assert o["assign"][0].tolist() == c["assign"]
    assert o["ttft"][0].tolist() == c["ttft"]
    assert o["ttlt"][0].tolist() == c["ttlt"]
    assert o["tbtmax"][0].tolist() == c["tbtmax"]
    assert o["counters"][0].tolist() == c["counters"]


def cluster(cfg, replicas, n_req, settings=None):
    return W.make_cluster(cfg, n_clusters=1, replicas=replicas, dispatch="jsq", n_req=n_req,
                          settings=settings)


SETS = [dict(policy=W.FCFS), dict(policy=W.BOOST, gamma=1e-3, **W.UNIBOOST),
        dict(policy=W.SARATHI), dict(policy=W.SRPT)]


@pytest.mark.parametrize("cfg", [1, 2])
def test_one_replica_is_the_plain_instance(cfg):
    w = W.make(cfg, n_traces=1, n_req=500, grid="comparators")
    j = oracle.jsq(w, 1)
    p = oracle.run(w)
    assert np.array_equal(j["status"], p["status"])
    ok = p["status"] == 0
    for key in ("ttft", "ttlt", "tbtmax", "pct"):
        assert np.array_equal(j[key][ok], p[key][ok]), key
    assert np.array_equal(j["counters"][ok, 0], p["counters"][ok])
    assert np.all(j["assign"] == 0)


def replay_router(arrival, assign, ttlt, R):
    """Each request's replica must hold the fewest requests not completed by
    its arrival (completion = arrival + TTLT), ties to the lowest replica."""
    done = arrival.astype(np.int64) + ttlt.astype(np.int64)
    for j in range(len(arrival)):
        held = [int(np.sum((assign[:j] == r) & (done[:j] > arrival[j]))) for r in range(R)]
        assert assign[j] == int(np.argmin(held)), (j, held, assign[j])


@pytest.mark.parametrize("cfg,R", [(1, 2), (2, 4), (3, 3)])
def test_router_replay_and_replicas_as_plain_instances(cfg, R):
    w = cluster(cfg, R, 400, SETS)
    o = oracle.jsq(w, R)
    assert o["rc"] == 0
    a, p, d = w.arrival_us[0], w.prompt[0], w.decode[0]
    for i in range(w.n_inst):
        replay_router(a, o["assign"][i], o["ttlt"][i], R)
        counts = np.bincount(o["assign"][i], minlength=R)
        assert counts.min() > 0
        for r in range(R):
            sel = np.nonzero(o["assign"][i] == r)[0]
            sub = W.Workload("replica", a[sel][None], p[sel][None], d[sel][None], w.engine,
                             w.settings[i:i + 1].copy())
            q = oracle.run(sub)
            assert q["rc"] == 0
            for key in ("ttft", "ttlt", "tbtmax"):
                assert np.array_equal(q[key][0], o[key][i][sel]), (i, r, key)
            assert np.array_equal(q["counters"][0], o["counters"][i, r])


def test_jsq_balances_better_than_round_robin():
    """At the same offered load (the bursty trace), the router that sees the
    queues gives a lower mean and P99 TTLT than round robin (FCFS in every
    replica); a sanity check on one seeded trace, not a theorem."""
    R, n = 4, 250
    w = cluster(3, R, n, [dict(policy=W.FCFS)])
    j = oracle.jsq(w, R)
    rr = W.make_cluster(3, n_clusters=1, replicas=R, dispatch="rr", n_req=n,
                        settings=[dict(policy=W.FCFS)])
    o = oracle.run(rr)
    assert j["ttlt"].astype(np.float64).mean() < o["ttlt"].astype(np.float64).mean()
    assert j["pct"][0, 1, 2] < oracle.percentile(o["ttlt"].ravel(), 99)


def test_jsq_rejects():
    w = one_trace([0, 5], [4, 4], [2, 2], [W.setting(0, W.FCFS)])
    assert oracle.jsq(w, 0)["rc"] != 0
    bad = one_trace([5, 0], [4, 4], [2, 2], [W.setting(0, W.FCFS)])
    assert oracle.jsq(bad, 2)["rc"] != 0


def test_fast_router_replay_agrees_with_the_slow_one():
    """The vectorised replay that checks the full-size GPU clusters accepts
    the oracle's routing and rejects any single changed decision."""
    from test_gpu_fullsize import replay_router_fast

    R = 4
    w = cluster(2, R, 200, [dict(policy=W.FCFS), dict(policy=W.BOOST, gamma=1e-3, **W.UNIBOOST)])
    o = oracle.jsq(w, R)
    a = w.arrival_us[0]
    rng = np.random.default_rng(3)
    for i in range(w.n_inst):
        asg, ttlt = o["assign"][i], o["ttlt"][i]
        replay_router(a, asg, ttlt, R)
        assert replay_router_fast(a, asg, ttlt, R)
        for j in rng.choice(len(a), 20, replace=False):
            bad = asg.copy()
            bad[j] = (bad[j] + 1 + rng.integers(R - 1)) % R
            assert not replay_router_fast(a, bad, ttlt, R), j
