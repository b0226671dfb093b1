"""Replicas behind a global router (paper: global dispatch policies, cluster
scale): the round-robin and balanced-random dispatch of workloads.make_cluster,
and cluster percentiles pooled over a group of replicas (the oracle side of
tas_percentiles_grouped). CPU only."""
import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import tas
from paper_2606_18431_amd import workloads as W


@pytest.mark.parametrize("dispatch", ["rr", "random"])
@pytest.mark.parametrize("R", [1, 3, 8])
def test_dispatch_partitions_the_global_trace(dispatch, R):
    N = 200
    w = W.make_cluster(1, n_clusters=2, replicas=R, dispatch=dispatch, n_req=N)
    assign = w.meta["assign"]
    for c in range(2):
        rep = assign[c]
        # every replica receives N requests; balanced random: each block of R is a permutation
        assert np.array_equal(np.bincount(rep, minlength=R), np.full(R, N))
        blocks = rep.reshape(N, R)
        if dispatch == "rr":
            assert np.array_equal(rep, np.arange(N * R) % R)
        else:
            assert all(np.array_equal(np.sort(b), np.arange(R)) for b in blocks)
        # the replicas' traces are the global trace split by the assignment
        merged_a = np.empty(N * R, np.int64)
        merged_p = np.empty(N * R, np.int32)
        for r in range(R):
            sel = np.nonzero(rep == r)[0]
            merged_a[sel] = w.arrival_us[c * R + r]
            merged_p[sel] = w.prompt[c * R + r]
            assert np.all(np.diff(w.arrival_us[c * R + r]) >= 0)
        assert np.all(np.diff(merged_a) >= 0)
        # the same lengths as the one-server trace of N*R requests, R times faster
        a1, p1, d1 = W._trace(1, c, N * R, w.engine)
        assert np.array_equal(merged_p, p1)
        assert np.array_equal(merged_a, a1 // R)
    if dispatch == "random" and R > 1:
        assert not np.array_equal(assign[0], np.arange(N * R) % R)


def test_single_replica_is_the_plain_workload():
    w = W.make_cluster(2, n_clusters=2, replicas=1, n_req=300,
                       settings=[dict(policy=W.BOOST, gamma=1e-3, **W.UNIBOOST)])
    plain = W.make(2, n_traces=2, n_req=300)
    assert np.array_equal(w.arrival_us, plain.arrival_us)
    assert np.array_equal(w.prompt, plain.prompt) and np.array_equal(w.decode, plain.decode)


def test_group_percentiles():
    w = W.make_cluster(1, n_clusters=1, replicas=4, dispatch="random", n_req=250)
    o = oracle.run(w, n_threads=4)
    assert o["rc"] == 0
    assert np.array_equal(oracle.group_percentiles(o, 1), o["pct"])
    g = oracle.group_percentiles(o, 4)
    assert g.shape == (w.meta["n_settings"], 3, 3)
    for s in range(w.meta["n_settings"]):
        for m, key in enumerate(("ttft", "ttlt", "tbtmax")):
            pooled = o[key][s * 4:(s + 1) * 4].ravel().astype(np.float64)
            ref = [np.quantile(pooled, q / 100, method="inverted_cdf") for q in (50, 90, 99)]
            assert g[s, m].tolist() == ref


def test_grouped_percentiles_rejects_without_context():
    with pytest.raises(tas.TasError):
        tas.tas_percentiles_grouped(None, 4, np.zeros(9, np.uint32))
