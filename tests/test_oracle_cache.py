"""Pins of the oracle's cache-aware boost signal (paper: interaction with
prefix/radix caching). With h expected cached prompt tokens the effective work
is max(w, P - h); cached tokens are not counted as processed, so the signal is
P - h during the prefill and P - h + dec after it. The engine is unchanged: it
still prefills every prompt token, and h only moves priorities.

The hand-worked schedules (q, q2) live with the others in
tests/golden/hand_worked.json; the per-iteration key and MemGuard guard rules
are replayed in test_oracle_invariants.py. Here: the special cases that reduce
to the plain signal, the range checks, and the generator of the hits.
"""
import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

BOOST = 2


def with_signal(w, signal, cached):
    sets = w.settings.copy()
    boost = sets["policy"] == BOOST
    sets["signal"][boost] = signal
    return W.Workload(w.name, w.arrival_us, w.prompt, w.decode, w.engine, sets, cached=cached)


def assert_same(a, b):
    for key in ("status", "ttft", "ttlt", "tbtmax", "counters", "pct"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_no_hits_is_the_plain_signal(cfg):
    """h = 0 everywhere: P - h + dec is P + dec, so every output equals the
    run with the plain signal."""
    w = W.make(cfg, n_traces=1, n_req=1500, grid="cache")
    zero = np.zeros_like(w.prompt)
    assert_same(oracle.run(with_signal(w, 2, zero)), oracle.run(with_signal(w, 0, None)))


def test_one_level_is_the_plain_signal():
    """k above every signal: all requests sit at level 0 under either signal,
    whatever the hits, so the schedules agree."""
    w = W.make(2, n_traces=1, n_req=1500, grid="cache")
    big = int((w.prompt.astype(np.int64) + w.decode).max()) + 1
    sets = w.settings.copy()
    sets["k"][sets["policy"] == BOOST] = big
    w2 = W.Workload(w.name, w.arrival_us, w.prompt, w.decode, w.engine, sets, cached=w.cached)
    assert_same(oracle.run(with_signal(w2, 2, w.cached)), oracle.run(with_signal(w2, 0, None)))


def test_hits_change_the_schedule():
    """With real hits the cache-aware signal differs from the plain one on a
    loaded trace, and only at BOOST instances (FCFS and SRPT ignore h)."""
    w = W.make(2, n_traces=1, n_req=2000, grid="cache")
    o = oracle.run(w)
    assert np.all(o["status"] == 0)
    s = w.settings
    for i in range(0, 6, 2):  # (plain, cache-aware) pairs
        assert s["signal"][i] == 0 and s["signal"][i + 1] == 2
        assert not np.array_equal(o["ttlt"][i], o["ttlt"][i + 1])
    plain = oracle.run(W.Workload(w.name, w.arrival_us, w.prompt, w.decode, w.engine,
                                  s[6:].copy()))
    assert_same({key: o[key][6:] for key in o if key != "rc"}, plain)


def test_cache_signal_range_checks():
    w = W.make(1, n_traces=1, n_req=300, grid="cache")
    assert oracle.run(w)["rc"] == 0
    for bad in (lambda h: h.__setitem__((0, 5), -1),
                lambda h: h.__setitem__((0, 7), int(w.prompt[0, 7]))):
        h = w.cached.copy()
        bad(h)
        o = oracle.run(W.Workload(w.name, w.arrival_us, w.prompt, w.decode, w.engine,
                                  w.settings, cached=h))
        assert o["rc"] != 0
    o = oracle.run(W.Workload(w.name, w.arrival_us, w.prompt, w.decode, w.engine, w.settings))
    assert o["rc"] != 0  # signal 2 without hits
    sets = w.settings.copy()
    sets["signal"][6] = 2  # FCFS
    o = oracle.run(W.Workload(w.name, w.arrival_us, w.prompt, w.decode, w.engine, sets,
                              cached=w.cached))
    assert o["rc"] != 0
    e = W.Engine()
    r = oracle.log([0], [8], [2], e, BOOST, gamma=1e-3, signal=2, cached=[8])
    assert r["rc"] != 0
    r = oracle.log([0], [8], [2], e, BOOST, gamma=1e-3, signal=2, cached=[7])
    assert r["rc"] == 0


def test_cached_tokens_generator():
    """Follow-up turns keep a new message of at least one token (h < P), first
    turns have no hits, and the draw is seeded and leaves the traces alone."""
    p = W.make(2, n_traces=1, n_req=4000).prompt[0]
    h = W.cached_tokens([2, 0], p)
    assert h.dtype == np.int32 and np.all(h >= 0) and np.all(h < p)
    assert 0.3 < np.mean(h > 0) < 0.5
    assert np.array_equal(h, W.cached_tokens([2, 0], p))
    w = W.make(2, n_traces=1, n_req=4000, grid="cache")
    assert np.array_equal(w.prompt[0], p) and np.array_equal(w.cached[0], h)
