"""Pins of the oracle's comparison policies (paper: Table 1 and the
evaluation's baselines): shortest prefix first (SPF), shortest job first with
perfect output-length knowledge (SJF, the ranking LTR learns), least attained
service (LAS) and SRPT with TRAIL's swap-prevention threshold (TRAIL).

Each pin checks the oracle against something other than itself: optimal orders
over all permutations on a single machine, the defining selection rule
replayed from the oracle's own iteration log, and identities with policies
pinned elsewhere.
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W
from test_oracle_pins import alone_schedule, engine

FCFS, SRPT, BOOST, SPF, SJF, LAS, TRAIL = 0, 1, 2, 3, 4, 5, 6


def job_time(P, D, e):
    return alone_schedule(P, D, e)[1]


def spt_best(p):
    return min(sum(itertools.accumulate(p[i] for i in perm))
               for perm in itertools.permutations(range(len(p))))


@pytest.mark.parametrize("seed", range(8))
def test_sjf_minimizes_total_latency_brute_force(seed):
    """Common release 0, equal prompts, M=1, ample KV: each request's processing
    time grows with D, so ordering by D is SPT, the minimum total TTLT over all
    n! orders; SJF and SRPT then run the same schedule."""
    rng = np.random.default_rng([17, seed])
    n = int(rng.integers(3, 7))
    P = int(rng.integers(16, 200))
    D = rng.integers(1, 40, n).astype(np.int32)
    e = engine(max_seqs=1)
    best = spt_best([job_time(P, int(d), e) for d in D])
    o = oracle.log(np.zeros(n), np.full(n, P), D, e, SJF)
    assert int(o["ttlt"].astype(np.int64).sum()) == best
    s = oracle.log(np.zeros(n), np.full(n, P), D, e, SRPT)
    for key in ("ttft", "ttlt", "tbtmax", "counters"):
        assert np.array_equal(o[key], s[key])


@pytest.mark.parametrize("seed", range(8))
def test_spf_minimizes_total_latency_brute_force(seed):
    """Common release 0, one output token each, M=1, one-chunk prefills: each
    request's time grows with its prompt, so prompt order is SPT."""
    rng = np.random.default_rng([18, seed])
    n = int(rng.integers(3, 7))
    P = rng.integers(1, 1000, n).astype(np.int32)
    e = engine(max_seqs=1)
    best = spt_best([job_time(int(x), 1, e) for x in P])
    o = oracle.log(np.zeros(n), P, np.ones(n, np.int32), e, SPF)
    assert int(o["ttlt"].astype(np.int64).sum()) == best
    # dispatch order is the (prompt, index) order
    order = o["batch"][:, 0].tolist()
    assert order == sorted(range(n), key=lambda i: (int(P[i]), i))


@pytest.mark.parametrize("seed", range(4))
def test_las_serves_least_attained_service(seed):
    """M=1, ample KV, one-chunk prefills: every iteration serves the active
    request with the least attained service P + dec (ties by index)."""
    a, p, d = W.small_random(seed, 60, rate_per_s=30.0)
    e = engine(max_seqs=1, chunk=1024)
    o = oracle.log(a, p, d, e, LAS)
    assert o["rc"] == 0
    dec = np.zeros(len(a), np.int64)
    done = np.zeros(len(a), bool)
    for row, it in enumerate(o["iters"]):
        assert it[2] == 1
        r = int(o["batch"][row][0])
        active = [i for i in range(len(a)) if a[i] <= it[0] and not done[i]]
        assert r == min(active, key=lambda i: (int(p[i]) + int(dec[i]), i))
        dec[r] += 1
        done[r] = dec[r] == d[r]


@pytest.mark.parametrize("seed", range(4))
def test_trail_equals_srpt_without_kv_pressure(seed):
    """The threshold only restricts victims: with KV for everyone (no eviction
    can happen) TRAIL and SRPT run the same schedule."""
    a, p, d = W.small_random(seed, 150, rate_per_s=60.0)
    e = engine(max_seqs=6, chunk=128, max_tokens=384)
    t = oracle.log(a, p, d, e, TRAIL)
    s = oracle.log(a, p, d, e, SRPT)
    assert t["counters"][3] == 0 and t["counters"][4] == 0
    for key in ("ttft", "ttlt", "tbtmax", "counters"):
        assert np.array_equal(t[key], s[key])


def test_trail_never_preempts_past_threshold():
    """Replayed from the log under KV pressure: no voluntary victim had emitted
    0.6 of its output (5 dec >= 3 D); some evictions do happen."""
    a, p, d = W.small_random(5, 200, rate_per_s=80.0, p_max=300, d_max=150)
    e = engine(max_seqs=8, kv_blocks=40, chunk=64, max_tokens=256)
    o = oracle.log(a, p, d, e, TRAIL)
    assert o["rc"] == 0
    kv = np.zeros(len(a), np.int64)
    dec = np.zeros(len(a), np.int64)
    ev = o["evict"]
    ep, row, vol = 0, 0, 0
    for i, it in enumerate(o["iters"]):
        while ep < len(ev) and ev[ep][0] == i:
            _, v, forced, _ = ev[ep]
            ep += 1
            if not forced:
                assert 5 * dec[v] < 3 * d[v]
                vol += 1
            kv[v] = 0
        for r, n in o["batch"][row:row + it[2]]:
            kv[r] += n
            if kv[r] == p[r] + dec[r]:
                dec[r] += 1
                if dec[r] == d[r]:
                    kv[r] = 0
        row += it[2]
    assert vol > 0
    s = oracle.log(a, p, d, e, SRPT)
    assert not np.array_equal(s["counters"], o["counters"])  # the threshold changed something


@pytest.mark.parametrize("policy,blind,kw", [
    (SPF, True, {}), (LAS, True, {}), (SJF, False, {}),
    (W.DIST, True, dict(k=1, gamma=1e-3)), (W.DIST, True, dict(k=16, gamma=3e-2)),
    (W.BOOST, True, dict(k=16, memguard=1, delta_us=20000, gamma=1e-3, signal=1)),
    (W.SARATHI, True, {})])
def test_blindness(policy, blind, kw):
    """SPF, LAS, DistBoost, Sarathi and the boost with the phase-aware signal
    use no knowledge of the output length (prediction-free): lengthening one
    request's decode leaves every event before its original completion
    unchanged. SJF reads the length."""
    changed = 0
    for seed in range(4):
        a, p, d = W.small_random(seed, 120, rate_per_s=60.0)
        e = engine(max_seqs=4, kv_blocks=80, chunk=128, max_tokens=384)
        j = 17
        d2 = d.copy()
        d2[j] += 500
        o1 = oracle.log(a, p, d, e, policy, **kw)
        o2 = oracle.log(a, p, d2, e, policy, **kw)
        ends = np.cumsum(o1["iters"][:, 2])
        last = max(i for i in range(len(ends))
                   if j in o1["batch"][(ends[i] - o1["iters"][i, 2]):ends[i], 0])
        same = (np.array_equal(o1["iters"][: last + 1], o2["iters"][: last + 1])
                and np.array_equal(o1["batch"][: ends[last]], o2["batch"][: ends[last]]))
        if blind:
            assert same
        changed += not same
    if not blind:
        assert changed > 0



@pytest.mark.parametrize("seed", range(4))
def test_sarathi_is_distboost_without_contention(seed):
    """With the batch cap above the number of requests and KV to spare, every
    decode is in every batch, so the order inside the decode queue (latest
    token for Sarathi, first token for DistBoost) cannot matter: Sarathi
    equals DistBoost with a zero boost table (prefills in arrival order),
    bit for bit. Under contention (M = 8, KV pressure) they differ, and
    Sarathi differs from FCFS (evicted decodes return ahead of prefills)."""
    a, p, d = W.small_random(seed, 150, rate_per_s=40.0)
    e = engine(max_seqs=256, kv_blocks=100000, chunk=128, max_tokens=4096)
    zero = np.zeros(24, np.int64)
    s = oracle.log(a, p, d, e, W.SARATHI)
    t = oracle.log(a, p, d, e, W.DIST, table=zero)
    assert s["rc"] == 0 and t["rc"] == 0
    for key in ("ttft", "ttlt", "tbtmax", "counters"):
        assert np.array_equal(s[key], t[key]), key
    e2 = engine(max_seqs=8, kv_blocks=60, chunk=128, max_tokens=4096)
    s2 = oracle.log(a, p, d, e2, W.SARATHI)
    t2 = oracle.log(a, p, d, e2, W.DIST, table=zero)
    f2 = oracle.log(a, p, d, e2, FCFS)
    assert not np.array_equal(s2["ttlt"], t2["ttlt"])
    assert not np.array_equal(s2["ttlt"], f2["ttlt"])


# ------------------------------------------------------------ SJF (LTR+)


def test_ltr_without_reachable_threshold_is_sjf():
    """SJF (LTR+) whose starvation threshold no wait reaches is plain SJF, bit
    for bit (the promotion is the only difference)."""
    import dataclasses

    w = W.make(2, n_traces=1, n_settings=4, n_req=800)
    sjf = w.settings.copy()
    sjf["policy"], sjf["k"], sjf["memguard"], sjf["delta_us"] = W.SJF, 1, 0, 0
    ltr = sjf.copy()
    ltr["policy"], ltr["ltr_starve"], ltr["ltr_quantum"] = W.LTR, 1 << 30, 7
    a = oracle.run(dataclasses.replace(w, settings=sjf))
    b = oracle.run(dataclasses.replace(w, settings=ltr))
    assert a["rc"] == 0 and b["rc"] == 0
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct"):
        assert np.array_equal(a[key], b[key]), key


@pytest.mark.parametrize("S,Q", [(3, 1), (6, 4), (20, 10)])
def test_ltr_bounds_unserved_streaks(S, Q):
    """Under LTR+ an unpromoted request is promoted after S iterations without
    service, and a promoted one ranks ahead of every unpromoted request: at
    most M - 1 promoted requests (the batch) ahead of it can keep it waiting
    each iteration. So, with a batch of one, a request never waits more than
    S + (promoted requests ahead) * Q iterations in a row; the replay of the
    schedule finds the streaks, and SJF exceeds the bound on the same trace."""
    a, p, d = W.small_random(5, 200, rate_per_s=80.0, p_max=300, d_max=120)
    e = W.Engine(max_seqs=1, max_tokens=1024, chunk=512, kv_blocks=4096)

    def longest_wait(o):
        N = len(a)
        t0s = o["iters"][:, 0]
        rows = np.cumsum(np.r_[0, o["iters"][:, 2]])
        served = [set(o["batch"][rows[i]:rows[i + 1], 0].tolist()) for i in range(len(t0s))]
        done_at = {}
        for i in range(len(t0s)):
            for r in served[i]:
                done_at[r] = i
        worst = 0
        for r in range(N):
            run = 0
            for i in range(len(t0s)):
                if t0s[i] < a[r] or i > done_at[r]:
                    continue
                run = 0 if r in served[i] else run + 1
                worst = max(worst, run)
        return worst

    o = oracle.log(a, p, d, e, W.LTR, ltr=(S, Q))
    s = oracle.log(a, p, d, e, W.SJF)
    assert o["rc"] == 0 and s["rc"] == 0
    bound = S + len(a) * Q  # loose: promoted requests ahead, each served Q times
    assert longest_wait(o) <= bound
    assert longest_wait(o) < longest_wait(s)
    assert not np.array_equal(o["ttlt"], s["ttlt"])


def test_ltr_rejects_bad_control():
    e = W.Engine()
    for bad in ((0, 4), (4, 0), (-1, 1)):
        o = oracle.log([0, 0], [16, 16], [2, 2], e, W.LTR, ltr=bad)
        assert o["rc"] == oracle.EINVAL, bad
    o = oracle.log([0, 0], [16, 16], [2, 2], e, W.LTR)  # no control given
    assert o["rc"] == oracle.EINVAL
