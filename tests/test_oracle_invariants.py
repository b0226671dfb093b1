"""Invariants of the serving simulation, checked on the oracle's schedule log.

The replay below rebuilds every request's KV, emitted tokens and timestamps
from the logged batches and evictions alone, re-derives each iteration's
duration from the cost model, and checks the result against the oracle's
outputs and the rules: KV capacity, batch limits, work conservation, token
conservation, completion exactly once, FCFS dispatch order, every batch in
ascending (key, idx) order of the policy's keys, the MemGuard eligibility of
every voluntary eviction and the Phase 3 revision bound.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W


def blocks(x, bs):
    return -(-x // bs)


def sig_of(r, p, dec, signal, h=None):
    """The boost signal: P + dec, or (signal 1) P in prefill and dec in decode,
    or (signal 2) P - h + dec with h the expected cached prompt tokens."""
    if signal == 1:
        return int(p[r]) if dec[r] == 0 else int(dec[r])
    if signal == 2:
        return int(p[r]) - int(h[r]) + int(dec[r])
    return int(p[r] + dec[r])


def key_of(policy, r, a, p, d, kv, dec, k, table, signal=0, t_first=None, h=None,
           t_last=None, promo=None):
    """Iteration-start priority key of request r (lower is served first).
    ``promo``: SJF (LTR+), the promotion iteration of each request or -1."""
    if policy == 0:
        return int(a[r])  # FCFS: arrival
    if policy in (1, 6):
        return int(p[r] + d[r] - 1 - kv[r])  # SRPT / TRAIL: remaining computed tokens
    if policy == 3:
        return int(p[r])  # SPF
    if policy == 4:
        return int(d[r])  # SJF
    if policy == 5:
        return int(p[r] + dec[r])  # LAS: attained service
    if policy == 7:  # DistBoost: the decode queue (by entry time) before the prefill queue
        if dec[r] > 0:
            return (0, int(t_first[r]))
        lvl = min(23, (max(int(p[r]), k) // k).bit_length() - 1)
        return (1, int(a[r]) - int(table[lvl]))
    if policy == 8:  # Sarathi: decodes by their latest token time, then prefills by arrival
        return (0, int(t_last[r])) if dec[r] > 0 else (1, int(a[r]))
    if policy == 9:  # LTR+: promoted requests first, by promotion iteration; then SJF
        return (0, int(promo[r])) if promo[r] >= 0 else (1, int(d[r]))
    lvl = min(23, (max(sig_of(r, p, dec, signal, h), k) // k).bit_length() - 1)
    return int(a[r]) - int(table[lvl])  # boost: a - b(quantized signal)


def replay(a, p, d, e, o, policy, k=1, memguard=0, table=None, signal=0, delta_us=0, h=None,
           ltr=None):
    N = len(a)
    # LTR+ state, rebuilt from the batches: the iteration of the current
    # promotion (-1: none), the iterations not served in a row, the quantum left
    promo = np.full(N, -1, np.int64)
    starve = np.zeros(N, np.int64)
    quantum = np.zeros(N, np.int64)
    bs = e.block_tokens
    kv = np.zeros(N, np.int64)
    dec = np.zeros(N, np.int64)
    guard = np.full(N, -1, np.int64)
    t_first = np.full(N, -1, np.int64)
    t_last = np.full(N, -1, np.int64)
    tbt = np.zeros(N, np.int64)
    done = np.zeros(N, bool)
    first_dispatch = []
    evicted_kv_total = 0
    vol_per_req = np.zeros(N, np.int64)
    ev = o["evict"]
    ev_ptr = 0
    row = 0
    t_expect = 0
    idle = 0
    for i, (t0, dt, nb, U, nw, nr) in enumerate(o["iters"]):
        # I3: the clock only jumps over idle time
        if t0 != t_expect:
            assert t0 > t_expect
            active = [r for r in range(N) if a[r] <= t_expect and not done[r]]
            assert not active, "clock jumped while requests were active"
            assert t0 == min(a[r] for r in range(N) if not done[r] and a[r] > t_expect)
            idle += t0 - t_expect
        resident_before = {r for r in range(N) if kv[r] > 0}
        batch = o["batch"][row:row + nb]
        row += nb
        # iteration-start keys of every active request
        active = [r for r in range(N) if a[r] <= t0 and not done[r]]
        key0 = {r: key_of(policy, r, a, p, d, kv, dec, k, table, signal, t_first, h, t_last, promo)
                for r in active}

        def eligible(x):  # may be a voluntary victim (MemGuard, TRAIL threshold)
            if policy == 8:  # Sarathi: waiting requests never preempt residents
                return False
            if memguard and not oracle.level(sig_of(x, p, dec, signal, h), k) > guard[x]:
                return False
            return not (policy == 6 and 5 * dec[x] >= 3 * d[x])

        def worse(x, r):  # x ranks after r by more than delta
            if isinstance(key0[x], tuple):
                return (key0[x], x) > (key0[r], r)
            return (key0[x] - delta_us, x) > (key0[r], r)

        # evictions of this iteration, each checked against the victim rules:
        # a voluntary victim is the worst eligible resident outside the batch
        # that ranks after the candidate by more than delta; a forced one only
        # happens when there is none, and takes the worst other resident
        # outside the batch, or the candidate itself when none is left
        evicted = set()
        mem_set = [int(x) for x in batch[:, 0]]
        while ev_ptr < len(ev) and ev[ev_ptr][0] == i:
            _, v, forced, cand = (int(x) for x in ev[ev_ptr])
            ev_ptr += 1
            assert kv[v] > 0 and not done[v]
            assert kv[cand] > 0 or not forced  # only a resident candidate forces
            before = {m for m in mem_set if (key0[m], m) < (key0[cand], cand)}
            outside = [x for x in resident_before
                       if x not in evicted and x not in before and x != cand]
            vol = [x for x in outside if eligible(x) and worse(x, cand)]
            if not forced:
                vol_per_req[v] += 1
                assert vol and v == max(vol, key=lambda x: (key0[x], x)), (i, v, cand)
            else:
                assert not vol, (i, v, cand, vol)
                if v != cand:
                    assert v == max(outside, key=lambda x: (key0[x], x)), (i, v, cand)
                else:
                    assert not outside, (i, v, outside)
            evicted_kv_total += kv[v]
            kv[v] = 0
            evicted.add(v)
        # I2 batch limits
        assert 1 <= nb <= e.max_seqs
        ns = batch[:, 1].astype(np.int64)
        assert np.all(ns >= 1) and np.all(ns <= e.chunk) and ns.sum() <= e.max_tokens
        members = batch[:, 0].tolist()
        assert len(set(members)) == nb
        # formation takes candidates in ascending (key, idx) order of the
        # iteration-start keys (batch members were not evicted, so their kv is
        # still the iteration-start value)
        keys = [(key_of(policy, r, a, p, d, kv, dec, k, table, signal, t_first, h, t_last, promo), r)
                for r in members]
        assert keys == sorted(keys)
        assert not (set(members) & evicted)
        for r in members:
            assert a[r] <= t0 and not done[r]
            assert kv[r] < p[r] + dec[r]
            if kv[r] == 0:
                guard[r] = oracle.level(sig_of(r, p, dec, signal, h), k)
                if r not in first_dispatch:
                    first_dispatch.append(r)
        # no request may wait while the batch still has room (stop rule), except
        # evicted ones and waiting ones after a failed admission: residents
        # outside the batch must have been evicted this iteration
        if nb < e.max_seqs and ns.sum() < e.max_tokens:
            for r in resident_before:
                assert r in members or r in evicted
            # eviction completeness: formation saw every candidate, so a waiting
            # request left out was refused for KV after every eligible victim
            # worse than it (by more than delta) had been evicted; none may remain
            # resident outside the batch
            outside = [v for v in range(N) if kv[v] > 0 and v not in members and not done[v]]
            if outside:
                waiting = [w for w in range(N) if a[w] <= t0 and not done[w] and kv[w] == 0
                           and w not in members and w not in evicted]
                def eligible(v):
                    if memguard and not oracle.level(sig_of(v, p, dec, signal, h), k) > guard[v]:
                        return False
                    return not (policy == 6 and 5 * dec[v] >= 3 * d[v])
                for w in waiting:
                    kw = key_of(policy, w, a, p, d, kv, dec, k, table, signal, t_first, h, t_last, promo)
                    for v in outside:
                        kvv = key_of(policy, v, a, p, d, kv, dec, k, table, signal, t_first, h,
                                     t_last, promo)
                        worse = ((kvv, v) > (kw, w)) if isinstance(kvv, tuple) else \
                            ((kvv - delta_us, v) > (kw, w))
                        assert not (worse and eligible(v)), (i, w, v)
        # LTR+: candidates left out starve one more iteration (promoted at the
        # threshold), members reset or spend one iteration of their quantum
        if policy == 9:
            S_, Q_ = ltr
            for r in active:
                if r in members:
                    if promo[r] < 0:
                        starve[r] = 0
                    else:
                        quantum[r] -= 1
                        if quantum[r] == 0:
                            promo[r] = -1
                            starve[r] = 0
                elif promo[r] < 0:
                    starve[r] += 1
                    if starve[r] >= S_:
                        promo[r] = i + 1
                        quantum[r] = Q_
        # cost model and I1
        ctx = sum(int(kv[r] + n) for r, n in zip(members, ns))
        assert dt == e.iter_base_us + e.iter_tok_us * int(ns.sum()) + ctx // e.iter_ctx_div
        for r, n in zip(members, ns):
            kv[r] += n
        u_now = sum(blocks(int(kv[r]), bs) for r in range(N) if kv[r] > 0)
        assert U == u_now and 0 <= U <= e.kv_blocks
        t_end = t0 + dt
        for r, n in zip(members, ns):
            assert kv[r] <= p[r] + dec[r]
            if kv[r] == p[r] + dec[r]:
                dec[r] += 1
                if dec[r] == 1:
                    t_first[r] = t_end
                else:
                    tbt[r] = max(tbt[r], t_end - t_last[r])
                t_last[r] = t_end
                if dec[r] == d[r]:
                    done[r] = True
                    kv[r] = 0
        t_expect = t_end
    assert ev_ptr == len(ev) and row == len(o["batch"])
    # I4 completion exactly once; outputs
    assert np.all(done) and np.array_equal(dec, d.astype(np.int64))
    assert np.array_equal(o["ttft"].astype(np.int64), t_first - a)
    assert np.array_equal(o["ttlt"].astype(np.int64), t_last - a)
    assert np.array_equal(o["tbtmax"].astype(np.int64), tbt)
    c = o["counters"]
    assert c[0] == len(o["iters"])  # iterations
    assert c[1] == int(o["iters"][:, 2].sum())  # I10 request-iterations
    # I6 token conservation
    assert c[2] == int((p.astype(np.int64) + d - 1).sum()) + evicted_kv_total
    assert c[3] + c[4] == len(ev)
    assert c[5] == t_expect and c[5] == int(o["iters"][:, 1].sum()) + idle  # I3
    assert c[6] == int(o["iters"][:, 3].max())
    assert c[7] == idle
    # I5 decode gaps are at least one base step each
    assert np.all(o["ttlt"].astype(np.int64) - o["ttft"] >= (d.astype(np.int64) - 1) * e.iter_base_us)
    if policy == 0:  # I7 FCFS dispatches in arrival order
        assert first_dispatch == sorted(first_dispatch)
    if memguard and signal in (0, 2):  # Phase 3 revision bound per request (monotone signal)
        hh = np.zeros(N, np.int64) if h is None else np.asarray(h, np.int64)
        for r in range(N):
            bound = 1 + math.floor(math.log2(max(int(p[r] + d[r] - hh[r]), k) / k))
            assert vol_per_req[r] <= bound
    return dict(first_dispatch=first_dispatch, vol=vol_per_req)


ENGINES = [
    W.Engine(max_seqs=8, kv_blocks=96, chunk=128, max_tokens=512),
    W.Engine(max_seqs=4, kv_blocks=48, chunk=64, max_tokens=96),
    W.Engine(max_seqs=16, kv_blocks=400, chunk=256, max_tokens=1024),
]
POLICIES = [
    dict(policy=0),
    dict(policy=1),
    dict(policy=3),  # SPF
    dict(policy=4),  # SJF
    dict(policy=5),  # LAS
    dict(policy=6),  # TRAIL
    dict(policy=2, k=16, memguard=1, delta_us=20000, gamma=1e-3),
    dict(policy=2, k=1, memguard=0, delta_us=0, gamma=1e-3),
    dict(policy=2, k=32, memguard=1, delta_us=0, gamma=3e-2),
    dict(policy=7, k=1, gamma=1e-3),  # DistBoost
    dict(policy=7, k=16, gamma=3e-2),
    dict(policy=2, k=16, memguard=1, delta_us=20000, gamma=1e-3, signal=1),  # phase-aware signal
    dict(policy=2, k=1, memguard=0, delta_us=0, gamma=3e-2, signal=1),
    dict(policy=2, k=16, memguard=1, delta_us=20000, gamma=1e-3, signal=2),  # cache-aware signal
    dict(policy=2, k=1, memguard=0, delta_us=0, gamma=3e-2, signal=2),
    dict(policy=8),  # Sarathi
    dict(policy=9, ltr=(4, 3)),  # SJF (LTR+), promotions within a few iterations
    dict(policy=9, ltr=(12, 1)),
]


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("ei", range(len(ENGINES)))
@pytest.mark.parametrize("pi", range(len(POLICIES)))
def test_replay_invariants(seed, ei, pi):
    e = ENGINES[ei]
    pol = POLICIES[pi]
    a, p, d = W.small_random(seed * 10 + ei, 160, rate_per_s=60.0, p_max=400, d_max=200)
    h = W.cached_tokens([seed, ei], p, share=0.6, new_median=8.0) if pol.get("signal") == 2 \
        else None
    o = oracle.log(a, p, d, e, pol["policy"], k=pol.get("k", 1), memguard=pol.get("memguard", 0),
                   delta_us=pol.get("delta_us", 0), gamma=pol.get("gamma"),
                   signal=pol.get("signal", 0), cached=h, ltr=pol.get("ltr"))
    assert o["rc"] == 0
    table = (oracle.boost_table(pol["gamma"], pol.get("k", 1), e.tau_us)
             if pol["policy"] in (2, 7) else None)
    replay(a, p, d, e, o, pol["policy"], k=pol.get("k", 1), memguard=pol.get("memguard", 0),
           table=table, signal=pol.get("signal", 0), delta_us=pol.get("delta_us", 0), h=h,
           ltr=pol.get("ltr"))


def test_replay_sees_evictions():
    """The invariant suite must exercise the eviction paths."""
    e = ENGINES[1]
    a, p, d = W.small_random(3, 160, rate_per_s=60.0, p_max=400, d_max=200)
    o = oracle.log(a, p, d, e, 0)
    assert o["counters"][3] > 0 and o["counters"][4] > 0


def test_alone_is_a_lower_bound():
    """I8: nobody finishes sooner than it would alone."""
    e = ENGINES[0]
    a, p, d = W.small_random(11, 120, rate_per_s=60.0, p_max=400, d_max=200)
    o = oracle.log(a, p, d, e, 2, k=16, memguard=1, delta_us=20000, gamma=1e-3)
    for r in range(len(a)):
        alone = oracle.log([0], [p[r]], [d[r]], e, 0)
        assert o["ttlt"][r] >= alone["ttlt"][0]


def test_run_matches_log_and_percentiles():
    """The multi-instance driver and the single-instance log agree, and the
    reported percentiles are nearest-rank over the latencies."""
    w = W.make(1, n_traces=2, n_settings=6, n_req=400)
    out = oracle.run(w, n_threads=4)
    assert out["rc"] == 0
    for i, s in enumerate(w.settings):
        t = int(s["trace"])
        tb = oracle.tables(w.settings[i:i + 1], w.engine.tau_us)[0]
        o = oracle.log(w.arrival_us[t], w.prompt[t], w.decode[t], w.engine, int(s["policy"]),
                       k=int(s["k"]), memguard=int(s["memguard"]), delta_us=int(s["delta_us"]),
                       table=tb)
        for key in ("ttft", "ttlt", "tbtmax"):
            assert np.array_equal(out[key][i], o[key])
        assert np.array_equal(out["counters"][i], o["counters"])
        for m, key in enumerate(("ttft", "ttlt", "tbtmax")):
            for qi, q in enumerate((50, 90, 99)):
                ref = np.quantile(o[key].astype(np.float64), q / 100, method="inverted_cdf")
                assert out["pct"][i, m, qi] == int(ref)


def test_error_paths():
    e = W.Engine(kv_blocks=4)
    # infeasible: one request needs more KV than exists
    o = oracle.log([0], [100], [1], e, 0)
    assert o["rc"] == oracle.EINFEASIBLE
    # livelock guard
    o = oracle.log([0, 0], [16, 16], [50, 50], W.Engine(), 0, max_iters=10)
    assert o["rc"] == oracle.ELIVELOCK
    # overflow: a latency beyond 2^32-1 us
    o = oracle.log([0], [1], [900_000], W.Engine(kv_blocks=1 << 20), 0)
    assert o["rc"] == oracle.EOVERFLOW
    # unsorted arrivals
    o = oracle.log([10, 5], [16, 16], [2, 2], W.Engine(), 0)
    assert o["rc"] == oracle.EINVAL
