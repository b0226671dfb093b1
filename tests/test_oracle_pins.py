"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names the paper passage (or the mathematical fact) it pins:
hand-worked schedules, closed forms, brute-force optimal orders on tiny
inputs, high-precision evaluation of the boost curve, library order
statistics, identities between policies, and invariants checked on the
oracle's own schedule log by an independent replay.
"""
import itertools
import json
import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "hand_worked.json")))


def engine(**kw):
    return W.Engine(**kw)


def table_of(vals):
    t = np.zeros(24, np.int64)
    t[: len(vals)] = vals
    t[len(vals):] = vals[-1] if vals else 0
    return t


# ------------------------------------------------------------ hand-worked


@pytest.mark.parametrize("case", GOLDEN["cases"], ids=[c["name"] for c in GOLDEN["cases"]])
def test_hand_worked_schedules(case):
    """Schedules derived by hand under the rules (Algorithm 1, Phase 2/3)."""
    e = engine(**case["engine"])
    tb = table_of(case["table"]) if "table" in case else None
    o = oracle.log(case["arrival"], case["prompt"], case["decode"], e, case["policy"],
                   k=case.get("k", 1), memguard=case.get("memguard", 0),
                   delta_us=case.get("delta_us", 0), table=tb, signal=case.get("signal", 0),
                   cached=case.get("cached"), ltr=case.get("ltr"))
    assert o["rc"] == 0
    assert o["ttft"].tolist() == case["ttft"]
    assert o["ttlt"].tolist() == case["ttlt"]
    assert o["tbtmax"].tolist() == case["tbtmax"]
    assert o["counters"].tolist() == case["counters"]


# ------------------------------------------------------------ MemGuard level


@pytest.mark.parametrize("k", [1, 16, 256, 1000])
def test_level_matches_real_log2(k):
    """Eq. memguard_level: w_hat = k 2^floor(log2(max(w,k)/k)), by exact rational
    comparison: level L satisfies k 2^L <= max(w,k) < k 2^(L+1)."""
    for w in list(range(1, 4097)) + [int(x) for x in np.unique(np.geomspace(4097, 1 << 17, 3000).astype(int))]:
        L = oracle.level(w, k)
        m = max(w, k)
        if L < 23:
            assert k * 2 ** L <= m < k * 2 ** (L + 1), (w, k, L)
        else:
            assert k * 2 ** 23 <= m


def test_level_paper_example_revision_points():
    """Phase 3: a 10k-token request with k=256 has at most 6 revision points
    (levels 0..5)."""
    levels = {oracle.level(w, 256) for w in range(1, 10001)}
    assert levels == set(range(6))
    assert 1 + math.floor(math.log2(10000 / 256)) == 6


def test_quantize_forms_agree():
    """The two printed quantizers, k 2^floor(log2(max(w,k)/k)) (Eq.
    memguard_level) and k 2^floor(log2(max(1, s/k))) (Algorithm 2), agree."""
    for k in (1, 3, 16, 256):
        for w in range(1, 5000):
            a = Fraction(max(w, k), k)
            b = max(Fraction(1), Fraction(w, k))
            assert a == b
            assert k * 2 ** oracle.level(w, k) == k * 2 ** (int(math.floor(math.log2(b))) if b < 2 ** 23 else 23)


# ------------------------------------------------------------ boost table

getcontext().prec = 60


def boost_us_decimal(gamma, w, tau):
    """tau * (1/gamma) ln(1/(1 - exp(-gamma w))) in 60-digit decimal arithmetic
    (Eq. boost_function), independent of the C library's log/exp."""
    g = Decimal(repr(gamma))
    x = g * Decimal(w)
    b = (Decimal(1) / (Decimal(1) - (-x).exp())).ln() / g
    return Decimal(repr(tau)) * b


@pytest.mark.parametrize("gamma", [1e-5, 3.1e-5, 1e-4, 3e-4, 1e-3, 3e-3, 1e-2, 3e-2, 1e-1])
@pytest.mark.parametrize("k", [1, 16, 256])
def test_boost_table_high_precision(gamma, k):
    """The fp64 table equals the correctly rounded high-precision value of
    tau * b_gamma(k 2^j), capped at 2^42 (within 1 us where the exact value
    sits within 1e-6 of a rounding tie)."""
    tb = oracle.boost_table(gamma, k, 5000.0)
    for j in range(24):
        ref = boost_us_decimal(gamma, k * 2 ** j, 5000.0)
        cap = Decimal(2) ** 42
        if ref >= cap:
            assert tb[j] == 2 ** 42
            continue
        r = int(ref.to_integral_value(rounding="ROUND_HALF_UP"))
        frac = ref - int(ref)
        if abs(frac - Decimal("0.5")) < Decimal("1e-6") * max(Decimal(1), ref / 10 ** 9):
            assert abs(int(tb[j]) - r) <= 1
        else:
            # fp64 carries ~16 significant digits: allow 1 ulp of the value
            tol = max(0, int(ref * Decimal("4e-16")))
            assert abs(int(tb[j]) - r) <= tol, (gamma, k, j, int(tb[j]), r)


def test_boost_table_monotone_and_limits():
    """b_gamma is decreasing in w (Eq. boost_function); large gamma gives a zero
    table (FCFS limit) and small gamma makes consecutive levels differ by about
    tau ln2 / gamma (least-attained-service limit)."""
    for g in np.geomspace(1e-6, 1.0, 25):
        for k in (1, 16, 256):
            tb = oracle.boost_table(g, k, 5000.0)
            assert np.all(np.diff(tb) <= 0)
            assert np.all(tb >= 0) and tb[0] <= 2 ** 42
    assert np.all(oracle.boost_table(1.0, 256, 5000.0) == 0)
    g = 1e-7
    tb = oracle.boost_table(g, 1, 5000.0)
    gaps = -np.diff(tb[:8]).astype(np.float64)
    assert np.allclose(gaps, 5000.0 * math.log(2) / g, rtol=1e-3)


def test_boost_bound_half_attained():
    """No-starvation section: the boost of a request with attained service w
    is at most b_gamma(w/2) because the quantized signal exceeds w/2."""
    for g in (1e-5, 1e-4, 1e-3, 1e-2):
        for k in (1, 16, 256):
            tb = oracle.boost_table(g, k, 5000.0)
            for w in (k, k + 1, 2 * k - 1, 3 * k, 1000, 4097, 33000):
                if w < k:
                    continue
                L = oracle.level(w, k)
                bound = boost_us_decimal(g, Decimal(w) / 2, 5000.0)
                assert Decimal(int(tb[L])) <= bound + 1


def test_boost_table_rejects_bad_arguments():
    for g, k in [(0.0, 256), (-1e-3, 256), (1e-3, 0)]:
        with pytest.raises(ValueError):
            oracle.boost_table(g, k, 5000.0)


# ------------------------------------------------------------ percentiles


@pytest.mark.parametrize("n", [1, 2, 3, 99, 100, 101, 1000, 4097])
def test_percentile_nearest_rank(n):
    """t_p = inf{t : Fbar(t) <= (100-p)/100} (Phase 4) is the smallest value
    whose empirical CDF reaches p/100: numpy's inverted_cdf quantile."""
    rng = np.random.default_rng(n)
    for dup in (False, True):
        v = rng.integers(0, 50 if dup else 1 << 32, n, dtype=np.uint64).astype(np.uint32)
        for q in (1, 50, 90, 95, 99, 100):
            ref = np.quantile(v.astype(np.float64), q / 100.0, method="inverted_cdf")
            assert oracle.percentile(v, q) == int(ref)
            srt = np.sort(v)
            assert oracle.percentile(v, q) == srt[math.ceil(Fraction(q * n, 100)) - 1]


# ------------------------------------------------------------ closed forms


def alone_schedule(P, D, e):
    """One request alone: prefill chunks of size <= c, then D-1 decode steps;
    step cost base + tok*n + floor(ctx/div) with ctx the KV after the step."""
    t = 0
    kv = 0
    while kv < P:
        n = min(P - kv, e.chunk, e.max_tokens)
        kv += n
        t += e.iter_base_us + e.iter_tok_us * n + kv // e.iter_ctx_div
    ttft = t
    gaps = []
    for j in range(1, D):
        dt = e.iter_base_us + e.iter_tok_us + (P + j) // e.iter_ctx_div
        t += dt
        gaps.append(dt)
    return ttft, t, max(gaps) if gaps else 0


@pytest.mark.parametrize("seed", range(6))
def test_single_request_closed_form(seed):
    rng = np.random.default_rng(seed)
    e = engine(chunk=int(rng.choice([16, 64, 1024])), max_tokens=2048)
    for _ in range(20):
        P, D = int(rng.integers(1, 3000)), int(rng.integers(1, 400))
        a = int(rng.integers(0, 10 ** 6))
        for pol in (0, 1, 2):
            o = oracle.log([a], [P], [D], e, pol, k=16, gamma=1e-3 if pol == 2 else None)
            f, l, g = alone_schedule(P, D, e)
            assert (o["ttft"][0], o["ttlt"][0], o["tbtmax"][0]) == (f, l, g)
            assert o["counters"][7] == a  # idle until the arrival


# ------------------------------------------------------------ brute force


def job_time(P, D, e):
    return alone_schedule(P, D, e)[1]


@pytest.mark.parametrize("seed", range(8))
def test_srpt_minimizes_total_latency_brute_force(seed):
    """M=1, ample KV, one prefill chunk: every request's processing time is
    fixed, so the schedule is a single machine. With common release 0 and equal
    prompts, SRPT's total TTLT equals the minimum over all n! orders (SPT
    optimality), and FCFS gives the identity order."""
    rng = np.random.default_rng([7, seed])
    n = int(rng.integers(3, 7))
    P = int(rng.integers(16, 200))
    D = rng.integers(1, 40, n).astype(np.int32)
    e = engine(max_seqs=1)
    p = [job_time(P, int(d), e) for d in D]
    best = min(sum(itertools.accumulate(p[i] for i in perm)) for perm in itertools.permutations(range(n)))
    o = oracle.log(np.zeros(n), np.full(n, P), D, e, 1)
    assert int(o["ttlt"].astype(np.int64).sum()) == best
    f = oracle.log(np.zeros(n), np.full(n, P), D, e, 0)
    assert f["ttlt"].astype(np.int64).tolist() == list(itertools.accumulate(p))


@pytest.mark.parametrize("seed", range(8))
def test_fcfs_minimizes_max_flow_time_brute_force(seed):
    """Single machine with release dates (M=1, ample KV, one prefill chunk):
    FIFO order minimizes the maximum flow time over all n! orders."""
    rng = np.random.default_rng([8, seed])
    n = int(rng.integers(3, 7))
    P = rng.integers(16, 300, n).astype(np.int32)
    D = rng.integers(1, 30, n).astype(np.int32)
    a = np.sort(rng.integers(0, 200_000, n)).astype(np.int64)
    e = engine(max_seqs=1)
    p = [job_time(int(P[i]), int(D[i]), e) for i in range(n)]

    def max_flow(order):
        t, worst = 0, 0
        for i in order:
            t = max(t, int(a[i])) + p[i]
            worst = max(worst, t - int(a[i]))
        return worst

    best = min(max_flow(perm) for perm in itertools.permutations(range(n)))
    o = oracle.log(a, P, D, e, 0)
    assert int(o["ttlt"].max()) == best


# ------------------------------------------------------------ identities


def rand_trace(seed, n=150, rate=40.0):
    return W.small_random(seed, n, rate_per_s=rate)


@pytest.mark.parametrize("seed", range(5))
def test_zero_boost_equals_fcfs(seed):
    """High gamma mimics FCFS (Formulation; fig. illustration discussion):
    BOOST with a zero table, no hysteresis and no MemGuard is FCFS exactly."""
    a, p, d = rand_trace(seed)
    for e in (engine(max_seqs=8, kv_blocks=64, chunk=128, max_tokens=512), engine(max_seqs=4)):
        f = oracle.log(a, p, d, e, 0)
        b = oracle.log(a, p, d, e, 2, k=1, table=np.zeros(24, np.int64))
        for key in ("ttft", "ttlt", "tbtmax", "counters"):
            assert np.array_equal(f[key], b[key])


@pytest.mark.parametrize("seed", range(4))
def test_huge_gap_table_is_quantized_las(seed):
    """Low gamma mimics least-attained-service: with boost gaps larger than the
    trace span, M=1, ample KV and one-chunk prefills, every iteration serves the
    active request with the smallest (level, arrival, idx)."""
    a, p, d = rand_trace(seed, n=60, rate=30.0)
    e = engine(max_seqs=1, chunk=1024)
    k = 16
    tb = np.array([(23 - j) * 10 ** 11 for j in range(24)], np.int64)
    o = oracle.log(a, p, d, e, 2, k=k, table=tb)
    assert o["rc"] == 0
    dec = np.zeros(len(a), np.int64)
    done = np.zeros(len(a), bool)
    row = 0
    for it in o["iters"]:
        t0 = it[0]
        assert it[2] == 1
        r, n = o["batch"][row]
        row += 1
        active = [i for i in range(len(a)) if a[i] <= t0 and not done[i]]
        best = min(active, key=lambda i: (oracle.level(int(p[i]) + int(dec[i]), k), a[i], i))
        assert r == best
        dec[r] += 1
        if dec[r] == d[r]:
            done[r] = True


@pytest.mark.parametrize("seed", range(4))
def test_boost_is_blind_to_decode_length(seed):
    """Prediction-free (Abstract; Formulation, blind policies): lengthening one
    request's decode changes nothing before that request's original
    completion. SRPT, which reads the length, is not blind."""
    a, p, d = rand_trace(seed, n=120, rate=60.0)
    e = engine(max_seqs=6, kv_blocks=80, chunk=128, max_tokens=384)
    j = 17
    d2 = d.copy()
    d2[j] += 500
    for pol, blind in ((2, True), (1, False)):
        kw = dict(k=16, memguard=1, delta_us=20000, gamma=3e-3) if pol == 2 else {}
        o1 = oracle.log(a, p, d, e, pol, **kw)
        o2 = oracle.log(a, p, d2, e, pol, **kw)
        # the iteration in which j finished originally
        ends = np.cumsum(o1["iters"][:, 2])
        last = max(i for i in range(len(ends)) if j in o1["batch"][(ends[i] - o1["iters"][i, 2]):ends[i], 0])
        same = (np.array_equal(o1["iters"][: last + 1], o2["iters"][: last + 1])
                and np.array_equal(o1["batch"][: ends[last]], o2["batch"][: ends[last]]))
        if blind:
            assert same
    # SRPT is expected to differ on at least one of these seeds; checked in aggregate below


def test_srpt_reads_decode_length():
    diffs = 0
    e = engine(max_seqs=2, chunk=128, max_tokens=384)
    for seed in range(6):
        a, p, d = rand_trace(seed, n=60, rate=80.0)
        d2 = d.copy()
        d2[5] += 2000
        o1 = oracle.log(a, p, d, e, 1)
        o2 = oracle.log(a, p, d2, e, 1)
        m = min(len(o1["batch"]), len(o2["batch"]))
        diffs += not np.array_equal(o1["batch"][:m], o2["batch"][:m])
    assert diffs > 0
