"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Every comparison is element by element and exact: the whole path is integer
arithmetic (the only floating-point step, the boost table, is checked equal
on the host). Inputs are the seeded workloads; sizes span many 64-wide chunks
and ragged tails, plus the degenerate cases.
"""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def gpu_run(w, **kw):
    from paper_2606_18431_amd import tas

    print(f"[gpu] {w.name} traces={w.n_traces} inst={w.n_inst} n_req={w.n_req} {kw}", flush=True)
    sim = tas.Simulation(w, **kw)
    sim.step()
    out = sim.results()
    out["tables"] = np.stack([sim.table(i) for i in range(w.n_inst)]) if w.n_inst else None
    sim.close()
    return out


def assert_parity(w, g, o, inst=None):
    inst = range(w.n_inst) if inst is None else inst
    for i in inst:
        assert g["status"][i] == o["status"][i] == 0, (i, g["status"][i], o["status"][i])
        for key in ("ttft", "ttlt", "tbtmax"):
            if not np.array_equal(g[key][i], o[key][i]):
                bad = np.nonzero(g[key][i] != o[key][i])[0]
                raise AssertionError(f"inst {i} {key}: {len(bad)} differ, first idx {bad[0]}: "
                                     f"gpu {g[key][i][bad[0]]} oracle {o[key][i][bad[0]]}")
        assert np.array_equal(g["counters"][i], o["counters"][i]), (i, g["counters"][i],
                                                                    o["counters"][i])
        assert np.array_equal(g["pct"][i], o["pct"][i]), (i, g["pct"][i], o["pct"][i])


def test_boost_tables_equal(torch):
    w = W.make(1, n_traces=1, n_settings=64, n_req=64)
    g = gpu_run(w)
    assert np.array_equal(g["tables"], oracle.tables(w.settings, w.engine.tau_us))


GOLD = json.load(open(os.path.join(HERE, "golden", "hand_worked.json")))["cases"]


@pytest.mark.parametrize("case", GOLD, ids=[c["name"] for c in GOLD])
def test_hand_worked_on_gpu(torch, case):
    e = W.Engine(**case["engine"])
    tb = case.get("table")
    s = W.setting(0, case["policy"], k=case.get("k", 1), memguard=case.get("memguard", 0),
                  delta_us=case.get("delta_us", 0), table=tb if tb is not None else None,
                  signal=case.get("signal", 0), ltr=case.get("ltr"))
    w = W.Workload(case["name"], np.array([case["arrival"]], np.int64),
                   np.array([case["prompt"]], np.int32), np.array([case["decode"]], np.int32),
                   e, np.stack([s]),
                   cached=np.array([case["cached"]], np.int32) if "cached" in case else None)
    g = gpu_run(w)
    assert g["rc"] == 0
    assert g["ttft"][0].tolist() == case["ttft"]
    assert g["ttlt"][0].tolist() == case["ttlt"]
    assert g["tbtmax"][0].tolist() == case["tbtmax"]
    assert g["counters"][0].tolist() == case["counters"]


@pytest.mark.parametrize("cfg,n_traces,n_settings,n_req", [
    (0, 1, 8, 1000),      # the tiny workload, full size
    (1, 2, 8, 3000),
    (2, 2, 8, 3000),      # KV pressure: many evictions
    (3, 2, 8, 5000),      # bursts and a length shift
    (4, 1, 8, 6000),      # max_seqs 256, 16384-token budget
    (5, 2, 8, 4000),      # the starvation mix under its policies (Sarathi: extended build)
])
def test_parity_reduced_configs(torch, cfg, n_traces, n_settings, n_req):
    w = W.make(cfg, n_traces=n_traces, n_settings=n_settings, n_req=n_req)
    o = oracle.run(w)
    assert o["rc"] == 0
    g = gpu_run(w)
    assert_parity(w, g, o)


@pytest.mark.parametrize("cfg,n_traces,n_req", [
    (1, 2, 3000),
    (2, 2, 3000),         # KV pressure: TRAIL's threshold and the victims matter
    (3, 1, 5000),
    (4, 1, 6000),
])
def test_parity_comparators(torch, cfg, n_traces, n_req):
    """FCFS, SRPT, SPF, SJF, LAS, TRAIL, UniBoost and vanilla boost on every trace.
    LAS starves long requests under load: where a latency exceeds 2^32-1 us both
    sides must report TAS_EOVERFLOW for that instance; every other instance is
    compared element by element."""
    w = W.make(cfg, n_traces=n_traces, n_req=n_req, grid="comparators")
    o = oracle.run(w)
    g = gpu_run(w)
    assert np.array_equal(g["status"], o["status"]), (g["status"], o["status"])
    assert set(np.unique(o["status"]).tolist()) <= {0, -5}
    assert_parity(w, g, o, inst=np.nonzero(o["status"] == 0)[0])


@pytest.mark.parametrize("cfg,list_cap", [(2, 192), (3, 128)])
def test_parity_comparators_with_spill(torch, cfg, list_cap):
    w = W.make(cfg, n_traces=1, n_req=4000, grid="comparators")
    o = oracle.run(w)
    g = gpu_run(w, list_cap=list_cap)
    assert np.array_equal(g["status"], o["status"]), (g["status"], o["status"])
    assert_parity(w, g, o, inst=np.nonzero(o["status"] == 0)[0])


@pytest.mark.parametrize("cfg,list_cap", [(2, 192), (4, 320), (3, 128)])
def test_parity_with_spill(torch, cfg, list_cap):
    """A small on-chip list forces the HBM spill, refill and radix-select paths."""
    w = W.make(cfg, n_traces=1, n_settings=8, n_req=4000)
    o = oracle.run(w)
    g = gpu_run(w, list_cap=list_cap)
    assert_parity(w, g, o)


def test_parity_with_minimum_list(torch):
    """The smallest allowed list (max_seqs + 64) still gives exact results:
    spilled waiting entries are brought back exactly when formation reaches
    them."""
    w = W.make(2, n_traces=1, n_settings=8, n_req=4000)
    o = oracle.run(w)
    g = gpu_run(w, list_cap=128)
    assert_parity(w, g, o)


def las_burst_workload(n=200):
    """Least-attained-service order with everyone arriving at once pauses old
    residents behind fresh arrivals, so more requests hold KV than max_seqs."""
    tb = [(23 - j) * 10 ** 11 for j in range(24)]
    return edge_workload(np.zeros(n), np.ones(n), np.full(n, 50),
                         W.Engine(max_seqs=8, kv_blocks=4096, chunk=64, max_tokens=512),
                         policies=[W.setting(0, W.BOOST, k=1, table=tb),
                                   W.setting(0, W.FCFS)])


def test_residents_beyond_list_are_retried_exactly(torch):
    """An instance whose residents outgrow the first-pass list reruns from
    scratch in the second pass with the large list: exact results."""
    w = las_burst_workload()
    o = oracle.run(w)
    assert o["rc"] == 0
    g = gpu_run(w, list_cap=72)
    assert_parity(w, g, o)


def test_residents_beyond_both_lists_fail_loudly(torch):
    """Without room in the retry list either, the instance reports
    TAS_ECAPACITY instead of a wrong schedule; the others are exact."""
    w = las_burst_workload()
    o = oracle.run(w)
    g = gpu_run(w, list_cap=72, retry_cap=72)
    assert g["rc"] == -8 and g["status"][0] == -8
    assert_parity(w, g, o, inst=[1])


def edge_workload(arrival, prompt, decode, engine, policies=None):
    a = np.asarray(arrival, np.int64)[None]
    p = np.asarray(prompt, np.int32)[None]
    d = np.asarray(decode, np.int32)[None]
    sets = policies or [W.setting(0, W.FCFS), W.setting(0, W.SRPT),
                        W.setting(0, W.BOOST, gamma=1e-3, **W.UNIBOOST),
                        W.setting(0, W.BOOST, gamma=1e-3, **W.VANILLA)]
    # expected prefix-cache hits for the cache-aware signal: a seeded draw
    # that keeps at least one prompt token of work
    h = W.cached_tokens(len(a[0]), p[0], share=0.7, new_median=4.0)[None] \
        if any(s["signal"] == 2 for s in sets) else None
    return W.Workload("edge", a, p, d, engine, np.stack(sets), cached=h)


EDGES = {
    "one_request": ([0], [5], [1], W.Engine()),
    "two_requests_same_time": ([7, 7], [100, 3], [4, 9], W.Engine(max_seqs=1)),
    "all_at_zero": (np.zeros(300), np.full(300, 40), np.arange(1, 301) % 17 + 1,
                    W.Engine(max_seqs=16, kv_blocks=64, chunk=32, max_tokens=256)),
    "all_decode_one": (np.arange(200) * 100, np.full(200, 33), np.ones(200),
                       W.Engine(max_seqs=8, kv_blocks=40)),
    "prompt_one": (np.arange(150) * 3000, np.ones(150), np.full(150, 20), W.Engine(max_seqs=4)),
    "long_prompts_many_chunks": (np.arange(80) * 20000, np.full(80, 4000), np.full(80, 3),
                                 W.Engine(max_seqs=4, chunk=512, max_tokens=1024, kv_blocks=600)),
    "kv_exactly_one_request": (np.zeros(40), np.full(40, 16), np.full(40, 17),
                               W.Engine(max_seqs=64, kv_blocks=2, block_tokens=16)),
    "block_size_one": (np.arange(120) * 500, np.full(120, 7), np.full(120, 9),
                       W.Engine(max_seqs=8, kv_blocks=60, block_tokens=1, chunk=5,
                                max_tokens=12)),
    "non_power_of_two_block": (np.arange(120) * 900, np.full(120, 50), np.full(120, 30),
                               W.Engine(max_seqs=8, kv_blocks=40, block_tokens=12, chunk=40,
                                        max_tokens=100)),
    "idle_gaps": (np.array([0, 10 ** 9, 2 * 10 ** 9, 2 * 10 ** 9 + 1]), [10, 20, 30, 40],
                  [3, 3, 3, 3], W.Engine()),
}


EXTENDED = [W.setting(0, W.SPF), W.setting(0, W.SJF), W.setting(0, W.LAS), W.setting(0, W.TRAIL),
            W.setting(0, W.DIST, gamma=1e-3),
            W.setting(0, W.BOOST, gamma=1e-3, signal=1, **W.UNIBOOST),
            W.setting(0, W.BOOST, gamma=1e-3, ada=dict(W.ADA, window=8, min_samples=4),
                      **W.UNIBOOST),
            W.setting(0, W.SARATHI), W.setting(0, W.BOOST, gamma=1e-3, signal=2, **W.UNIBOOST),
            W.setting(0, W.LTR, ltr=(3, 2))]


@pytest.mark.parametrize("extended", [False, True], ids=["base", "extended"])
@pytest.mark.parametrize("name", sorted(EDGES))
def test_edge_cases(torch, name, extended):
    """Each case under the base policies (fixed kernel build) and under the
    comparators, DistBoost, Sarathi, the phase-aware and cache-aware signals
    and adaptive gamma (the extended build)."""
    a, p, d, e = EDGES[name]
    w = edge_workload(a, p, d, e, EXTENDED if extended else None)
    o = oracle.run(w)
    ok = o["status"] == 0
    assert ok.all() or extended  # LAS may overflow on long idle gaps (status compared)
    g = gpu_run(w)
    assert np.array_equal(g["status"], o["status"])
    assert_parity(w, g, o, inst=np.nonzero(ok)[0])
    if extended:
        assert np.array_equal(g["gamma"].view(np.int64), o["gamma"].view(np.int64))
        assert np.array_equal(g["switches"], o["switches"])


def test_largest_request_count(torch):
    """2^20 - 1 requests per trace, the most the boundary accepts (request
    indices fill the packed key's 21-bit field with room to spare): groups
    of eight short requests every 70 ms into a server of four sequences
    (about 0.8 utilisation, 1.5 M iterations) under FCFS, UniBoost and SJF
    (LTR+), every latency and percentile equal to the oracle."""
    n = (1 << 20) - 1
    rng = np.random.default_rng(20)
    a = (np.arange(n) // 8).astype(np.int64) * 70_000
    p = rng.integers(16, 257, n).astype(np.int32)
    d = rng.integers(1, 9, n).astype(np.int32)
    sets = [W.setting(0, W.FCFS), W.setting(0, W.BOOST, gamma=1e-3, **W.UNIBOOST),
            W.setting(0, W.LTR, ltr=(8, 4))]
    w = W.Workload("largest-n", a[None], p[None], d[None], W.Engine(max_seqs=4),
                   np.stack(sets))
    o = oracle.run(w)
    assert o["rc"] == 0
    assert_parity(w, gpu_run(w), o)


@pytest.mark.parametrize("div", [1, 2, 3, 7, 64, 100, 997, (1 << 20) + 7, (1 << 31) - 1])
def test_cost_model_divisors(torch, div):
    """floor(sum(kv + n) / div) for divisors from 1 to 2^31 - 1."""
    a, p, d = W.small_random(7, 400, rate_per_s=60.0)
    e = W.Engine(max_seqs=16, kv_blocks=300, chunk=64, max_tokens=256, iter_ctx_div=div)
    w = edge_workload(a, p, d, e)
    o = oracle.run(w)
    assert o["rc"] == 0
    assert_parity(w, gpu_run(w), o)


def test_context_sum_beyond_32_bits(torch):
    """300 resident prompts of 2^24 - 3 tokens: the batch's summed context
    passes 2^32 during prefill."""
    n, P = 300, (1 << 24) - 3
    e = W.Engine(max_seqs=n, max_tokens=n * 32767, chunk=32767,
                 kv_blocks=n * ((P + 1 + 15) // 16), iter_tok_us=0, iter_ctx_div=(1 << 31) - 1)
    w = edge_workload(np.zeros(n), np.full(n, P), np.full(n, 2), e)
    o = oracle.run(w)
    assert o["rc"] == 0
    assert o["counters"][:, 0].max() > 500
    assert_parity(w, gpu_run(w), o)


def test_more_than_64_arrivals_at_once(torch):
    a = np.concatenate([np.zeros(150), np.full(200, 50_000)])
    w = edge_workload(a, np.full(350, 20), np.full(350, 5),
                      W.Engine(max_seqs=32, kv_blocks=200, chunk=64, max_tokens=512))
    o = oracle.run(w)
    assert_parity(w, gpu_run(w), o)


def test_error_livelock(torch):
    w = edge_workload([0, 0], [16, 16], [50, 50], W.Engine(max_iters=10))
    g = gpu_run(w)
    assert g["rc"] == -6 and np.all(g["status"] == -6)


def test_error_overflow(torch):
    w = edge_workload([0], [1], [900_000], W.Engine(kv_blocks=1 << 20),
                      policies=[W.setting(0, W.FCFS)])
    g = gpu_run(w)
    assert g["rc"] == -5


def test_error_spill_capacity(torch):
    """A spill too small to hold the waiting queue is reported, not hidden."""
    w = W.make(2, n_traces=1, n_settings=4, n_req=3000)
    g = gpu_run(w, list_cap=128, spill_cap=16, retry_cap=128)
    assert g["rc"] == -8 and np.any(g["status"] == -8)


@pytest.mark.parametrize("n_req", [1, 2, 3, 5, 1001, 1003])
def test_percentiles_at_unaligned_row_sizes(torch, n_req):
    """Request counts that are not multiples of 4 put the latency rows of
    most instances off a 16-byte boundary: the percentile kernel reads a
    head, an aligned body and a tail of every row; all nine percentiles and
    every latency equal the oracle's."""
    w = W.make(1, n_traces=2, n_settings=6, n_req=n_req)
    o = oracle.run(w)
    assert o["rc"] == 0
    assert_parity(w, gpu_run(w), o)


def test_deterministic_and_order_independent(torch):
    w = W.make(2, n_traces=2, n_settings=6, n_req=2500)
    g1 = gpu_run(w)
    g2 = gpu_run(w)
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct"):
        assert np.array_equal(g1[key], g2[key])
    perm = np.random.default_rng(1).permutation(w.n_inst)
    g3 = gpu_run(w.subset(perm))
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct"):
        assert np.array_equal(g3[key], g1[key][perm])


@pytest.mark.parametrize("cfg", [1, 2])
def test_parity_sensitivity_grid(torch, cfg):
    """The paper's sensitivity study: UniBoost over k and delta beside FCFS."""
    w = W.make(cfg, n_traces=2, n_req=3000, grid="sensitivity")
    o = oracle.run(w)
    assert o["rc"] == 0
    assert_parity(w, gpu_run(w), o)


@pytest.mark.parametrize("chunk", [128, 512, 2048])
def test_parity_chunk_sizes(torch, chunk):
    """The prefill chunk of the paper's chunk-size study."""
    import dataclasses

    w = W.make(2, n_traces=1, n_settings=8, n_req=3000)
    w = dataclasses.replace(w, engine=dataclasses.replace(w.engine, chunk=chunk))
    o = oracle.run(w)
    assert o["rc"] == 0
    assert_parity(w, gpu_run(w), o)


def work_estimate(w):
    """The first launch's ranking: per trace, the sum of D + ceil(P / chunk);
    times 5 for policies that re-key every batch member at every token, else 4."""
    c = w.engine.chunk
    work = [int(sum(int(d) + -(-int(p) // c) for p, d in zip(w.prompt[t], w.decode[t])))
            for t in range(w.n_traces)]
    return [work[int(s["trace"])] * (5 if int(s["policy"]) in (W.SRPT, W.TRAIL, W.LAS,
                                                                  W.SARATHI) else 4)
            for s in w.settings]


def test_launch_order_follows_previous_work(torch):
    """The first run takes the instances longest first by the work estimate,
    later runs by the loop steps each instance ran in the previous run (each
    order a permutation; the steps are the same in every run), and every run
    gives the same results, equal to the oracle."""
    from paper_2606_18431_amd import tas

    w = W.make(2, n_traces=3, n_settings=8, n_req=2000)
    o = oracle.run(w)
    sim = tas.Simulation(w)
    n = w.n_inst
    work = torch.zeros(n, dtype=torch.int64, device="cuda")
    order = torch.zeros(n, dtype=torch.int32, device="cuda")
    tas.tas_schedule(sim.ctx, work, order)
    prev = work.cpu().numpy()
    assert prev.tolist() == work_estimate(w)
    for k in range(3):
        print(f"[gpu] launch order, run {k}", flush=True)
        sim.step()
        g = sim.results()
        assert_parity(w, g, o)
        tas.tas_schedule(sim.ctx, work, order)
        d, od = work.cpu().numpy(), order.cpu().numpy()
        # 4 steps per iteration at least
        assert np.all(d >= 4 * g["counters"][:, 0]) and sorted(od.tolist()) == list(range(n))
        if k > 0:
            assert np.array_equal(d, prev)  # deterministic
        # most work first, ties by index
        assert od.tolist() == sorted(range(n), key=lambda i: (-int(prev[i]), i))
        prev = d.copy()
    sim.close()


@pytest.mark.parametrize("n", [1000, 16383, 16384])
def test_launch_order_permutation_at_size(torch, n):
    """The order kernel at up to its largest size (one LDS sort of 16384):
    every run's order is a permutation of the instances, most work (loop
    steps) in the previous run first; results of the ordered run equal the
    oracle on a sample."""
    from paper_2606_18431_amd import tas

    w = W.make(1, n_traces=256, n_settings=64, n_req=100).subset(np.arange(n))
    sim = tas.Simulation(w)
    work = torch.zeros(n, dtype=torch.int64, device="cuda")
    order = torch.zeros(n, dtype=torch.int32, device="cuda")
    prev = np.asarray(work_estimate(w), np.int64)
    for k in range(2):
        print(f"[gpu] launch order at {n} instances, run {k}", flush=True)
        sim.step()
        tas.tas_schedule(sim.ctx, work, order)
        d, od = work.cpu().numpy(), order.cpu().numpy()
        assert np.array_equal(np.sort(od), np.arange(n)) and np.all(d > 0)
        assert np.array_equal(od, np.lexsort((np.arange(n), -prev)))
        prev = d.copy()
    g = sim.results()
    sim.close()
    assert g["rc"] == 0 and np.all(prev >= 4 * g["counters"][:, 0])
    sel = np.unique(np.concatenate([np.arange(8), np.arange(n - 8, n),
                                    np.random.default_rng(n).choice(n, 16, replace=False)]))
    o = oracle.run(w.subset(sel))
    for j, i in enumerate(sel):
        for key in ("ttft", "ttlt", "tbtmax"):
            assert np.array_equal(g[key][i], o[key][j]), (i, key)
        assert np.array_equal(g["counters"][i], o["counters"][j]), i


@pytest.mark.parametrize("cfg,n_traces,n_req,ltr", [
    (1, 2, 3000, (8, 4)),
    (2, 2, 3000, (8, 4)),      # KV pressure: promoted requests evict residents
    (2, 1, 3000, (40, 16)),
    (3, 1, 5000, (24, 2)),
    (4, 1, 12000, (64, 32)),   # 256 sequences: queues form after the first 6000 requests
])
def test_parity_ltr(torch, cfg, n_traces, n_req, ltr):
    """SJF (LTR+) with thresholds low enough that promotions, quantum expiries
    and demotions happen all along; with max_seqs 64 the first-pass list holds
    192 entries, so instances whose queue outgrows it rerun with the large
    list (LTR+ keeps every request on chip)."""
    import dataclasses

    w = W.make(cfg, n_traces=n_traces, n_settings=4, n_req=n_req)
    s = np.stack([W.setting(t, W.LTR, ltr=ltr) for t in range(n_traces)] +
                 [W.setting(t, W.SJF) for t in range(n_traces)])
    w = dataclasses.replace(w, settings=s)
    o = oracle.run(w)
    g = gpu_run(w)
    assert (o["status"] == g["status"]).all(), (o["status"], g["status"])
    ok = o["status"] == 0
    assert ok.any()
    for key in ("ttft", "ttlt", "tbtmax", "counters", "pct"):
        assert np.array_equal(g[key][ok], o[key][ok]), key
    # the control changed the schedule somewhere
    n = n_traces
    assert any(not np.array_equal(o["ttlt"][i], o["ttlt"][n + i]) for i in range(n) if ok[i])
