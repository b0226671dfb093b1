"""Pins of the adaptive gamma (paper: Phase 4, gamma-Ada: Eq. gamma_estimator
and Algorithm 2 UpdateGamma, called once per iteration of Algorithm 1) in the
CPU oracle.

- hand-worked schedules (golden/ada_hand.json): the estimator over the tail
  band, the EMA, the eps floor, both clips, the min-samples rule and the order
  in which requests finishing in one iteration enter the window;
- beta = 0 freezes gamma: the run equals the fixed-gamma run on the table of
  gamma0's grid point;
- the grid is log-spaced with geometric midpoints, and its tables are the
  boost tables of its points;
- a replay of the oracle's schedule log with code of its own: the window of
  the last W completions, nearest-rank t95/t99 (numpy's inverted-CDF
  quantile), the estimator written from the tail-band definition
  -(ln Fbar(t99) - ln Fbar(t95)) / (t99 - t95), the EMA, the clip and the
  log-nearest grid cell, and every batch in ascending (key, idx) order for the
  keys of the logged cell's table.
"""
import collections
import json
import math
import os

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = json.load(open(os.path.join(HERE, "golden", "ada_hand.json")))
TAU = 5000.0


def one_instance(arrival, prompt, decode, engine, **setting):
    s = np.stack([W.setting(0, **setting)])
    return W.Workload("t", np.asarray([arrival], np.int64), np.asarray([prompt], np.int32),
                      np.asarray([decode], np.int32), engine, s)


def case_run(c):
    w = one_instance(c["arrival"], c["prompt"], c["decode"], W.Engine(), policy=c["policy"],
                     k=c["k"], memguard=c["memguard"], delta_us=c["delta_us"],
                     gamma=c["gamma0"], ada=c["ada"])
    return oracle.run(w, n_threads=1)


@pytest.mark.parametrize("c", GOLDEN["cases"], ids=lambda c: c["name"])
def test_ada_hand_worked(c):
    o = case_run(c)
    assert o["rc"] == 0
    assert o["ttlt"][0].tolist() == c["ttlt"]
    assert math.isclose(o["gamma"][0], c["gamma_final"], rel_tol=1e-12, abs_tol=0.0)
    assert o["switches"][0] == c["switches"]
    lg = oracle.log(c["arrival"], c["prompt"], c["decode"], W.Engine(), c["policy"], k=c["k"],
                    memguard=c["memguard"], delta_us=c["delta_us"], gamma=c["gamma0"],
                    ada=c["ada"])
    assert lg["rc"] == 0 and lg["cell"][-1] == c["cell_final"]
    assert lg["gamma"][-1] == o["gamma"][0]


def test_ada_window_order_matters():
    """The window-order case is sensitive to the order: index order would give
    another gamma (so the pin above really checks the batch order)."""
    c = next(c for c in GOLDEN["cases"] if c["name"] == "ada_window_batch_order")
    alt = 5000.0 * math.log(5.0) / 2000.0
    assert not math.isclose(c["gamma_final"], alt, rel_tol=1e-3)


def ada_setting(gamma0, ada, k=1):
    return W.setting(0, W.BOOST, k=k, gamma=gamma0, ada=ada)


def test_ada_grid_is_log_spaced():
    ada = dict(W.ADA)
    grid, bound, tabs = oracle.ada_grid(ada_setting(1e-3, ada), TAU)
    G = ada["grid"]
    assert len(grid) == G and grid[0] == ada["gamma_min"]
    assert math.isclose(grid[-1], ada["gamma_max"], rel_tol=1e-14)
    step = math.log(ada["gamma_max"] / ada["gamma_min"]) / (G - 1)
    assert np.allclose(np.diff(np.log(grid)), step, rtol=1e-10, atol=0)
    assert np.allclose(bound, np.sqrt(grid[:-1] * grid[1:]), rtol=1e-15, atol=0)
    for j in (0, 7, G - 1):
        assert np.array_equal(tabs[j], oracle.boost_table(grid[j], 1, TAU))


@pytest.mark.parametrize("seed", range(3))
def test_ada_beta_zero_is_the_fixed_table(seed):
    """beta = 0: gamma never moves, so the run is the fixed-gamma run with the
    table of the grid point nearest gamma0 (2.5e-3 -> 10^-2.6)."""
    ada = dict(W.ADA, beta=0.0, window=20, min_samples=20)
    e = W.Engine(max_seqs=8, kv_blocks=96, chunk=128, max_tokens=512)
    a, p, d = W.small_random(seed, 300, rate_per_s=60.0, p_max=400, d_max=200)
    g0 = 2.5e-3
    grid, _, tabs = oracle.ada_grid(ada_setting(g0, ada, k=16), TAU)
    j = int(np.argmin(np.abs(np.log(grid) - math.log(g0))))
    assert math.isclose(grid[j], 10 ** -2.6, rel_tol=1e-12)
    wa = one_instance(a, p, d, e, policy=W.BOOST, k=16, memguard=1, delta_us=20000, gamma=g0,
                      ada=ada)
    wf = one_instance(a, p, d, e, policy=W.BOOST, k=16, memguard=1, delta_us=20000,
                      table=tabs[j])
    oa, of = oracle.run(wa, n_threads=1), oracle.run(wf, n_threads=1)
    assert oa["rc"] == 0 and of["rc"] == 0
    for key in ("ttft", "ttlt", "tbtmax", "counters"):
        assert np.array_equal(oa[key], of[key])
    assert oa["gamma"][0] == g0 and oa["switches"][0] == 0
    assert oa["counters"][0, 3] > 0  # the trace exercises voluntary evictions


def level(w, k):
    return min(23, (max(w, k) // k).bit_length() - 1)


def ada_replay(a, p, d, e, lg, gamma0, ada, k):
    """Replay one adaptive instance's log (see the module docstring)."""
    grid, _, tabs = oracle.ada_grid(ada_setting(gamma0, ada, k=k), TAU)
    ln_tail = -(math.log(0.01) - math.log(0.05))  # -(ln Fbar(t99) - ln Fbar(t95))
    window = collections.deque(maxlen=int(ada["window"]))
    N = len(a)
    kv = np.zeros(N, np.int64)
    dec = np.zeros(N, np.int64)
    gamma = gamma0
    ev = lg["evict"]
    ep = row = 0
    checked = 0
    for i, (t0, dt, nb, U, nw, nr) in enumerate(lg["iters"]):
        # UpdateGamma at the start of the iteration
        if len(window) >= ada["min_samples"]:
            x = np.asarray(window, np.float64)
            t95 = np.quantile(x, 0.95, method="inverted_cdf")
            t99 = np.quantile(x, 0.99, method="inverted_cdf")
            per_us = ln_tail / max(t99 - t95, ada["eps_us"])
            g = (1 - ada["beta"]) * gamma + ada["beta"] * (per_us * TAU)
            gamma = min(max(g, ada["gamma_min"]), ada["gamma_max"])
        assert math.isclose(lg["gamma"][i], gamma, rel_tol=1e-12, abs_tol=0.0), i
        dist = np.abs(np.log(grid) - math.log(lg["gamma"][i]))
        order = np.argsort(dist)
        if dist[order[1]] - dist[order[0]] > 1e-9:
            assert lg["cell"][i] == order[0], i
            checked += 1
        tab = tabs[lg["cell"][i]]
        while ep < len(ev) and ev[ep][0] == i:
            kv[ev[ep][1]] = 0
            ep += 1
        batch = lg["batch"][row:row + nb]
        row += nb
        keys = [(int(a[r]) - int(tab[level(int(p[r] + dec[r]), k)]), int(r)) for r, _ in batch]
        assert keys == sorted(keys), i  # formation takes candidates in key order
        t_end = t0 + dt
        for r, n in batch:
            kv[r] += n
            if kv[r] == p[r] + dec[r]:
                dec[r] += 1
                if dec[r] == d[r]:
                    kv[r] = 0
                    window.append(min(int(t_end - a[r]), 2**32 - 1))
    assert row == len(lg["batch"])
    return checked


ADA_CASES = [
    (dict(W.ADA, window=24, min_samples=20, beta=0.05, grid=41), 16, 1, 20000),
    (dict(W.ADA, window=40, min_samples=30, beta=0.2, grid=21, eps_us=200.0), 1, 0, 0),
    (dict(W.ADA, window=64, min_samples=64, beta=1.0, grid=64, gamma_min=1e-4,
          gamma_max=3e-1), 32, 1, 0),
]


@pytest.mark.parametrize("seed", range(3))
@pytest.mark.parametrize("ci", range(len(ADA_CASES)))
def test_ada_replay(seed, ci):
    ada, k, mg, dl = ADA_CASES[ci]
    e = [W.Engine(max_seqs=8, kv_blocks=96, chunk=128, max_tokens=512),
         W.Engine(max_seqs=16, kv_blocks=400, chunk=256, max_tokens=1024)][seed % 2]
    a, p, d = W.small_random(seed * 7 + ci, 400, rate_per_s=60.0, p_max=400, d_max=200)
    lg = oracle.log(a, p, d, e, W.BOOST, k=k, memguard=mg, delta_us=dl, gamma=1e-3, ada=ada)
    assert lg["rc"] == 0
    checked = ada_replay(a, p, d, e, lg, 1e-3, ada, k)
    assert checked > 0.9 * len(lg["iters"])
    cells = lg["cell"]
    assert np.count_nonzero(np.diff(cells)) > 0  # gamma left its first grid cell
    # the run() outputs agree with the log
    w = one_instance(a, p, d, e, policy=W.BOOST, k=k, memguard=mg, delta_us=dl, gamma=1e-3,
                     ada=ada)
    o = oracle.run(w, n_threads=1)
    assert np.array_equal(o["ttlt"][0], lg["ttlt"])
    assert o["gamma"][0] == lg["gamma"][-1]
    grid = oracle.ada_grid(ada_setting(1e-3, ada, k=k), TAU)[0]
    c0 = int(np.argmin(np.abs(np.log(grid) - math.log(1e-3))))  # the cell of gamma0
    assert o["switches"][0] == np.count_nonzero(np.diff(np.concatenate([[c0], cells])))


def test_ada_rejects_bad_parameters():
    a, p, d = W.small_random(0, 20)
    e = W.Engine()
    good = dict(W.ADA)
    bad = [dict(good, beta=1.5), dict(good, beta=-0.1), dict(good, window=0),
           dict(good, window=4096), dict(good, min_samples=300), dict(good, grid=1),
           dict(good, grid=65), dict(good, gamma_min=0.0), dict(good, gamma_max=1e-6),
           dict(good, eps_us=0.0)]
    for b in bad:
        lg = oracle.log(a, p, d, e, W.BOOST, gamma=1e-3, ada=b)
        assert lg["rc"] == oracle.EINVAL, b
    lg = oracle.log(a, p, d, e, W.BOOST, gamma=0.5, ada=good)  # gamma0 above gamma_max
    assert lg["rc"] == oracle.EINVAL
    lg = oracle.log(a, p, d, e, W.FCFS, gamma=1e-3, ada=good)  # adaptive gamma is BOOST only
    assert lg["rc"] == oracle.EINVAL


def test_golden_values_follow_closed_forms():
    """The stored adaptive-gamma cases agree with their closed-form derivation
    (tests/golden/ada_hand_calc.py: isolated-request latencies, the tail-band
    estimator, the EMA and the clip), independently of the oracle."""
    import json
    import sys

    sys.path.insert(0, os.path.join(os.path.dirname(__file__), "golden"))
    import ada_hand_calc as C

    cases = {c["name"]: c for c in json.load(open(os.path.join(
        os.path.dirname(__file__), "golden", "ada_hand.json")))["cases"]}
    exp = C.expected()
    assert set(exp) <= set(cases)
    for name, e in exp.items():
        assert cases[name]["gamma_final"] == pytest.approx(e["gamma_final"], rel=1e-12), name
    assert cases["ada_estimator"]["ttlt"][:20] == exp["ada_estimator"]["ttlt_alone"]
    assert cases["ada_eps_floor"]["ttlt"] == [C.alone(100, 5)] * 21
