"""CPU oracle of the tail-aware serving simulation (ctypes binding).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg. The product package never imports it, and it
imports nothing from the product package except the seeded input records
(``paper_2606_18431_amd.workloads``, which holds no scheduling arithmetic).

The C source (``tas_oracle.c``) is plain and sequential; see its header for the
paper passages it follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "tas_oracle.c")
LIB = os.path.join(HERE, "libtas_oracle.so")
LEVELS = 24
EINVAL, EINFEASIBLE, EOVERFLOW, ELIVELOCK, ESTATE = -1, -2, -5, -6, -7


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, plain C11, pthreads)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        # -ffp-contract=off: every floating-point step of the adaptive gamma is one
        # rounded IEEE operation (no fused multiply-add)
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-D_GNU_SOURCE", "-fPIC", "-shared",
                               "-ffp-contract=off", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm",
                               "-lpthread"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        L.tas_oracle_boost_table.argtypes = [f64, i32, f64, P]
        L.tas_oracle_boost_table.restype = ctypes.c_int
        L.tas_oracle_run.argtypes = [i32, i32, P, P, P, P, i32, P, P, P, P, P, P, P, i64,
                                     P, P, P, P, P, P, P, P, P, P, P, i32]
        L.tas_oracle_run.restype = ctypes.c_int
        L.tas_oracle_log.argtypes = [i32, P, P, P, P, i32, i32, i32, i64, P, P, i32, P, P, i64,
                                     P, P, P, P, P, i64, P, i64, P, i64, P, P, P]
        L.tas_oracle_jsq.argtypes = [i32, P, P, P, P, i32, i32, i32, i32, i64, P, P, i32, P, P,
                                     i64, P, P, P, P, P, P, P]
        L.tas_oracle_jsq.restype = ctypes.c_int
        L.tas_oracle_ada_grid.argtypes = [P, i32, P, P, P]
        L.tas_oracle_ada_grid.restype = ctypes.c_int
        L.tas_oracle_log.restype = ctypes.c_int
        L.tas_oracle_level.argtypes = [i64, i32]
        L.tas_oracle_level.restype = ctypes.c_int32
        L.tas_oracle_percentile.argtypes = [P, i32, i32]
        L.tas_oracle_percentile.restype = ctypes.c_uint32
        _lib = L
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _cached(h, shape):
    """Expected prefix-cache hit tokens as a contiguous int32 array, or None."""
    if h is None:
        return None
    h = np.ascontiguousarray(h, np.int32)
    assert h.shape == shape, (h.shape, shape)
    return h


def boost_table(gamma: float, k: int, tau_us: float = 5000.0) -> np.ndarray:
    out = np.zeros(LEVELS, np.int64)
    rc = lib().tas_oracle_boost_table(float(gamma), int(k), float(tau_us), _p(out))
    if rc:
        raise ValueError(f"boost table rejected (gamma={gamma}, k={k}, tau={tau_us})")
    return out


def tables(settings: np.ndarray, tau_us: float) -> np.ndarray:
    """The oracle's own boost tables for a settings array: an explicit table
    where one is given, else the table of gamma; zeros for FCFS/SRPT."""
    out = np.zeros((len(settings), LEVELS), np.int64)
    for i, s in enumerate(settings):
        if int(s["policy"]) not in (2, 7):  # the boost policies
            continue
        if int(s["table_given"]):
            out[i] = s["boost_us"]
        else:
            out[i] = boost_table(float(s["gamma"]), int(s["k"]), tau_us)
    return out


ADA_FIELDS = ("ada_beta", "ada_gamma_min", "ada_gamma_max", "ada_eps_us", "ada_window",
              "ada_min_samples", "ada_grid")


def ada_params(s, tau_us: float) -> np.ndarray:
    """The oracle's 10 adaptive-gamma parameters of one setting record
    {on, gamma0, beta, gamma_min, gamma_max, eps_us, window, min_samples,
    grid, tau_us} (on = 0 when the setting does not adapt gamma)."""
    if not int(s["ada"]):
        return np.zeros(10, np.float64)
    return np.array([1.0, float(s["gamma"])] + [float(s[f]) for f in ADA_FIELDS] +
                    [float(tau_us)], np.float64)


def ada_grid(s, tau_us: float = 5000.0):
    """(grid [G], midpoints [G-1], tables [G, 24]) of an adaptive setting."""
    prm = ada_params(s, tau_us)
    G = int(s["ada_grid"])
    grid, bound = np.zeros(64, np.float64), np.zeros(64, np.float64)
    tab = np.zeros((64, LEVELS), np.int64)
    rc = lib().tas_oracle_ada_grid(_p(prm), int(s["k"]), _p(grid), _p(bound), _p(tab))
    if rc:
        raise ValueError("adaptive-gamma parameters rejected")
    return grid[:G].copy(), bound[:G - 1].copy(), tab[:G].copy()


def _eng(engine) -> np.ndarray:
    return np.array([engine.max_seqs, engine.max_tokens, engine.chunk, engine.kv_blocks,
                     engine.block_tokens, engine.iter_base_us, engine.iter_tok_us,
                     engine.iter_ctx_div], np.int32)


def run(w, n_threads: int | None = None, max_iters: int | None = None):
    """Simulate every instance of workload ``w``. Returns a dict of host arrays:
    ttft/ttlt/tbtmax [n_inst, n_req] uint32, counters [n_inst, 8] int64,
    pct [n_inst, 3, 3] uint32, status [n_inst] int32, gamma [n_inst] float64
    (final adaptive gamma, 0 when fixed), switches [n_inst] int64, rc."""
    s = w.settings
    n_inst, n_req = len(s), w.n_req
    arr = np.ascontiguousarray(w.arrival_us, np.int64)
    pr = np.ascontiguousarray(w.prompt, np.int32)
    de = np.ascontiguousarray(w.decode, np.int32)
    ch = _cached(w.cached, de.shape)
    tr = np.ascontiguousarray(s["trace"], np.int32)
    po = np.ascontiguousarray(s["policy"], np.int32)
    kk = np.ascontiguousarray(s["k"], np.int32)
    mg = np.ascontiguousarray(s["memguard"], np.int32)
    dl = np.ascontiguousarray(s["delta_us"], np.int64)
    tb = np.ascontiguousarray(tables(s, w.engine.tau_us))
    ada = np.ascontiguousarray(np.stack([ada_params(x, w.engine.tau_us) for x in s])
                               if n_inst else np.zeros((0, 10)), np.float64)
    sg = np.ascontiguousarray(s["signal"], np.int32)
    lt = np.ascontiguousarray(np.stack([s["ltr_starve"], s["ltr_quantum"]], axis=1)
                              if n_inst else np.zeros((0, 2)), np.int32)
    out = dict(
        ttft=np.zeros((n_inst, n_req), np.uint32),
        ttlt=np.zeros((n_inst, n_req), np.uint32),
        tbtmax=np.zeros((n_inst, n_req), np.uint32),
        counters=np.zeros((n_inst, 8), np.int64),
        pct=np.zeros((n_inst, 3, 3), np.uint32),
        status=np.zeros(n_inst, np.int32),
        gamma=np.zeros(n_inst, np.float64),
        switches=np.zeros(n_inst, np.int64),
    )
    mi = w.engine.max_iters if max_iters is None else max_iters
    nt = n_threads or os.cpu_count() or 1
    rc = lib().tas_oracle_run(w.n_traces, n_req, _p(arr), _p(pr), _p(de),
                              None if ch is None else _p(ch), n_inst, _p(tr),
                              _p(po), _p(kk), _p(mg), _p(dl), _p(tb), _p(_eng(w.engine)),
                              int(mi), _p(out["ttft"]), _p(out["ttlt"]), _p(out["tbtmax"]),
                              _p(out["counters"]), _p(out["pct"]), _p(out["status"]), _p(ada),
                              _p(sg), _p(lt), _p(out["gamma"]), _p(out["switches"]), int(nt))
    out["rc"] = rc
    return out


def log(arrival, prompt, decode, engine, policy, k=1, memguard=0, delta_us=0, table=None,
        gamma=None, ada=None, signal=0, cached=None, max_iters=None, cap_iter=1 << 20,
        cap_batch=1 << 22, cap_evict=1 << 20, ltr=None):
    """Run one instance and return its schedule log (see tas_oracle.h). ``ada``:
    adaptive-gamma parameters as in workloads.ADA (gamma is the start);
    ``cached``: expected prefix-cache hit tokens per request (signal 2);
    ``ltr``: (starvation threshold, quantum) of an LTR instance."""
    arrival = np.ascontiguousarray(arrival, np.int64)
    prompt = np.ascontiguousarray(prompt, np.int32)
    decode = np.ascontiguousarray(decode, np.int32)
    ch = _cached(cached, decode.shape)
    n = len(arrival)
    if table is None:
        table = (boost_table(gamma, k, engine.tau_us) if gamma is not None
                 else np.zeros(LEVELS, np.int64))
    table = np.ascontiguousarray(table, np.int64)
    prm = np.zeros(10, np.float64)
    if ada is not None:
        prm = np.array([1.0, float(gamma), ada["beta"], ada["gamma_min"], ada["gamma_max"],
                        ada["eps_us"], ada["window"], ada["min_samples"], ada["grid"],
                        float(engine.tau_us)], np.float64)
    o = dict(ttft=np.zeros(n, np.uint32), ttlt=np.zeros(n, np.uint32),
             tbtmax=np.zeros(n, np.uint32), counters=np.zeros(8, np.int64))
    it = np.zeros((cap_iter, 8), np.int64)
    bt = np.zeros((cap_batch, 2), np.int32)
    ev = np.zeros((cap_evict, 4), np.int64)
    ni, nb, ne = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    mi = engine.max_iters if max_iters is None else max_iters
    lt = None if ltr is None else np.ascontiguousarray(ltr, np.int32)
    rc = lib().tas_oracle_log(n, _p(arrival), _p(prompt), _p(decode),
                              None if ch is None else _p(ch), policy, k, memguard,
                              int(delta_us), _p(table), _p(prm), int(signal),
                              None if lt is None else _p(lt), _p(_eng(engine)), int(mi),
                              _p(o["ttft"]), _p(o["ttlt"]), _p(o["tbtmax"]), _p(o["counters"]),
                              _p(it), cap_iter, _p(bt), cap_batch, _p(ev), cap_evict,
                              ctypes.byref(ni), ctypes.byref(nb), ctypes.byref(ne))
    o["rc"] = rc
    o["iters"] = it[: ni.value, :6].copy()
    o["cell"] = it[: ni.value, 6].copy()
    o["gamma"] = it[: ni.value, 7].copy().view(np.float64)
    o["batch"] = bt[: nb.value].copy()
    o["evict"] = ev[: ne.value].copy()
    return o


def level(w: int, k: int) -> int:
    return int(lib().tas_oracle_level(int(w), int(k)))


def group_percentiles(out, group: int) -> np.ndarray:
    """Nearest-rank percentiles pooled over groups of `group` adjacent
    instances of an oracle.run() result: [n_inst/group, 3, 3]."""
    n = out["ttft"].shape[0] // group
    res = np.zeros((n, 3, 3), np.uint32)
    for g in range(n):
        for m, key in enumerate(("ttft", "ttlt", "tbtmax")):
            pooled = np.ascontiguousarray(out[key][g * group:(g + 1) * group].ravel())
            for j, q in enumerate((50, 90, 99)):
                res[g, m, j] = percentile(pooled, q)
    return res


def percentile(values: np.ndarray, q: int) -> int:
    v = np.ascontiguousarray(values, np.uint32)
    return int(lib().tas_oracle_percentile(_p(v), len(v), int(q)))


def jsq(w, replicas: int, n_threads: int | None = None, max_iters: int | None = None):
    """Every instance of workload ``w`` as a cluster of ``replicas`` replicas
    behind a join-shortest-queue router over the instance's trace (see
    tas_oracle_jsq). Returns ttft/ttlt/tbtmax and assign [n_inst, n_req],
    counters [n_inst, replicas, 8], gamma and switches [n_inst, replicas],
    pct [n_inst, 3, 3] (nearest rank over the whole trace), status [n_inst]."""
    from concurrent.futures import ThreadPoolExecutor

    s = w.settings
    n_inst, n_req, R = len(s), w.n_req, int(replicas)
    tb = np.ascontiguousarray(tables(s, w.engine.tau_us))
    eng = _eng(w.engine)
    mi = w.engine.max_iters if max_iters is None else max_iters
    out = dict(ttft=np.zeros((n_inst, n_req), np.uint32), ttlt=np.zeros((n_inst, n_req), np.uint32),
               tbtmax=np.zeros((n_inst, n_req), np.uint32),
               assign=np.zeros((n_inst, n_req), np.int32),
               counters=np.zeros((n_inst, R, 8), np.int64), gamma=np.zeros((n_inst, R)),
               switches=np.zeros((n_inst, R), np.int64), pct=np.zeros((n_inst, 3, 3), np.uint32),
               status=np.zeros(n_inst, np.int32))

    def one(i):
        t = int(s[i]["trace"])
        arr = np.ascontiguousarray(w.arrival_us[t], np.int64)
        pr = np.ascontiguousarray(w.prompt[t], np.int32)
        de = np.ascontiguousarray(w.decode[t], np.int32)
        ch = None if w.cached is None else np.ascontiguousarray(w.cached[t], np.int32)
        prm = np.ascontiguousarray(ada_params(s[i], w.engine.tau_us), np.float64)
        lt = np.array([s[i]["ltr_starve"], s[i]["ltr_quantum"]], np.int32)
        bufs = [np.zeros(n_req, np.uint32) for _ in range(3)] + [np.zeros(n_req, np.int32),
                                                                  np.zeros((R, 8), np.int64),
                                                                  np.zeros(R), np.zeros(R, np.int64)]
        rc = lib().tas_oracle_jsq(n_req, _p(arr), _p(pr), _p(de), None if ch is None else _p(ch),
                                  R, int(s[i]["policy"]), int(s[i]["k"]), int(s[i]["memguard"]),
                                  int(s[i]["delta_us"]), _p(tb[i]), _p(prm), int(s[i]["signal"]),
                                  _p(lt), _p(eng), int(mi), *[_p(b) for b in bufs])
        out["status"][i] = rc
        if rc == 0:
            for key, b in zip(("ttft", "ttlt", "tbtmax", "assign", "counters", "gamma",
                               "switches"), bufs):
                out[key][i] = b
            for m, key in enumerate(("ttft", "ttlt", "tbtmax")):
                for j, q in enumerate((50, 90, 99)):
                    out["pct"][i, m, j] = percentile(bufs[m], q)

    nt = max(1, min(n_threads or os.cpu_count() or 1, n_inst))
    with ThreadPoolExecutor(nt) as ex:
        list(ex.map(one, range(n_inst)))
    out["rc"] = int(next((x for x in out["status"] if x), 0))
    return out
