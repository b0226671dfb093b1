"""Seeded synthetic serving workloads: request traces and policy-setting grids.

This module only draws inputs. It holds none of the scheduling arithmetic: no
priorities, no boost curve, no batch formation. Both the HIP path and the CPU
oracle consume exactly the arrays produced here.

Request model (paper, section "Formulation", Notation): request i is the tuple
(a_i arrival time, s_pre prompt length known at arrival, s_dec decode length
not revealed to a blind policy). Traces are stored structure-of-arrays,
trace-major, arrival-sorted: ``arrival_us[t, i]`` (int64 microseconds,
non-decreasing in i), ``prompt[t, i]`` and ``decode[t, i]`` (int32 tokens, >= 1).

Five workloads are defined (``make(cfg)``):

0  tiny: 1 trace x 8 settings, 1,000 requests, Poisson 4 req/s, seed 0.
1  chat-heavy sweep: 64 traces x 64 settings, 10,000 requests, utilisation 0.85.
2  reasoning-heavy under KV pressure: 64 x 64, 10,000 requests, 8,192 KV blocks.
3  bursty arrivals + decode-length shift: 128 x 32, 20,000 requests, 2-state MMPP.
4  large sweep: 256 x 64, 50,000 requests, 60/40 blend of the 1 and 2 laws.
5  starvation: 32 x 8, 20,000 requests, 90% short (~125 / 100) and 10% long
   (2000 / 6000) requests, Poisson at utilisation 0.99 (the paper's
   starvation study), under its policies (UniBoost, Sarathi, SJF, SRPT, ...).

The policy-parameter grid per trace: setting 0 = FCFS, setting 1 = oracle-length
SRPT, then pairs (UniBoost with MemGuard, vanilla boost) over log-spaced gamma.
``make(cfg, grid="comparators")`` instead runs every trace under the paper's
comparison policies (FCFS, SRPT, SPF, SJF, LAS, TRAIL, Sarathi) beside UniBoost
and vanilla boost; ``make(cfg, grid="ada")`` runs fixed against adaptive gamma (Phase 4);
``make(cfg, grid="ladder")`` runs the paper's design phases (DistBoost to the
full UniBoost) and the phase-aware signal.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

FCFS, SRPT, BOOST, SPF, SJF, LAS, TRAIL, DIST, SARATHI, LTR = 0, 1, 2, 3, 4, 5, 6, 7, 8, 9
POLICY_NAMES = {FCFS: "fcfs", SRPT: "srpt", BOOST: "boost", SPF: "spf", SJF: "sjf", LAS: "las",
                TRAIL: "trail", DIST: "distboost", SARATHI: "sarathi", LTR: "ltr"}
LEVELS = 24

# One numpy record per instance; field order mirrors the C struct tas_setting.
SETTING_DTYPE = np.dtype(
    [
        ("trace", np.int32),
        ("policy", np.int32),
        ("k", np.int32),
        ("memguard", np.int32),
        ("delta_us", np.int64),
        ("gamma", np.float64),
        ("table_given", np.int32),
        ("ada", np.int32),
        ("boost_us", np.int64, (LEVELS,)),
        ("ada_beta", np.float64),
        ("ada_gamma_min", np.float64),
        ("ada_gamma_max", np.float64),
        ("ada_eps_us", np.float64),
        ("ada_window", np.int32),
        ("ada_min_samples", np.int32),
        ("ada_grid", np.int32),
        ("signal", np.int32),
        ("ltr_starve", np.int32),
        ("ltr_quantum", np.int32),
    ]
)


@dataclasses.dataclass
class Engine:
    """Serving-engine limits and the integer iteration cost model.

    Iteration time in microseconds = base + tok * sum(n) + floor(sum(ctx) / div).
    """

    max_seqs: int = 64
    max_tokens: int = 8192
    chunk: int = 1024
    kv_blocks: int = 16384
    block_tokens: int = 16
    iter_base_us: int = 5000
    iter_tok_us: int = 2
    iter_ctx_div: int = 100
    max_iters: int = 4_000_000  # ends a runaway instance with a livelock error
    tau_us: float = 5000.0  # microseconds per token of boost (one decode step)


@dataclasses.dataclass
class Workload:
    name: str
    arrival_us: np.ndarray  # int64 [n_traces, n_req]
    prompt: np.ndarray  # int32 [n_traces, n_req]
    decode: np.ndarray  # int32 [n_traces, n_req]
    engine: Engine
    settings: np.ndarray  # SETTING_DTYPE [n_inst]
    meta: dict = dataclasses.field(default_factory=dict)
    # expected prefix-cache hit tokens, int32 [n_traces, n_req] with
    # 0 <= h < prompt, or None; read by settings with signal 2
    cached: np.ndarray | None = None

    @property
    def n_traces(self) -> int:
        return int(self.arrival_us.shape[0])

    @property
    def n_req(self) -> int:
        return int(self.arrival_us.shape[1])

    @property
    def n_inst(self) -> int:
        return int(self.settings.shape[0])

    def subset(self, inst_ids) -> "Workload":
        """The same traces with only the chosen instances (order kept)."""
        inst_ids = np.asarray(inst_ids, dtype=np.int64)
        return dataclasses.replace(self, settings=self.settings[inst_ids].copy())


# ---------------------------------------------------------------- settings


def setting(trace, policy, k=1, memguard=0, delta_us=0, gamma=0.0, table=None, ada=None,
            signal=0, ltr=None):
    """One instance record. ``ada``: adaptive-gamma parameters (keys of ADA
    without the ``ada_`` prefix, e.g. ``dict(ADA)``), gamma being the start.
    ``signal`` 1: Algorithm 2's phase-aware boost signal (BOOST); 2: the
    cache-aware signal P - h + dec (BOOST; needs the workload's ``cached``).
    ``ltr``: (starvation threshold, quantum) in iterations of an LTR setting
    (default LTR_CONTROL)."""
    s = np.zeros((), dtype=SETTING_DTYPE)
    s["trace"], s["policy"], s["k"], s["memguard"] = trace, policy, k, memguard
    s["delta_us"], s["gamma"], s["signal"] = delta_us, gamma, signal
    if policy == LTR:
        s["ltr_starve"], s["ltr_quantum"] = LTR_CONTROL if ltr is None else ltr
    if ada is not None:
        s["ada"] = 1
        for key, v in ada.items():
            s["ada_" + key] = v
    if table is not None:
        t = np.asarray(table, dtype=np.int64)
        s["boost_us"][: len(t)] = t
        s["boost_us"][len(t):] = t[-1] if len(t) else 0
        s["table_given"] = 1
    return s


UNIBOOST = dict(k=256, memguard=1, delta_us=100_000)  # defaults k=256, delta=0.1 s
# SJF (LTR+): a request not served for 512 iterations in a row (about 2.5-5 s
# at the workloads' 5-10 ms steps) is promoted for 64 iterations of service;
# the paper states the mechanism, not its parameters
LTR_CONTROL = (512, 64)
VANILLA = dict(k=1, memguard=0, delta_us=0)
# Adaptive gamma: EMA weight per iteration, clip bounds = grid ends (10 grid
# points per decade), floor of the tail band in us, window of completed
# requests and the samples needed before the first update.
ADA = dict(beta=0.01, gamma_min=1e-5, gamma_max=1e-1, eps_us=1000.0, window=256,
           min_samples=64, grid=41)


def settings_grid(n_traces: int, n_settings: int) -> np.ndarray:
    """Per trace: FCFS, SRPT, then (UniBoost, vanilla) pairs over a gamma grid
    log-spaced on [1e-5, 1e-1] per token. Instance id = trace * S + s."""
    assert n_settings >= 4 and n_settings % 2 == 0
    g = (n_settings - 2) // 2
    gammas = 10.0 ** np.linspace(-5.0, -1.0, g)
    out = np.zeros(n_traces * n_settings, dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s in range(n_settings):
            if s == 0:
                rec = setting(t, FCFS)
            elif s == 1:
                rec = setting(t, SRPT)
            else:
                var = VANILLA if (s - 2) % 2 else UNIBOOST
                rec = setting(t, BOOST, gamma=float(gammas[(s - 2) // 2]), **var)
            out[t * n_settings + s] = rec
    return out


def comparator_settings(n_traces: int, gamma: float = 1e-3) -> np.ndarray:
    """Per trace, 10 settings: FCFS, SRPT, SPF, SJF, LAS, TRAIL, then UniBoost and
    vanilla boost at one gamma, then Sarathi and SJF (LTR+). Instance id =
    trace * 10 + s."""
    per = [dict(policy=FCFS), dict(policy=SRPT), dict(policy=SPF), dict(policy=SJF),
           dict(policy=LAS), dict(policy=TRAIL), dict(policy=BOOST, gamma=gamma, **UNIBOOST),
           dict(policy=BOOST, gamma=gamma, **VANILLA), dict(policy=SARATHI), dict(policy=LTR)]
    out = np.zeros(n_traces * len(per), dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s, kw in enumerate(per):
            out[t * len(per) + s] = setting(t, **kw)
    return out


# ---------------------------------------------------------------- lengths


def _lognormal(rng, n, median, sigma, lo, hi):
    z = rng.standard_normal(n)
    return np.clip(np.rint(np.exp(math.log(median) + sigma * z)), lo, hi).astype(np.int32)


def _pareto(rng, n, alpha, xm, lo, hi):
    u = 1.0 - rng.random(n)  # (0, 1]
    return np.clip(np.rint(xm * u ** (-1.0 / alpha)), lo, hi).astype(np.int32)


def _decode_reasoning(rng, n):
    """80% lognormal(median 150, sigma 1) + 20% Pareto(alpha 1.5, min 2000), clip 32768."""
    heavy = rng.random(n) < 0.2
    ln = _lognormal(rng, n, 150, 1.0, 1, 32768)
    pa = _pareto(rng, n, 1.5, 2000, 1, 32768)
    return np.where(heavy, pa, ln).astype(np.int32)


# ---------------------------------------------------------------- load calibration


def offered_cost_us(prompt, decode, eng: Engine):
    """Expected busy microseconds each request adds, for arrival-rate calibration.

    Every iteration a request takes part in costs base/M_eff (its share of the
    fixed cost), plus tok per computed token, plus ctx/div per token of context.
    M_eff is the concurrency the KV budget allows. Calibration only: it sets the
    Poisson rate and never enters the simulation.
    """
    p = prompt.astype(np.float64)
    d = decode.astype(np.float64)
    c = float(eng.chunk)
    nch = np.ceil(p / c)
    mean_ctx = np.mean((p + d / 2.0) * d) / np.mean(d)
    m_eff = min(float(eng.max_seqs), eng.kv_blocks * eng.block_tokens / mean_ctx)
    prefill_ctx = c * (nch - 1.0) * nch / 2.0 + p
    decode_ctx = (d - 1.0) * p + (d - 1.0) * d / 2.0
    return (
        (nch + d - 1.0) * eng.iter_base_us / m_eff
        + eng.iter_tok_us * (p + d - 1.0)
        + (prefill_ctx + decode_ctx) / eng.iter_ctx_div
    )


def _poisson_arrivals(rng, n, lam_per_us):
    gaps = rng.exponential(1.0 / lam_per_us, n)
    return np.floor(np.cumsum(gaps)).astype(np.int64)


def _mmpp_arrivals(rng, n, lam0, lam1, dwell_us):
    """2-state Markov-modulated Poisson arrivals; start state drawn from the
    stationary law (equal mean dwell => 1/2 each)."""
    state = int(rng.random() < 0.5)
    t = 0.0
    out = []
    count = 0
    while count < n:
        d = rng.exponential(dwell_us)
        lam = lam1 if state else lam0
        expect = lam * d
        m = int(expect + 6.0 * math.sqrt(expect + 1.0) + 8)
        while True:
            gaps = rng.exponential(1.0 / lam, m)
            cs = np.cumsum(gaps)
            if cs[-1] > d:
                break
            m *= 2
        inside = t + cs[cs <= d]
        out.append(inside)
        count += inside.size
        t += d
        state ^= 1
    arr = np.concatenate(out)[:n]
    return np.floor(arr).astype(np.int64)


# ---------------------------------------------------------------- configs


def _engine(cfg: int) -> Engine:
    if cfg == 0:
        return Engine(kv_blocks=16384)
    if cfg == 1:
        return Engine(kv_blocks=32768)
    if cfg == 2:
        return Engine(kv_blocks=8192)
    if cfg == 3:
        return Engine(kv_blocks=16384)
    if cfg == 4:
        return Engine(max_seqs=256, max_tokens=16384, kv_blocks=32768)
    if cfg == 5:
        return Engine(kv_blocks=32768)
    raise ValueError(cfg)


SHAPES = {0: (1, 8, 1000), 1: (64, 64, 10000), 2: (64, 64, 10000), 3: (128, 32, 20000),
          4: (256, 64, 50000), 5: (32, 8, 20000)}
NAMES = {0: "tiny", 1: "chat-heavy", 2: "reasoning-kv-pressure", 3: "bursty-shift",
         4: "large-sweep", 5: "starvation"}


def _trace(cfg: int, trace: int, n: int, eng: Engine):
    rng = np.random.default_rng(0 if cfg == 0 else [cfg, trace])
    if cfg == 0:
        p = _lognormal(rng, n, 512, 1.0, 16, 4096)
        d = _lognormal(rng, n, 200, 1.2, 1, 8192)
        arr = _poisson_arrivals(rng, n, 4.0e-6)
        return arr, p, d
    if cfg == 1:
        p = _lognormal(rng, n, 768, 1.0, 16, 4096)
        d = _lognormal(rng, n, 180, 1.0, 1, 4096)
        rho = 0.85
    elif cfg == 2:
        p = _lognormal(rng, n, 256, 1.0, 16, 4096)
        d = _decode_reasoning(rng, n)
        rho = 0.9
    elif cfg == 3:
        p = _lognormal(rng, n, 512, 1.0, 16, 4096)
        half = n // 2
        d = np.concatenate([_lognormal(rng, half, 150, 1.2, 1, 8192),
                            _lognormal(rng, n - half, 900, 1.2, 1, 8192)])
        post = slice(half, n)
        lam_avg = 0.8 * (n - half) / offered_cost_us(p[post], d[post], eng).sum()
        lam_b = lam_avg / 3.5  # time-average rate of {1x, 6x} with equal dwell
        arr = _mmpp_arrivals(rng, n, lam_b, 6.0 * lam_b, 30.0e6)
        return arr, p, d
    elif cfg == 5:
        # the paper's starvation mix: 90% short (about 125 prompt, 100 output)
        # and 10% long (2000 prompt, 6000 output) requests, Poisson at 0.99
        long = rng.random(n) < 0.1
        p = np.where(long, 2000, _lognormal(rng, n, 125, 0.2, 64, 256)).astype(np.int32)
        d = np.where(long, 6000, 100).astype(np.int32)
        rho = 0.99
    elif cfg == 4:
        chat = rng.random(n) < 0.6
        p = np.where(chat, _lognormal(rng, n, 768, 1.0, 16, 4096),
                     _lognormal(rng, n, 256, 1.0, 16, 4096)).astype(np.int32)
        d = np.where(chat, _lognormal(rng, n, 180, 1.0, 1, 4096),
                     _decode_reasoning(rng, n)).astype(np.int32)
        rho = 0.95
    else:
        raise ValueError(cfg)
    lam = rho * n / offered_cost_us(p, d, eng).sum()
    arr = _poisson_arrivals(rng, n, lam)
    return arr, p, d


def cached_tokens(seed, prompt: np.ndarray, share: float = 0.5, new_median: float = 64.0,
                  new_sigma: float = 1.0) -> np.ndarray:
    """Expected prefix-cache hit tokens for a multi-turn mix (paper: interaction
    with prefix/radix caching, where the hits are the earlier turns' tokens). A
    ``share`` of the requests are follow-up turns whose prompt is the
    conversation so far plus a new message of lognormal length (median
    ``new_median`` tokens, clipped to [1, P]); their hits are P minus that
    message. The other requests are first turns with no hits. Seeded by
    ``seed`` on a stream of its own, so the traces are unchanged."""
    rng = np.random.default_rng([104729, *np.atleast_1d(seed).tolist()])
    p = np.asarray(prompt, np.int64)
    follow = rng.random(p.shape) < share
    z = rng.standard_normal(p.shape)
    new = np.clip(np.rint(np.exp(math.log(new_median) + new_sigma * z)), 1, p)
    return np.where(follow, p - new, 0).astype(np.int32)


def cache_settings(n_traces: int) -> np.ndarray:
    """Per trace, 8 settings: UniBoost at gamma 1e-3 and 1e-2 and vanilla boost
    at 1e-3, each with the signal P + dec and with the cache-aware signal
    P - h + dec, then FCFS and SRPT. Instance id = trace * 8 + s."""
    per = []
    for g, var in ((1e-3, UNIBOOST), (1e-2, UNIBOOST), (1e-3, VANILLA)):
        per.append(dict(policy=BOOST, gamma=g, **var))
        per.append(dict(policy=BOOST, gamma=g, signal=2, **var))
    per += [dict(policy=FCFS), dict(policy=SRPT)]
    out = np.zeros(n_traces * len(per), dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s, kw in enumerate(per):
            out[t * len(per) + s] = setting(t, **kw)
    return out


def starvation_settings(n_traces: int, gamma: float = 1e-3) -> np.ndarray:
    """Per trace, the policies of the paper's starvation study and their
    neighbours (8 settings): UniBoost at one gamma, Sarathi, SJF, SRPT, then
    FCFS, vanilla boost, TRAIL and DistBoost. (LAS starves the long requests
    past the 32-bit latency range at this load.) Instance id = trace * 8 + s."""
    per = [dict(policy=BOOST, gamma=gamma, **UNIBOOST), dict(policy=SARATHI), dict(policy=SJF),
           dict(policy=SRPT), dict(policy=FCFS), dict(policy=BOOST, gamma=gamma, **VANILLA),
           dict(policy=TRAIL), dict(policy=DIST, gamma=gamma)]
    out = np.zeros(n_traces * len(per), dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s, kw in enumerate(per):
            out[t * len(per) + s] = setting(t, **kw)
    return out


def sensitivity_settings(n_traces: int, gamma: float = 1e-3) -> np.ndarray:
    """Per trace, the paper's sensitivity study (UniBoost at one gamma): the
    bin size k in {64, 256, 512, 1024} tokens at delta 0.1 s, then the
    hysteresis delta in {0, 0.3, 0.5} s at k = 256, then FCFS (8 settings).
    Instance id = trace * 8 + s."""
    per = [dict(policy=BOOST, gamma=gamma, k=k, memguard=1, delta_us=100_000)
           for k in (64, 256, 512, 1024)]
    per += [dict(policy=BOOST, gamma=gamma, k=256, memguard=1, delta_us=d)
            for d in (0, 300_000, 500_000)]
    per.append(dict(policy=FCFS))
    out = np.zeros(n_traces * len(per), dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s, kw in enumerate(per):
            out[t * len(per) + s] = setting(t, **kw)
    return out


def ada_settings(n_traces: int, ada: dict | None = None) -> np.ndarray:
    """Per trace, 8 settings: for gamma0 in (1e-4, 1e-3, 1e-2) UniBoost with that
    fixed gamma and UniBoost with adaptive gamma started there, then vanilla
    boost with adaptive gamma from 1e-3, then FCFS. Instance id = trace * 8 + s."""
    ada = dict(ADA if ada is None else ada)
    per = []
    for g0 in (1e-4, 1e-3, 1e-2):
        per.append(dict(policy=BOOST, gamma=g0, **UNIBOOST))
        per.append(dict(policy=BOOST, gamma=g0, ada=ada, **UNIBOOST))
    per.append(dict(policy=BOOST, gamma=1e-3, ada=ada, **VANILLA))
    per.append(dict(policy=FCFS))
    out = np.zeros(n_traces * len(per), dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s, kw in enumerate(per):
            out[t * len(per) + s] = setting(t, **kw)
    return out


def ladder_settings(n_traces: int, gamma: float = 1e-3, ada: dict | None = None) -> np.ndarray:
    """Per trace, 8 settings along the paper's design phases at one gamma:
    DistBoost (Phase 1, k = 1), UniBoost-Base (Phase 2: k = 1, no MemGuard,
    hysteresis 0.1 s), + MemGuard (Phase 3: k = 256), + adaptive gamma (the
    full UniBoost), the Phase 3 setting and vanilla boost with Algorithm 2's
    phase-aware signal, then FCFS and SRPT. Instance id = trace * 8 + s."""
    ada = dict(ADA if ada is None else ada)
    per = [dict(policy=DIST, gamma=gamma, k=1),
           dict(policy=BOOST, gamma=gamma, k=1, memguard=0, delta_us=100_000),
           dict(policy=BOOST, gamma=gamma, **UNIBOOST),
           dict(policy=BOOST, gamma=gamma, ada=ada, **UNIBOOST),
           dict(policy=BOOST, gamma=gamma, signal=1, **UNIBOOST),
           dict(policy=BOOST, gamma=gamma, signal=1, **VANILLA),
           dict(policy=FCFS), dict(policy=SRPT)]
    out = np.zeros(n_traces * len(per), dtype=SETTING_DTYPE)
    for t in range(n_traces):
        for s, kw in enumerate(per):
            out[t * len(per) + s] = setting(t, **kw)
    return out


def make(cfg: int, n_traces: int | None = None, n_settings: int | None = None,
         n_req: int | None = None, grid: str = "sweep") -> Workload:
    """Build workload ``cfg``. The optional overrides shrink it (fewer traces,
    settings or requests) for tests; traces keep their seeds, so trace t of a
    shrunk workload equals trace t of the full one when n_req is unchanged.
    ``grid="comparators"`` replaces the settings grid by comparator_settings,
    ``grid="ada"`` by ada_settings, ``grid="ladder"`` by ladder_settings and
    ``grid="cache"`` by cache_settings, with expected prefix-cache hits drawn
    by cached_tokens for every trace, ``grid="sensitivity"`` by
    sensitivity_settings."""
    T0, S0, N0 = SHAPES[cfg]
    T = T0 if n_traces is None else n_traces
    S = S0 if n_settings is None else n_settings
    N = N0 if n_req is None else n_req
    eng = _engine(cfg)
    arr = np.empty((T, N), np.int64)
    pr = np.empty((T, N), np.int32)
    de = np.empty((T, N), np.int32)
    for t in range(T):
        arr[t], pr[t], de[t] = _trace(cfg, t, N, eng)
    if grid == "comparators":
        sets = comparator_settings(T)
        S = len(sets) // T
    elif grid == "ada":
        sets = ada_settings(T)
        S = 8
    elif grid == "ladder":
        sets = ladder_settings(T)
        S = 8
    elif grid == "cache":
        sets = cache_settings(T)
        S = 8
    elif grid == "sensitivity":
        sets = sensitivity_settings(T)
        S = 8
    elif cfg == 5:
        sets = starvation_settings(T)
        S = 8
    elif cfg == 0 and S == 8:
        st = [setting(0, FCFS), setting(0, SRPT)]
        st += [setting(0, BOOST, gamma=g, **UNIBOOST)
               for g in (1e-4, 3e-4, 1e-3, 3e-3, 1e-2, 3e-2)]
        sets = np.stack(st * T)
        sets["trace"] = np.repeat(np.arange(T), 8)
    else:
        sets = settings_grid(T, S)
    cached = None
    if grid == "cache":
        cached = np.stack([cached_tokens([cfg, t], pr[t]) for t in range(T)])
    return Workload(NAMES[cfg], arr, pr, de, eng, sets,
                    meta=dict(cfg=cfg, n_traces=T, n_settings=S, n_req=N, grid=grid),
                    cached=cached)


def make_cluster(cfg: int, n_clusters: int, replicas: int, dispatch: str = "rr",
                 n_req: int | None = None, settings: list | None = None) -> Workload:
    """Replicas behind a global router (paper: global dispatch policies and
    cluster scale). Cluster c receives the requests of one global trace: the
    trace of workload ``cfg`` with ``n_req * replicas`` requests whose time
    axis is compressed ``replicas`` times (the router sees ``replicas`` times
    the rate that loads one replica to the workload's utilisation). The
    router assigns them to replicas, each replica schedules its own requests:

    - ``dispatch="rr"``: round robin, request i goes to replica i mod R;
    - ``dispatch="random"``: balanced random, each block of R consecutive
      requests goes to a uniformly random permutation of the replicas (the
      assignment is drawn here, seeded, and is an input of both sides);
    - ``dispatch="jsq"``: join the shortest queue, decided during the
      simulation (the replica holding the fewest unfinished requests at the
      arrival, ties to the lowest). The workload then keeps the global traces
      whole (trace c = cluster c, R * n_req requests) with one instance per
      (cluster, setting); ``meta["replicas"]`` tells the simulation how many
      replicas each instance has.

    Every replica receives ``n_req`` requests. Instances are ordered cluster,
    setting, replica, so the R replicas of a (cluster, setting) are R adjacent
    instances (``tas_percentiles_grouped`` with group R reduces over them).
    Traces are ordered cluster, replica. ``settings``: keyword dicts for
    ``setting`` (default FCFS, UniBoost at gamma 1e-3, vanilla boost, Sarathi:
    the paper compares UniBoost with the Sarathi engine under each router)."""
    T0, _, N0 = SHAPES[cfg]
    N = N0 if n_req is None else n_req
    R = int(replicas)
    eng = _engine(cfg)
    per = settings if settings is not None else [
        dict(policy=FCFS), dict(policy=BOOST, gamma=1e-3, **UNIBOOST),
        dict(policy=BOOST, gamma=1e-3, **VANILLA), dict(policy=SARATHI)]
    if dispatch == "jsq":
        arr = np.empty((n_clusters, N * R), np.int64)
        pr = np.empty((n_clusters, N * R), np.int32)
        de = np.empty((n_clusters, N * R), np.int32)
        for c in range(n_clusters):
            a, p, d = _trace(cfg, c, N * R, eng)
            arr[c], pr[c], de[c] = a // R, p, d
        sets = np.stack([setting(c, **kw) for c in range(n_clusters) for kw in per])
        return Workload(f"{NAMES[cfg]} cluster", arr, pr, de, eng, sets,
                        meta=dict(cfg=cfg, n_clusters=n_clusters, replicas=R, dispatch=dispatch,
                                  n_settings=len(per), n_req=N))
    arr = np.empty((n_clusters * R, N), np.int64)
    pr = np.empty((n_clusters * R, N), np.int32)
    de = np.empty((n_clusters * R, N), np.int32)
    assign = np.empty((n_clusters, N * R), np.int32)
    for c in range(n_clusters):
        a, p, d = _trace(cfg, c, N * R, eng)
        a = a // R  # R times the arrival rate
        if dispatch == "rr":
            rep = np.arange(N * R, dtype=np.int64) % R
        elif dispatch == "random":
            rng = np.random.default_rng([cfg, c, R, 7919])
            rep = np.concatenate([rng.permutation(R) for _ in range(N)])
        else:
            raise ValueError(dispatch)
        assign[c] = rep
        for r in range(R):
            sel = np.nonzero(rep == r)[0]
            arr[c * R + r], pr[c * R + r], de[c * R + r] = a[sel], p[sel], d[sel]
    sets = np.zeros(n_clusters * len(per) * R, dtype=SETTING_DTYPE)
    i = 0
    for c in range(n_clusters):
        for kw in per:
            for r in range(R):
                sets[i] = setting(c * R + r, **kw)
                i += 1
    return Workload(f"{NAMES[cfg]} cluster", arr, pr, de, eng, sets,
                    meta=dict(cfg=cfg, n_clusters=n_clusters, replicas=R, dispatch=dispatch,
                              n_settings=len(per), n_req=N, assign=assign))


def small_random(seed: int, n_req: int, *, rate_per_s: float = 20.0, p_med=64, d_med=20,
                 p_max=512, d_max=256):
    """A small random trace (for tests): lognormal lengths, Poisson arrivals."""
    rng = np.random.default_rng([99, seed])
    p = _lognormal(rng, n_req, p_med, 1.0, 1, p_max)
    d = _lognormal(rng, n_req, d_med, 1.0, 1, d_max)
    arr = _poisson_arrivals(rng, n_req, rate_per_s * 1e-6)
    return arr, p, d
