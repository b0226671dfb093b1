"""Benchmark: simulated request-iterations per second on one MI355X.

One step = one pass of the whole path over one synthetic sweep: the
simulation kernel over every (trace, policy setting) instance, then the
percentile kernel. Inputs (traces, settings) are resident in HBM before the
timed region. Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 4]
                 [--grid sweep|ada|comparators|ladder|cache] [--no-ada]

Roofline: the simulation kernel is counted against HBM bandwidth with
algorithmic bytes of 32 B per request-iteration (read + write of the request's
kv / emitted / last-token / max-gap state) plus 28 B per request-instance
(16 B of trace in, 12 B of latencies out). `traffic` comes from the committed
rocprofv3 counter summary when it was taken on the current kernel sources.
The CPU baseline is the oracle, timed on the host cores over three traces'
settings (a bounded sample of the same sweep).
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
BYTES_PER_REQITER = 32
BYTES_PER_REQINST = 28
COUNTERS_FILE = os.path.join(ROOT, "profiles", "sim_kernel_counters.json")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("tas_sim.hip", "tas_internal.h"):
        h.update(open(os.path.join(ROOT, "paper_2606_18431_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch from the committed counter summary, if it matches
    the current kernel source and workload; else None."""
    try:
        d = json.load(open(COUNTERS_FILE))
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != kernel_source_hash() or d.get("workload") != workload:
        return None
    return d.get("hbm_bytes_per_launch")


def host_cpus():
    """(logical CPUs of the host, CPUs this process may run on, CPU model)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        allowed = len(os.sched_getaffinity(0))
    except AttributeError:
        allowed = os.cpu_count() or 1
    return os.cpu_count() or 1, allowed, model


def default_cpu_threads() -> int:
    # every CPU this process may use, up to 16 (a one-GPU share of the host)
    return max(1, min(16, host_cpus()[1]))


def cpu_sample(w):
    """The CPU baseline's sample: the first three traces under every setting."""
    traces = np.unique(w.settings["trace"])[:3]
    return traces, np.nonzero(np.isin(w.settings["trace"], traces))[0]


def cpu_baseline(w, n_threads: int):
    import oracle

    oracle.build()
    # 10-20 s of oracle work on 16 threads at the large sweep
    traces, sel = cpu_sample(w)
    sub = w.subset(sel)
    tic = time.perf_counter()
    o = oracle.run(sub, n_threads=n_threads)
    dt = time.perf_counter() - tic
    reqit = int(o["counters"][:, 1].sum())
    nproc, allowed, model = host_cpus()
    return o, sel, dict(value=reqit / dt, unit="request-iterations/s", cores=n_threads,
                        kind="oracle", seconds=round(dt, 3), host_cpus=nproc,
                        cpus_allowed=allowed, cpu_model=model,
                        sample=f"traces {', '.join(str(int(t)) for t in traces)} under every setting "
                               f"({len(sel)} of {w.n_inst} instances, {reqit} request-iterations)")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=4, choices=[0, 1, 2, 3, 4, 5])
    ap.add_argument("--traces", type=int, default=None, help="shrink the sweep (testing)")
    ap.add_argument("--grid", default="sweep",
                    choices=["sweep", "ada", "comparators", "ladder", "cache", "sensitivity"],
                    help="settings grid per trace (default: the gamma sweep)")
    ap.add_argument("--chunk", type=int, default=0,
                    help="prefill chunk in tokens instead of the workload's (the paper's chunk "
                         "sensitivity: 128 / 512 / 1024 / 2048)")
    ap.add_argument("--no-ada", action="store_true",
                    help="run the adaptive settings of the grid with gamma fixed at its start")
    ap.add_argument("--cluster", type=int, default=0,
                    help="R > 0: clusters of R replicas behind a global router (the workload's "
                         "traces, R times the rate, split by --dispatch); reports the cluster "
                         "percentiles pooled over each cluster's replicas")
    ap.add_argument("--dispatch", default="rr", choices=["rr", "random", "jsq"],
                    help="global router: round robin, balanced random (both split the traces "
                         "before the run), or join-shortest-queue (decided during the run, "
                         "one workgroup per cluster)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU baseline")
    ap.add_argument("--cpu-threads", type=int, default=0,
                    help="oracle threads (default: every CPU this process may use, up to 16)")
    ap.add_argument("--list-cap", type=int, default=0,
                    help="on-chip candidate list per instance (0: the library default)")
    ap.add_argument("--check", action="store_true",
                    help="run the checking build (libtas_check.so): every instance's state is "
                         "verified after each iteration")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (the reference for "
                         "scaling rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this path runs on one GPU; --gpus {args.gpus} is not supported "
              "(instances are independent: several GPUs would each take a block of traces)",
              file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2606_18431_amd import tas
    from paper_2606_18431_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        n = 1 << 30
        src = torch.ones(n // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "ok": bool(dst[-1].item() == 1)}))
        return
    if args.cluster:
        R = args.cluster
        n_cl = args.traces or max(1, W.SHAPES[args.workload][0] // R)
        w = W.make_cluster(args.workload, n_clusters=n_cl, replicas=R, dispatch=args.dispatch,
                           n_req=W.SHAPES[args.workload][2] // R)
        per_rep = w.n_req // R if args.dispatch == "jsq" else w.n_req
        name = f"{W.NAMES[args.workload]}: {n_cl} clusters x {R} replicas ({args.dispatch} " \
               f"dispatch) x {w.meta['n_settings']} settings x {per_rep} requests per replica"
    else:
        w = W.make(args.workload, n_traces=args.traces, grid=args.grid)
        name = f"{W.NAMES[args.workload]}: {w.n_traces} traces x {w.meta['n_settings']} " \
               f"settings x {w.n_req} requests"
    if args.grid != "sweep":
        name += f", {args.grid} settings grid"
    if args.no_ada:
        w.settings["ada"] = 0
        name += " with gamma fixed"
    if args.chunk:
        w.engine = dataclasses.replace(w.engine, chunk=args.chunk)
        name += f", chunk {args.chunk}"
    if args.check:
        tas.select_library(tas.CHECK_LIB_PATH)
        name += ", checking build"
    print(f"[bench] building {name}", file=sys.stderr, flush=True)
    sim = tas.Simulation(w, device=dev, list_cap=args.list_cap)
    stream = torch.cuda.current_stream()

    first_ms = None  # the first launch: instances in the launch order estimated from the inputs
    for i in range(args.warmup):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        sim.run(stream)
        e1.record(stream)
        sim.percentiles(stream)
        torch.cuda.synchronize()
        if i == 0:
            first_ms = float(e0.elapsed_time(e1))
        print(f"[bench] warmup {i} done", file=sys.stderr, flush=True)

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    tic = time.perf_counter()
    for e0, e1, e2 in ev:
        e0.record(stream)
        sim.run(stream)
        e1.record(stream)
        sim.percentiles(stream)
        e2.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - tic
    sim_ms = float(np.mean([a.elapsed_time(b) for a, b, _ in ev]))
    pct_ms = float(np.mean([b.elapsed_time(c) for _, b, c in ev]))
    step_ms = float(np.mean([a.elapsed_time(c) for a, _, c in ev]))
    out = sim.results(latencies=False)
    # LAS can starve a long request past the 32-bit latency range at full load;
    # the comparator grid reports those instances instead of failing
    overflowed = int(np.sum(out["status"] == tas.TAS_EOVERFLOW))
    tolerated = args.grid == "comparators" and bool(
        np.all(np.isin(out["status"], (0, tas.TAS_EOVERFLOW))))
    if out["rc"] != 0 and not tolerated:
        print(f"[bench] device error {out['rc']}: {tas.tas_strerror(out['rc'])}", file=sys.stderr)
        sys.exit(1)
    reqiters = int(out["counters"][:, 1].sum())
    iters = int(out["counters"][:, 0].sum())
    n_reqinst = w.n_inst * w.n_req
    value = reqiters / (step_ms / 1e3)
    alg_bytes = BYTES_PER_REQITER * reqiters + BYTES_PER_REQINST * n_reqinst
    achieved = alg_bytes / (sim_ms / 1e3) / 1e9
    traffic = measured_traffic(name)

    res = {
        "metric": "simulated request-iterations/sec (1 GPU)",
        "value": value,
        "unit": "request-iterations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": step_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic (seeded traces; no datasets)",
        "config": {"workload": name, "instances": w.n_inst, "requests_per_instance": w.n_req,
                   "max_seqs": w.engine.max_seqs, "max_tokens": w.engine.max_tokens,
                   "kv_blocks": w.engine.kv_blocks, "request_iterations": reqiters,
                   "iterations": iters, "sim_kernel_ms": sim_ms, "pctl_kernel_ms": pct_ms,
                   "first_launch_sim_kernel_ms": first_ms,
                   "wall_s": wall, "lds_list_cap": tas.tas_list_cap(sim.ctx),
                   "overflowed_instances": overflowed},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS, "traffic": traffic,
                     "kernel": "cluster_kernel" if args.cluster and args.dispatch == "jsq"
                     else "sim_kernel",
                     "algorithmic_bytes_per_launch": alg_bytes},
    }
    if args.cluster:  # cluster percentiles pooled over each cluster's replicas
        S = w.meta["n_settings"]
        if args.dispatch == "jsq":  # one instance per (cluster, setting) already
            gp, stride = out["pct"].astype(np.int64), 1
        else:
            gp, stride = sim.group_percentiles(args.cluster).astype(np.int64), args.cluster
        per = gp.reshape(w.meta["n_clusters"], S, 3, 3)
        res["config"]["cluster_p99_ttlt_us_mean"] = {
            W.POLICY_NAMES[int(w.settings["policy"][s * stride])] + f"_s{s}":
            float(per[:, s, 1, 2].mean()) for s in range(S)}
        res["config"]["cluster_p99_tbt_us_mean"] = {
            W.POLICY_NAMES[int(w.settings["policy"][s * stride])] + f"_s{s}":
            float(per[:, s, 2, 2].mean()) for s in range(S)}
    if not args.cluster:
        # P99 TTFT / TTLT / TBT (us) per setting, averaged over the traces where
        # it finished; the 64-setting sweep shows FCFS, SRPT and the UniBoost /
        # vanilla pair nearest gamma = 1e-3
        S = w.meta["n_settings"]
        p99 = out["pct"].astype(np.float64).reshape(-1, S, 3, 3)[:, :, :, 2]
        ok = (out["status"] == 0).reshape(-1, S)
        pick = list(range(S))
        if S > 9:
            g = np.abs(np.log10(w.settings["gamma"][2:S]) + 3.0)
            s0 = 2 + 2 * (int(np.argmin(g)) // 2)
            pick = [0, 1, s0, s0 + 1]
        res["config"]["p99_us_ttft_ttlt_tbt"] = {
            W.POLICY_NAMES[int(w.settings["policy"][s])] + f"_s{s}":
            [float(v) for v in p99[ok[:, s], s].mean(axis=0)] for s in pick if ok[:, s].any()}
    if args.grid == "comparators" and not args.cluster:
        # percentile slowdown against UniBoost on the same trace (the paper's
        # 100 (M_pi(p) / M_UniBoost(p) - 1)), TTLT at P50 / P90 / P99
        S = w.meta["n_settings"]
        pct = out["pct"].astype(np.float64).reshape(-1, S, 3, 3)[:, :, 1, :]
        ok = (out["status"] == 0).reshape(-1, S)
        uni = next(s for s in range(S) if int(w.settings["policy"][s]) == W.BOOST)
        res["config"]["ttlt_slowdown_vs_uniboost_pct"] = {  # traces where both finished
            W.POLICY_NAMES[int(w.settings["policy"][s])] + f"_s{s}":
            [float(v) for v in (100.0 * (pct[:, s] / pct[:, uni] - 1.0))[ok[:, s] & ok[:, uni]]
             .mean(axis=0)]
            for s in range(S) if s != uni}
    if args.workload == 5 and not args.cluster:  # short and long requests apart
        lat = sim.results()["ttlt"].astype(np.float64) / 1e6
        longm = np.asarray(w.decode)[w.settings["trace"]] == 6000
        S = w.meta["n_settings"]
        for cls, m in (("short", ~longm), ("long", longm)):
            res["config"][f"{cls}_ttlt_s"] = {
                W.POLICY_NAMES[int(w.settings["policy"][s])] + f"_s{s}": {
                    "mean": float(np.mean([lat[i][m[i]].mean() for i in range(s, w.n_inst, S)])),
                    "p99": float(np.mean([np.percentile(lat[i][m[i]], 99, method="inverted_cdf")
                                          for i in range(s, w.n_inst, S)]))}
                for s in range(S)}
    timed = None
    if not args.no_cpu and not args.cluster:
        # the CPU sample's outputs of the last timed launch, kept for the parity check
        _, sel = cpu_sample(w)
        lat = [torch.empty((w.n_inst, w.n_req), dtype=torch.int32, device=dev) for _ in range(3)]
        tas.tas_latencies(sim.ctx, *lat, stream=stream)
        ix = torch.as_tensor(sel, device=dev)
        timed = {k: t.index_select(0, ix).cpu().numpy().view(np.uint32)
                 for k, t in zip(("ttft", "ttlt", "tbtmax"), lat)}
        del lat
        for k in ("counters", "pct", "status"):
            timed[k] = out[k][sel]
    sim.close()
    if timed is not None:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        o, sel, cb = cpu_baseline(w, args.cpu_threads or default_cpu_threads())
        res["cpu_baseline"] = cb
        # the sample, checked element by element against the timed launch's outputs
        bad = [k for k in ("ttft", "ttlt", "tbtmax", "counters", "pct", "status")
               if not np.array_equal(timed[k], o[k])]
        res["sample_parity"] = not bad
        if bad:
            res["sample_parity_mismatch"] = bad
    print(json.dumps(res))
    if res.get("sample_parity") is False:
        print(f"[bench] the timed launch differs from the oracle: {res['sample_parity_mismatch']}",
              file=sys.stderr)
        sys.exit(1)


if __name__ == "__main__":
    main()
