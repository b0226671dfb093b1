"""Write fullsize_digests.json: the CPU oracle's per-instance output digests
for every instance of the chat-heavy, reasoning-heavy and bursty sweeps, for
the large sweep's checked subset (every 64th instance and all settings of
four traces), and for every instance of the large-sweep traces under the
comparator grid (SJF (LTR+) among them), the adaptive-gamma, phase-ladder and
cache-aware grids, and for every instance of the starvation mix. Calls only
the oracle and the seeded input generator.

    python tests/golden/make_fullsize_digests.py [--threads N] [--only KEY ...]

Keys: 1, 2, 3, 4, 4-comparators, 4-ada, 4-ladder, 4-cache, 5 (--only
recomputes those and keeps the rest of an existing file). About two hours on
8 host threads in all.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

import oracle  # noqa: E402
from paper_2606_18431_amd import workloads as W  # noqa: E402
from digests import input_digest, instance_digests, large_sweep_subset  # noqa: E402

OUT = os.path.join(HERE, "fullsize_digests.json")
KEYS = ("1", "2", "3", "4", "4-comparators", "4-ada", "4-ladder", "4-cache", "5")


def make(key: str):
    """The workload of a key: a configuration, or the large-sweep traces
    under another settings grid."""
    cfg, _, grid = key.partition("-")
    return W.make(int(cfg), grid=grid or "sweep")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    ap.add_argument("--only", nargs="*", default=None, help="keys to (re)compute")
    ap.add_argument("--inputs-only", action="store_true",
                    help="refresh only the input digests of an existing file (after a "
                         "change of the settings record that leaves the workloads alone)")
    args = ap.parse_args()
    if args.inputs_only:
        res = json.load(open(OUT))
        for key, ent in res["workloads"].items():
            ent["inputs"] = input_digest(make(key))
        with open(OUT, "w") as f:
            json.dump(res, f, indent=1)
            f.write("\n")
        return
    oracle.build()
    res = {"what": "oracle output digests per instance (see digests.py)", "workloads": {}}
    keys = KEYS
    if args.only is not None:
        res = json.load(open(OUT))
        keys = args.only
    for key in keys:
        w = make(key)
        cfg = int(key.split("-")[0])
        sel = large_sweep_subset(w) if key == "4" else None
        sub = w if sel is None else w.subset(sel)
        tic = time.perf_counter()
        o = oracle.run(sub, n_threads=args.threads)
        dt = time.perf_counter() - tic
        # LAS starves long requests past the 32-bit latency range under full
        # load: that status is part of the digest
        assert o["rc"] in (0, -5), (key, o["rc"])
        dig = instance_digests(o["ttft"], o["ttlt"], o["tbtmax"], o["counters"], o["pct"],
                               o["status"])
        ent = {"name": W.NAMES[cfg] + ("" if "-" not in key else ", " + key.split("-")[1] + " grid"),
               "n_inst": w.n_inst, "n_req": w.n_req, "rc": int(o["rc"]),
               "failed": int((o["status"] != 0).sum()),
               "inputs": input_digest(w), "reqiters": int(o["counters"][:, 1].sum()),
               "oracle_seconds": round(dt, 1), "threads": args.threads,
               "digests": "".join(dig)}
        if sel is not None:
            ent["instances"] = [int(i) for i in sel]
        res["workloads"][key] = ent
        print(f"{key}: {len(dig)} instances, {ent['reqiters']} request-iterations, "
              f"{dt:.0f} s", flush=True)
        del o
    with open(OUT, "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")


if __name__ == "__main__":
    main()
