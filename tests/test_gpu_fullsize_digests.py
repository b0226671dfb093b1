"""Every instance at full size: the chat-heavy (4096 x 10,000), reasoning-heavy
(4096 x 10,000) and bursty (4096 x 20,000) sweeps, the large sweep's checked
subset (every 64th instance and all settings of four traces, 508 of 16,384 x
50,000), every instance of the large-sweep traces under the comparator grid
(2,560, SJF (LTR+) among them), the adaptive-gamma, phase-ladder and
cache-aware grids (2,048 each), and every instance of the starvation mix
(256 x 20,000), each simulated in one tas_run in the launch configuration
the benchmark times, against the CPU oracle.

The oracle's outputs are stored as per-instance digests
(tests/golden/fullsize_digests.json, written by make_fullsize_digests.py from
the oracle alone): equal digests mean equal per-request TTFT, TTLT and maximum
gap, counters, percentiles and status. A mismatching instance is rerun on the
oracle here, which names the first differing element."""
import json
import os
import sys

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
from digests import input_digest, instance_digests, large_sweep_subset  # noqa: E402
from make_fullsize_digests import KEYS, make  # noqa: E402

pytestmark = pytest.mark.gpu
GOLD = json.load(open(os.path.join(HERE, "golden", "fullsize_digests.json")))["workloads"]


@pytest.fixture(scope="module")
def torch():
    import torch

    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def explain(w, i, got):
    """The first element where instance i differs from the oracle."""
    o = oracle.run(w.subset([i]))
    for key in ("ttft", "ttlt", "tbtmax"):
        bad = np.nonzero(got[key] != o[key][0])[0]
        if len(bad):
            j = bad[0]
            return f"{key}: {len(bad)} requests differ, first {j}: gpu {got[key][j]} oracle {o[key][0][j]}"
    for key in ("counters", "pct", "status"):
        if not np.array_equal(got[key], o[key][0]):
            return f"{key}: gpu {got[key]} oracle {o[key][0]}"
    return "no difference on rerun"


@pytest.mark.parametrize("key", KEYS)
def test_every_instance_matches_oracle_digest(torch, key):
    from paper_2606_18431_amd import tas

    if key not in GOLD:
        pytest.skip(f"no stored digests for {key} (make_fullsize_digests.py --only {key})")
    ref = GOLD[key]
    w = make(key)
    assert input_digest(w) == ref["inputs"], "the input generator drifted"
    sel = np.asarray(ref["instances"], np.int64) if "instances" in ref else np.arange(w.n_inst)
    if key == "4":
        assert np.array_equal(sel, large_sweep_subset(w))
    print(f"[gpu] full-size digests {ref['name']}: {w.n_inst} instances x {w.n_req}, "
          f"checking {len(sel)}", flush=True)
    sim = tas.Simulation(w)
    sim.step()
    g = sim.results(latencies=False)
    # (LAS overflows the 32-bit latency range on the comparator grid: those
    # instances are compared by their status)
    assert g["rc"] == ref.get("rc", 0), tas.tas_strerror(g["rc"])
    dev = sim.pct.device
    lat = [torch.empty((w.n_inst, w.n_req), dtype=torch.int32, device=dev) for _ in range(3)]
    tas.tas_latencies(sim.ctx, *lat)
    ix = torch.as_tensor(sel, device=dev)
    got = {k: t.index_select(0, ix).cpu().numpy().view(np.uint32)
           for k, t in zip(("ttft", "ttlt", "tbtmax"), lat)}
    del lat
    sim.close()
    torch.cuda.empty_cache()
    for k in ("counters", "pct", "status"):
        got[k] = g[k][sel]
    dig = instance_digests(got["ttft"], got["ttlt"], got["tbtmax"], got["counters"],
                           got["pct"], got["status"])
    want = ref["digests"]
    n = len(want) // 16
    assert n == len(sel)
    bad = [j for j in range(n) if dig[j] != want[16 * j:16 * (j + 1)]]
    if bad:
        j = bad[0]
        detail = explain(w, int(sel[j]), {k: v[j] for k, v in got.items()})
        raise AssertionError(f"{len(bad)} of {n} instances differ from the oracle; first: "
                             f"instance {int(sel[j])}: {detail}")
    if ref.get("failed", 0) == 0:  # (failed instances' counters are not compared)
        assert int(got["counters"][:, 1].sum()) == ref["reqiters"]
