"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle's C source is built a second time with -fsanitize=address,undefined
(every finding fatal) and driven, in a child Python process that preloads the
ASan runtime, over seeded workloads that reach every code path the tests use:
the five workloads' laws and every settings grid (comparators, adaptive gamma,
the phase ladder, the cache-aware signal), the schedule log, the
join-shortest-queue router, one-request traces and heavy KV pressure. The
child must exit cleanly with no sanitizer report, and its outputs must equal
the uninstrumented oracle's bit for bit.
"""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import workloads as W

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def scenarios():
    """(name, callable) pairs; each callable returns a dict of arrays."""
    out = []
    for cfg in (0, 1, 2, 3, 4):
        def run_cfg(cfg=cfg):
            w = W.make(cfg, n_traces=1, n_settings=8, n_req=250)
            return oracle.run(w, n_threads=2)
        out.append((f"sweep{cfg}", run_cfg))
    for grid in ("comparators", "ada", "ladder", "cache"):
        def run_grid(grid=grid):
            return oracle.run(W.make(2, n_traces=1, n_req=250, grid=grid), n_threads=2)
        out.append((grid, run_grid))

    def kv_pressure():  # a large trace under a small KV budget: many evictions
        w = W.make(2, n_traces=1, n_settings=4, n_req=1200)
        w.engine.kv_blocks = 1024
        return oracle.run(w, n_threads=2)
    out.append(("kv_pressure", kv_pressure))

    def ltr_control():  # SJF (LTR+) with promotions, demotions and evictions
        w = W.make(2, n_traces=1, n_settings=4, n_req=800)
        w.settings = np.stack([W.setting(0, W.LTR, ltr=(6, 3)), W.setting(0, W.LTR)])
        return oracle.run(w, n_threads=2)
    out.append(("ltr", ltr_control))

    def one_request():
        w = W.make(1, n_traces=1, n_settings=6, n_req=1)
        return oracle.run(w, n_threads=1)
    out.append(("one_request", one_request))

    def schedule_log():
        arr, p, d = W.small_random(7, 300)
        eng = W.Engine(max_seqs=8, max_tokens=512, chunk=128, kv_blocks=96)
        o = oracle.log(arr, p, d, eng, W.BOOST, k=16, memguard=1, delta_us=20000,
                       gamma=1e-3)
        return {k: v for k, v in o.items() if isinstance(v, np.ndarray)} | {"rc": o["rc"]}
    out.append(("log", schedule_log))

    def router():
        w = W.make_cluster(4, n_clusters=1, replicas=4, dispatch="jsq", n_req=500)
        return oracle.jsq(w, 4, n_threads=2)
    out.append(("jsq", router))
    return out


def run_all(dest=None):
    res = {}
    for name, fn in scenarios():
        o = fn()
        for k, v in o.items():
            res[f"{name}.{k}"] = np.asarray(v)
    if dest:
        np.savez(dest, **res)
    return res


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    d = tmp_path_factory.mktemp("san")
    lib = str(d / "libtas_oracle_san.so")
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c11", "-D_GNU_SOURCE", "-fPIC", "-shared",
                           "-ffp-contract=off", "-fsanitize=address,undefined",
                           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                           "-o", lib, oracle.SRC, "-lm", "-lpthread"])
    return asan, lib, d


def test_oracle_clean_under_asan_ubsan(sanitized_lib):
    asan, lib, d = sanitized_lib
    dest = str(d / "san_out.npz")
    code = (f"import sys; sys.path[:0] = [{ROOT!r}, {HERE!r}]; import oracle; "
            f"oracle.LIB = {lib!r}; oracle._lib = None; "
            f"import test_oracle_sanitize as t; t.run_all({dest!r}); print('child ok')")
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan + (":" + env["LD_PRELOAD"] if env.get("LD_PRELOAD") else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:verify_asan_link_order=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=900)
    report = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, report
    assert "child ok" in r.stdout, report
    for marker in ("runtime error", "AddressSanitizer", "UndefinedBehaviorSanitizer"):
        assert marker not in r.stderr, report
    got = np.load(dest)
    ref = run_all()
    assert sorted(got.files) == sorted(ref), (sorted(got.files), sorted(ref))
    for k in ref:
        assert np.array_equal(got[k], ref[k]), k
