"""The C-ABI library on the host: it loads, exports every symbol that
include/tas.h declares, builds the same boost tables as the oracle, and rejects
invalid inputs before touching the GPU (no compute calls here)."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from paper_2606_18431_amd import tas
from paper_2606_18431_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "tas.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(tas_[a-z_]+)\s*\(", src)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    lib = tas.lib()
    names = declared_functions()
    assert len(names) == 19
    for n in names:
        assert hasattr(lib, n), n
    assert set(tas.EXPORTS) <= set(names)


def test_checking_build_exports_the_same_symbols():
    """libtas_check.so (every instance's state verified after each
    iteration) is a drop-in replacement: the same entry points."""
    assert os.path.exists(tas.CHECK_LIB_PATH), "libtas_check.so is missing: run the build"
    lib = ctypes.CDLL(tas.CHECK_LIB_PATH)
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_struct_layouts_match_header(tmp_path):
    """The ctypes mirrors have the C compiler's size and field offsets."""
    structs = [tas.tas_setting, tas.tas_params, tas.tas_traces]
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "tas.h"', 'int main(void) {']
    for st in structs:
        n = st.__name__
        lines.append(f'printf("{n} %zu\\n", sizeof({n}));')
        for f, _ in st._fields_:
            lines.append(f'printf("{n}.{f} %zu\\n", offsetof({n}, {f}));')
    lines.append('return 0; }')
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), "-o", str(exe),
                           str(src)])
    got = dict(l.split() for l in subprocess.check_output([str(exe)], text=True).splitlines())
    for st in structs:
        n = st.__name__
        assert int(got[n]) == ctypes.sizeof(st), n
        for f, _ in st._fields_:
            assert int(got[f"{n}.{f}"]) == getattr(st, f).offset, (n, f)
    assert ctypes.sizeof(tas.tas_setting) == W.SETTING_DTYPE.itemsize
    for f, _ in tas.tas_setting._fields_:
        assert W.SETTING_DTYPE.fields[f][1] == getattr(tas.tas_setting, f).offset, f


@pytest.mark.parametrize("k", [1, 7, 16, 256])
def test_boost_table_matches_oracle(k):
    """Both sides evaluate the gamma-Boost curve on the host in fp64; the tables
    (the only floating-point step of the path) agree bit for bit."""
    for g in np.concatenate([np.geomspace(1e-6, 2.0, 60), 10.0 ** np.linspace(-5, -1, 31)]):
        for tau in (5000.0, 1234.5):
            assert np.array_equal(tas.tas_boost_table(g, k, tau), oracle.boost_table(g, k, tau))


@pytest.mark.parametrize("k", [1, 16, 256])
def test_ada_grid_matches_oracle(k):
    """The adaptive-gamma grid, midpoints and tables agree bit for bit with the
    oracle's own construction."""
    for ada in (dict(W.ADA), dict(W.ADA, grid=2, gamma_min=2e-3, gamma_max=10.0),
                dict(W.ADA, grid=64, gamma_min=1e-6, gamma_max=3.0)):
        for tau in (5000.0, 777.25):
            s = W.setting(0, W.BOOST, k=k, gamma=ada["gamma_min"], ada=ada)
            g1, b1, t1 = tas.tas_ada_grid(s, tau)
            g2, b2, t2 = oracle.ada_grid(s, tau)
            assert np.array_equal(g1, g2) and np.array_equal(b1, b2) and np.array_equal(t1, t2)


def test_ada_settings_rejected():
    w = small()
    good = dict(W.ADA)
    bad = [dict(good, beta=1.5), dict(good, beta=-0.1), dict(good, window=0),
           dict(good, window=4096), dict(good, min_samples=300), dict(good, grid=1),
           dict(good, grid=65), dict(good, gamma_min=0.0), dict(good, gamma_max=1e-6),
           dict(good, eps_us=0.0), dict(good, eps_us=float("inf"))]
    for b in bad:
        s = w.settings.copy()
        s[2] = W.setting(int(s[2]["trace"]), W.BOOST, k=256, memguard=1, gamma=1e-3, ada=b)
        assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL, b
        with pytest.raises(tas.TasError):
            tas.tas_ada_grid(s[2])
    s = w.settings.copy()
    s[2] = W.setting(int(s[2]["trace"]), W.BOOST, gamma=0.5, ada=good)  # gamma0 > gamma_max
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL
    s = w.settings.copy()
    s[0]["ada"] = 1  # FCFS
    for f, v in good.items():
        s[0]["ada_" + f] = v
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL
    s = w.settings.copy()
    s[2] = W.setting(int(s[2]["trace"]), W.BOOST, gamma=1e-3, ada=good,
                     table=np.arange(24)[::-1])  # explicit table and adaptive gamma
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL
    s = w.settings.copy()
    s[2] = W.setting(int(s[2]["trace"]), W.BOOST, gamma=1e-3, ada=good)
    s[2]["ada"] = 2
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL


def test_ada_window_fits_lds():
    """The largest window still leaves room for the default list."""
    w = small()
    s = w.settings.copy()
    s[2] = W.setting(int(s[2]["trace"]), W.BOOST, gamma=1e-3, ada=dict(W.ADA, window=2048))
    t, _ = tas.make_traces(w.arrival_us, w.prompt, w.decode)
    p, _ = tas.make_params(w.engine, s)
    p0, _ = tas.make_params(w.engine, w.settings)
    extra = tas.tas_workspace_bytes(t, p) - tas.tas_workspace_bytes(t, p0)
    assert extra > 0  # the adaptive block, the gamma and switch outputs


def test_boost_table_rejects():
    for g, k, tau in [(0.0, 1, 5000.0), (-1.0, 1, 5000.0), (1e-3, 0, 5000.0), (1e-3, 1, 0.0),
                      (float("nan"), 1, 5000.0), (float("inf"), 1, 5000.0)]:
        with pytest.raises(tas.TasError):
            tas.tas_boost_table(g, k, tau)


def small():
    return W.make(1, n_traces=2, n_settings=6, n_req=50)


def create_rc(w, settings=None, engine=None, ws_bytes=None, cached=None, **kw):
    t, keep_t = tas.make_traces(w.arrival_us, w.prompt, w.decode, cached)
    p, keep_p = tas.make_params(engine or w.engine, w.settings if settings is None else settings,
                                **kw)
    need = tas.tas_workspace_bytes(t, p)
    ctx = ctypes.c_void_p()
    # a fake, aligned, non-null device address: every rejection below happens
    # before the first HIP call, so it is never dereferenced
    addr = 1 << 40
    rc = tas.lib().tas_create(ctypes.byref(t), ctypes.byref(p), addr,
                              need if ws_bytes is None else ws_bytes, ctypes.byref(ctx))
    assert not ctx.value
    return rc, need


def test_workspace_bytes_and_nomem():
    w = small()
    rc, need = create_rc(w, ws_bytes=1)
    assert need > 0 and rc == tas.TAS_ENOMEM


def test_rejects_invalid_traces():
    w = small()
    bad = small()
    bad.arrival_us[0, 5] = bad.arrival_us[0, 4] - 1  # unsorted
    assert create_rc(bad)[0] == tas.TAS_EINVAL
    bad = small()
    bad.prompt[1, 3] = 0
    assert create_rc(bad)[0] == tas.TAS_EINVAL
    bad = small()
    bad.decode[1, 3] = 0
    assert create_rc(bad)[0] == tas.TAS_EINVAL
    bad = small()
    bad.arrival_us[0, 0] = -1
    assert create_rc(bad)[0] == tas.TAS_EINVAL
    bad = small()
    bad.arrival_us[1, -1] = 1 << 41
    assert create_rc(bad)[0] == tas.TAS_EINVAL
    bad = small()
    bad.prompt[0, 0], bad.decode[0, 0] = 1 << 23, 1 << 23
    assert create_rc(bad)[0] == tas.TAS_EINVAL
    assert w.n_req > 0


def test_rejects_invalid_settings():
    w = small()
    cases = []
    s = w.settings.copy(); s[0]["trace"] = 5; cases.append(s)
    s = w.settings.copy(); s[0]["policy"] = 9; cases.append(s)           # unknown policy
    s = w.settings.copy(); s[0]["policy"] = 8; s[0]["memguard"] = 1; cases.append(s)  # Sarathi
    s = w.settings.copy(); s[0]["policy"] = -1; cases.append(s)
    s = w.settings.copy(); s[0]["policy"] = 5; s[0]["memguard"] = 1; cases.append(s)  # LAS + MemGuard
    s = w.settings.copy(); s[1]["policy"] = 6; s[1]["delta_us"] = 5; cases.append(s)  # TRAIL + delta
    s = w.settings.copy(); s[0]["memguard"] = 1; cases.append(s)          # FCFS with MemGuard
    s = w.settings.copy(); s[1]["delta_us"] = 10; cases.append(s)         # SRPT with delta
    s = w.settings.copy(); s[2]["k"] = 0; cases.append(s)
    s = w.settings.copy(); s[2]["delta_us"] = -1; cases.append(s)
    s = w.settings.copy(); s[2]["gamma"] = 0.0; cases.append(s)
    s = w.settings.copy(); s[2]["table_given"] = 1; s[2]["boost_us"][:] = np.arange(24); cases.append(s)
    s = w.settings.copy(); s[2]["table_given"] = 1; s[2]["boost_us"][:] = -1; cases.append(s)
    s = w.settings.copy(); s[2]["table_given"] = 1; s[2]["boost_us"][0] = (1 << 42) + 1; cases.append(s)
    for s in cases:
        assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL


def test_rejects_invalid_engine():
    w = small()
    for kw in (dict(max_seqs=0), dict(chunk=0), dict(chunk=10000, max_tokens=8192),
               dict(chunk=40000, max_tokens=65536),
               dict(kv_blocks=0), dict(block_tokens=0), dict(iter_base_us=0),
               dict(iter_ctx_div=0), dict(max_iters=0), dict(tau_us=0.0)):
        e = W.Engine(**{**W.Engine().__dict__, **kw})
        assert create_rc(w, engine=e)[0] == tas.TAS_EINVAL
        t, _ = tas.make_traces(w.arrival_us, w.prompt, w.decode)
        p, _ = tas.make_params(e, w.settings)
        assert tas.tas_workspace_bytes(t, p) == 0
    # candidate list too small for the batch cap, or beyond the LDS limit
    assert create_rc(w, list_cap=64)[0] == tas.TAS_EINVAL
    assert create_rc(w, list_cap=4033)[0] == tas.TAS_EINVAL
    assert create_rc(w, list_cap=1 << 16)[0] == tas.TAS_EINVAL


def test_rejects_infeasible_request():
    w = small()
    w.prompt[0, 0] = 4000
    w.decode[0, 0] = 4000
    e = W.Engine(kv_blocks=400)  # 7999 tokens need 500 blocks
    assert create_rc(w, engine=e)[0] == tas.TAS_EINFEASIBLE


def test_strerror_covers_codes():
    for code in range(-8, 1):
        assert tas.tas_strerror(code) != "unknown error"


def test_cache_signal_inputs():
    """Expected prefix-cache hits: accepted with 0 <= h < P, laid out in the
    workspace only when given, and required by (only) signal 2 of BOOST."""
    w = small()
    h = W.cached_tokens(0, w.prompt)
    s = w.settings.copy()
    s[2]["signal"] = 2
    t0, _ = tas.make_traces(w.arrival_us, w.prompt, w.decode)
    t1, _ = tas.make_traces(w.arrival_us, w.prompt, w.decode, h)
    p, _ = tas.make_params(w.engine, s)
    p0, _ = tas.make_params(w.engine, w.settings)
    assert tas.tas_workspace_bytes(t1, p0) - tas.tas_workspace_bytes(t0, p0) == \
        -(-(w.prompt.size * 4) // 256) * 256
    # valid inputs get as far as the size check of a 1-byte workspace
    assert create_rc(w, settings=s, cached=h, ws_bytes=1)[0] == tas.TAS_ENOMEM
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL  # signal 2 without hits
    assert create_rc(w, cached=h, ws_bytes=1)[0] == tas.TAS_ENOMEM  # hits, no signal 2
    for r, v in ((0, -1), (1, None)):
        bad = h.copy()
        bad[r, 3] = int(w.prompt[r, 3]) if v is None else v
        assert create_rc(w, settings=s, cached=bad)[0] == tas.TAS_EINVAL
    for pol, sig in ((W.FCFS, 2), (W.DIST, 2), (W.BOOST, 3)):
        s2 = w.settings.copy()
        s2[2] = W.setting(int(s2[2]["trace"]), pol, gamma=1e-3)
        s2[2]["signal"] = sig
        assert create_rc(w, settings=s2, cached=h)[0] == tas.TAS_EINVAL
    with pytest.raises(ValueError):
        tas.make_traces(w.arrival_us, w.prompt, w.decode, h[:1])


def test_jsq_replicas_validation():
    """Clusters behind the join-shortest-queue router: replica counts in
    [2, 16], all lists and adaptive windows within the LDS; workspace grows with
    the replicas (spill, lists and the router's arrays per replica)."""
    w = W.make_cluster(1, n_clusters=1, replicas=4, dispatch="jsq", n_req=30)
    t, _ = tas.make_traces(w.arrival_us, w.prompt, w.decode)
    sizes = []
    for r in (0, 2, 4, 16):
        p, _ = tas.make_params(w.engine, w.settings, jsq_replicas=r)
        sizes.append(tas.tas_workspace_bytes(t, p))
    assert sizes[0] > 0 and sizes[0] < sizes[1] < sizes[2] < sizes[3]
    for r in (-1, 17):
        p, _ = tas.make_params(w.engine, w.settings, jsq_replicas=r)
        assert tas.tas_workspace_bytes(t, p) == 0
    assert create_rc(w, ws_bytes=1, jsq_replicas=4)[0] == tas.TAS_ENOMEM  # valid so far
    s = w.settings.copy()
    s[1] = W.setting(0, W.BOOST, gamma=1e-3, ada=dict(W.ADA))  # gamma adapts per replica
    assert create_rc(w, settings=s, ws_bytes=1, jsq_replicas=4)[0] == tas.TAS_ENOMEM
    s[1] = W.setting(0, W.BOOST, gamma=1e-3, ada=dict(W.ADA, window=2048, min_samples=64))
    assert create_rc(w, settings=s, jsq_replicas=8)[0] == tas.TAS_EINVAL  # windows > LDS
    big = W.Engine(max_seqs=256, max_tokens=16384, kv_blocks=32768)
    assert create_rc(w, engine=big, jsq_replicas=16)[0] == tas.TAS_EINVAL  # 16 lists > LDS
    assert create_rc(w, engine=big, ws_bytes=1, jsq_replicas=8)[0] == tas.TAS_ENOMEM


def test_bench_refuses_more_than_one_gpu():
    """bench.py runs one GPU; asked for more it exits with a message before
    touching the GPU."""
    r = subprocess.run([os.environ.get("PYTHON", "python3"), os.path.join(ROOT, "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_ltr_control_validation():
    """SJF (LTR+) needs a starvation threshold and a quantum in [1, 32767]; the
    other policies must leave both at zero."""
    w = small()
    for bad in ((0, 4), (4, 0), (32768, 4), (4, 32768), (-1, 4)):
        s = w.settings.copy()
        s[0] = W.setting(int(s[0]["trace"]), W.LTR, ltr=bad)
        assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL, bad
    s = w.settings.copy()
    s[0]["ltr_starve"] = 8  # FCFS with an LTR field
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL
    s = w.settings.copy()
    s[0] = W.setting(int(s[0]["trace"]), W.LTR, ltr=(32767, 32767))
    assert create_rc(w, settings=s)[0] != tas.TAS_EINVAL  # valid (the copy needs a GPU)
    s[0]["policy"] = 10  # beyond the last policy
    assert create_rc(w, settings=s)[0] == tas.TAS_EINVAL
