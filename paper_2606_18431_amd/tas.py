"""ctypes binding of the C ABI in include/tas.h (argument marshalling only).

Every step of the simulation runs in the HIP kernels of ``libtas.so``; this
module converts numpy / PyTorch arguments to the C structs and pointers. It
raises if the library is missing: there is no CPU fallback.

The functions keep the C names (``tas_create``, ``tas_run``, ...).
``Simulation`` bundles them for one workload, allocating the device workspace
and outputs as PyTorch tensors (PyTorch provides device memory and streams).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import workloads as W

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libtas.so")
# the checking build: the same entry points, and every instance's state is
# verified after each iteration (a violation fails it with TAS_ESTATE)
CHECK_LIB_PATH = os.path.join(PKG, "libtas_check.so")
LEVELS = 24

TAS_OK, TAS_EINVAL, TAS_EINFEASIBLE, TAS_ENOMEM, TAS_EHIP = 0, -1, -2, -3, -4
TAS_EOVERFLOW, TAS_ELIVELOCK, TAS_ESTATE, TAS_ECAPACITY = -5, -6, -7, -8
TAS_LTR = 9


class TasError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: {tas_strerror(code)} ({code})")
        self.code = code


class tas_traces(ctypes.Structure):
    _fields_ = [("n_traces", ctypes.c_int32), ("n_req", ctypes.c_int32),
                ("arrival_us", ctypes.c_void_p), ("prompt", ctypes.c_void_p),
                ("decode", ctypes.c_void_p), ("cached", ctypes.c_void_p)]


class tas_setting(ctypes.Structure):
    _fields_ = [("trace", ctypes.c_int32), ("policy", ctypes.c_int32), ("k", ctypes.c_int32),
                ("memguard", ctypes.c_int32), ("delta_us", ctypes.c_int64),
                ("gamma", ctypes.c_double), ("table_given", ctypes.c_int32),
                ("ada", ctypes.c_int32), ("boost_us", ctypes.c_int64 * LEVELS),
                ("ada_beta", ctypes.c_double), ("ada_gamma_min", ctypes.c_double),
                ("ada_gamma_max", ctypes.c_double), ("ada_eps_us", ctypes.c_double),
                ("ada_window", ctypes.c_int32), ("ada_min_samples", ctypes.c_int32),
                ("ada_grid", ctypes.c_int32), ("signal", ctypes.c_int32),
                ("ltr_starve", ctypes.c_int32), ("ltr_quantum", ctypes.c_int32)]


class tas_params(ctypes.Structure):
    _fields_ = [("max_seqs", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
                ("chunk", ctypes.c_int32), ("kv_blocks", ctypes.c_int32),
                ("block_tokens", ctypes.c_int32), ("iter_base_us", ctypes.c_int32),
                ("iter_tok_us", ctypes.c_int32), ("iter_ctx_div", ctypes.c_int32),
                ("max_iters", ctypes.c_int64), ("tau_us", ctypes.c_double),
                ("list_cap", ctypes.c_int32), ("spill_cap", ctypes.c_int32),
                ("n_inst", ctypes.c_int32), ("retry_cap", ctypes.c_int32),
                ("inst", ctypes.c_void_p), ("jsq_replicas", ctypes.c_int32)]


assert ctypes.sizeof(tas_setting) == W.SETTING_DTYPE.itemsize == 288

EXPORTS = ["tas_workspace_bytes", "tas_create", "tas_run", "tas_percentiles",
           "tas_percentiles_grouped", "tas_latencies",
           "tas_counters", "tas_gamma", "tas_status", "tas_instance_status", "tas_destroy",
           "tas_strerror", "tas_boost_table", "tas_ada_grid", "tas_instance_table",
           "tas_list_cap", "tas_replicas", "tas_schedule", "tas_create_static"]
STATIC_WORKSPACE_BYTES = 64 << 20

_lib = None


def lib():
    """Load libtas.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                              "or python -m paper_2606_18431_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        L.tas_workspace_bytes.argtypes = [P, P]
        L.tas_workspace_bytes.restype = ctypes.c_size_t
        L.tas_create.argtypes = [P, P, P, ctypes.c_size_t, ctypes.POINTER(P)]
        L.tas_create_static.argtypes = [P, P, ctypes.POINTER(P)]
        L.tas_create_static.restype = ctypes.c_int
        for name in ("tas_create", "tas_run", "tas_percentiles", "tas_percentiles_grouped",
                     "tas_latencies", "tas_counters",
                     "tas_gamma", "tas_status", "tas_instance_status", "tas_boost_table",
                     "tas_ada_grid", "tas_instance_table"):
            getattr(L, name).restype = ctypes.c_int
        L.tas_run.argtypes = [P, P]
        L.tas_percentiles.argtypes = [P, P, P]
        L.tas_percentiles_grouped.argtypes = [P, i32, P, P]
        L.tas_latencies.argtypes = [P, P, P, P, P]
        L.tas_counters.argtypes = [P, P, P]
        L.tas_gamma.argtypes = [P, P, P, P]
        L.tas_replicas.argtypes = [P, P, P, P, P, P]
        L.tas_schedule.argtypes = [P, P, P, P]
        L.tas_ada_grid.argtypes = [P, f64, P, P, P]
        L.tas_status.argtypes = [P]
        L.tas_instance_status.argtypes = [P, P, P]
        L.tas_destroy.argtypes = [P]
        L.tas_destroy.restype = None
        L.tas_strerror.argtypes = [ctypes.c_int]
        L.tas_strerror.restype = ctypes.c_char_p
        L.tas_boost_table.argtypes = [f64, i32, f64, P]
        L.tas_instance_table.argtypes = [P, i32, P]
        L.tas_list_cap.argtypes = [P]
        L.tas_list_cap.restype = i32
        _lib = L
    return _lib


def select_library(path: str) -> str:
    """Make the library at `path` the one that later calls load (LIB_PATH, or
    CHECK_LIB_PATH); returns the previous path. A context belongs to the
    library that created it: finish with it before switching back."""
    global LIB_PATH, _lib
    prev = LIB_PATH
    LIB_PATH, _lib = path, None
    return prev


def _ptr(x):
    """Device or host address of a torch tensor or numpy array (or None)."""
    if x is None:
        return None
    if isinstance(x, np.ndarray):
        assert x.flags["C_CONTIGUOUS"]
        return x.ctypes.data
    assert x.is_contiguous()
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        return None
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def tas_strerror(code: int) -> str:
    return lib().tas_strerror(int(code)).decode()


def _check(rc: int, what: str):
    if rc != TAS_OK:
        raise TasError(rc, what)


def make_traces(arrival_us: np.ndarray, prompt: np.ndarray, decode: np.ndarray,
                cached: np.ndarray | None = None):
    """tas_traces over host arrays [n_traces, n_req] (``cached``: expected
    prefix-cache hit tokens, or None); returns (struct, keepalive)."""
    a = np.ascontiguousarray(arrival_us, np.int64)
    p = np.ascontiguousarray(prompt, np.int32)
    d = np.ascontiguousarray(decode, np.int32)
    h = None if cached is None else np.ascontiguousarray(cached, np.int32)
    if a.ndim == 1:
        a, p, d = a[None], p[None], d[None]
        h = None if h is None else h[None]
    if h is not None and h.shape != p.shape:
        raise ValueError(f"cached has shape {h.shape}, prompts {p.shape}")
    t = tas_traces(a.shape[0], a.shape[1], a.ctypes.data, p.ctypes.data, d.ctypes.data,
                   None if h is None else h.ctypes.data)
    return t, (a, p, d, h)


def make_params(engine: W.Engine, settings: np.ndarray, list_cap: int = 0, spill_cap: int = 0,
                max_iters: int | None = None, retry_cap: int = 0, jsq_replicas: int = 0):
    """tas_params for an engine and a SETTING_DTYPE array; returns (struct, keepalive)."""
    s = np.ascontiguousarray(settings, W.SETTING_DTYPE)
    p = tas_params(engine.max_seqs, engine.max_tokens, engine.chunk, engine.kv_blocks,
                   engine.block_tokens, engine.iter_base_us, engine.iter_tok_us,
                   engine.iter_ctx_div, int(engine.max_iters if max_iters is None else max_iters),
                   float(engine.tau_us), int(list_cap), int(spill_cap), len(s), int(retry_cap),
                   s.ctypes.data if len(s) else None, int(jsq_replicas))
    return p, s


def jsq_replicas_of(w: W.Workload) -> int:
    """Replicas behind the join-shortest-queue router for a workload made by
    make_cluster(dispatch="jsq"), else 0."""
    return int(w.meta["replicas"]) if w.meta.get("dispatch") == "jsq" else 0


def tas_workspace_bytes(traces: tas_traces, params: tas_params) -> int:
    return int(lib().tas_workspace_bytes(ctypes.byref(traces), ctypes.byref(params)))


def tas_create(traces: tas_traces, params: tas_params, ws, ws_bytes: int | None = None):
    """Returns a context handle (int). ``ws`` is a device tensor (or address)."""
    ctx = ctypes.c_void_p()
    addr = ws if isinstance(ws, int) else _ptr(ws)
    nbytes = ws_bytes if ws_bytes is not None else ws.numel() * ws.element_size()
    rc = lib().tas_create(ctypes.byref(traces), ctypes.byref(params), addr, nbytes,
                          ctypes.byref(ctx))
    _check(rc, "tas_create")
    return ctx.value


def tas_create_static(traces: tas_traces, params: tas_params):
    """tas_create with the library's static device workspace (no device
    memory is allocated). Returns a context handle (int)."""
    ctx = ctypes.c_void_p()
    rc = lib().tas_create_static(ctypes.byref(traces), ctypes.byref(params), ctypes.byref(ctx))
    _check(rc, "tas_create_static")
    return ctx.value


def tas_run(ctx, stream=None):
    _check(lib().tas_run(ctx, _stream(stream)), "tas_run")


def tas_percentiles(ctx, out, stream=None):
    _check(lib().tas_percentiles(ctx, _ptr(out), _stream(stream)), "tas_percentiles")


def tas_percentiles_grouped(ctx, group: int, out, stream=None):
    _check(lib().tas_percentiles_grouped(ctx, int(group), _ptr(out), _stream(stream)),
           "tas_percentiles_grouped")


def tas_latencies(ctx, ttft=None, ttlt=None, tbtmax=None, stream=None):
    _check(lib().tas_latencies(ctx, _ptr(ttft), _ptr(ttlt), _ptr(tbtmax), _stream(stream)),
           "tas_latencies")


def tas_counters(ctx, out, stream=None):
    _check(lib().tas_counters(ctx, _ptr(out), _stream(stream)), "tas_counters")


def tas_gamma(ctx, gamma=None, switches=None, stream=None):
    _check(lib().tas_gamma(ctx, _ptr(gamma), _ptr(switches), _stream(stream)), "tas_gamma")


def tas_replicas(ctx, assign=None, counters=None, gamma=None, switches=None, stream=None):
    _check(lib().tas_replicas(ctx, _ptr(assign), _ptr(counters), _ptr(gamma), _ptr(switches),
                              _stream(stream)), "tas_replicas")


def tas_schedule(ctx, work=None, order=None, stream=None):
    _check(lib().tas_schedule(ctx, _ptr(work), _ptr(order), _stream(stream)), "tas_schedule")


def tas_ada_grid(setting, tau_us: float = 5000.0):
    """(grid [G], midpoints [G-1], tables [G, 24]) of an adaptive setting record."""
    rec = np.ascontiguousarray(np.asarray(setting, W.SETTING_DTYPE).reshape(1))
    G = int(rec[0]["ada_grid"])
    if not 2 <= G <= 64:
        raise TasError(TAS_EINVAL, "tas_ada_grid")
    grid, bound = np.zeros(G, np.float64), np.zeros(max(G - 1, 1), np.float64)
    tabs = np.zeros((G, LEVELS), np.int64)
    _check(lib().tas_ada_grid(rec.ctypes.data, float(tau_us), grid.ctypes.data,
                              bound.ctypes.data, tabs.ctypes.data), "tas_ada_grid")
    return grid, bound[:G - 1], tabs


def tas_instance_status(ctx, out, stream=None):
    _check(lib().tas_instance_status(ctx, _ptr(out), _stream(stream)), "tas_instance_status")


def tas_status(ctx) -> int:
    return int(lib().tas_status(ctx))


def tas_destroy(ctx):
    if ctx:
        lib().tas_destroy(ctx)


def tas_boost_table(gamma: float, k: int, tau_us: float = 5000.0) -> np.ndarray:
    out = np.zeros(LEVELS, np.int64)
    _check(lib().tas_boost_table(float(gamma), int(k), float(tau_us), out.ctypes.data),
           "tas_boost_table")
    return out


def tas_instance_table(ctx, inst: int) -> np.ndarray:
    out = np.zeros(LEVELS, np.int64)
    _check(lib().tas_instance_table(ctx, int(inst), out.ctypes.data), "tas_instance_table")
    return out


def tas_list_cap(ctx) -> int:
    return int(lib().tas_list_cap(ctx))


def _host(t, stream):
    """Copy a device tensor to a host numpy array once the work enqueued on
    `stream` has finished (the whole device is synchronised, so any stream,
    torch's or a raw handle, is covered)."""
    import torch

    torch.cuda.synchronize(t.device)
    return t.cpu().numpy()


class Simulation:
    """One workload on one GPU: workspace, outputs and the C-ABI calls."""

    def __init__(self, w: W.Workload, device="cuda", list_cap: int = 0, spill_cap: int = 0,
                 max_iters: int | None = None, retry_cap: int = 0):
        import torch

        self.w = w
        self.torch = torch
        self._tr, self._keep_t = make_traces(w.arrival_us, w.prompt, w.decode, w.cached)
        self.replicas = jsq_replicas_of(w)
        self._pa, self._keep_p = make_params(w.engine, w.settings, list_cap, spill_cap,
                                             max_iters, retry_cap, self.replicas)
        self.ws_bytes = tas_workspace_bytes(self._tr, self._pa)
        if self.ws_bytes == 0:
            raise TasError(TAS_EINVAL, "tas_workspace_bytes")
        self.ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        off = (-self.ws.data_ptr()) % 256
        self.ctx = tas_create(self._tr, self._pa, self.ws.data_ptr() + off, self.ws_bytes)
        n, m = w.n_inst, w.n_req
        self.pct = torch.zeros((n, 3, 3), dtype=torch.int32, device=device)
        self.counters = torch.zeros((n, 8), dtype=torch.int64, device=device)
        self.gamma_buf = torch.zeros(n, dtype=torch.float64, device=device)
        self.switch_buf = torch.zeros(n, dtype=torch.int64, device=device)
        self.status_buf = torch.zeros(n, dtype=torch.int32, device=device)
        self.m = m
        # the stream of the latest run: copies and status calls follow it
        # (every call on one context is ordered on one stream)
        self.stream = None

    def run(self, stream=None):
        self.stream = stream
        tas_run(self.ctx, stream)

    def percentiles(self, stream=None):
        self.stream = stream
        tas_percentiles(self.ctx, self.pct, stream)

    def step(self, stream=None):
        """One pass of the whole path: simulate every instance, then reduce."""
        self.run(stream)
        self.percentiles(stream)

    def results(self, latencies: bool = True):
        """Synchronise and copy everything to host numpy arrays (on the
        stream of the latest run)."""
        torch = self.torch
        n = self.w.n_inst
        st = self.stream
        out = {}
        if latencies:
            lat = [torch.empty((n, self.m), dtype=torch.int32, device=self.pct.device)
                   for _ in range(3)]
            tas_latencies(self.ctx, *lat, stream=st)
            for key, t in zip(("ttft", "ttlt", "tbtmax"), lat):
                out[key] = _host(t, st).view(np.uint32)
        tas_counters(self.ctx, self.counters, st)
        tas_gamma(self.ctx, self.gamma_buf, self.switch_buf, st)
        tas_instance_status(self.ctx, self.status_buf, st)
        out["rc"] = tas_status(self.ctx)
        out["counters"] = _host(self.counters, st)
        out["gamma"] = _host(self.gamma_buf, st)
        out["switches"] = _host(self.switch_buf, st)
        out["status"] = _host(self.status_buf, st)
        out["pct"] = _host(self.pct, st).view(np.uint32)
        if self.replicas > 1:  # the router's assignment and the replicas' counters
            asg = torch.empty((n, self.m), dtype=torch.int32, device=self.pct.device)
            rc = torch.empty((n, self.replicas, 8), dtype=torch.int64, device=self.pct.device)
            rg = torch.empty((n, self.replicas), dtype=torch.float64, device=self.pct.device)
            rs = torch.empty((n, self.replicas), dtype=torch.int64, device=self.pct.device)
            tas_replicas(self.ctx, asg, rc, rg, rs, stream=st)
            out["assign"] = _host(asg, st)
            out["rcounters"] = _host(rc, st)
            out["rgamma"] = _host(rg, st)
            out["rswitches"] = _host(rs, st)
        return out

    def group_percentiles(self, group: int, stream=None) -> np.ndarray:
        """Percentiles pooled over groups of `group` adjacent instances
        [n_inst/group, 3, 3] (synchronises)."""
        torch = self.torch
        st = self.stream if stream is None else stream
        out = torch.empty((self.w.n_inst // group, 3, 3), dtype=torch.int32,
                          device=self.pct.device)
        tas_percentiles_grouped(self.ctx, group, out, st)
        return _host(out, st).view(np.uint32)

    def table(self, inst: int) -> np.ndarray:
        return tas_instance_table(self.ctx, inst)

    def close(self):
        if getattr(self, "ctx", None):
            tas_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
