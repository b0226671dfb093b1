"""Per-instance digests of simulation outputs (test infrastructure).

A digest is the first 8 bytes of BLAKE2b over one instance's outputs in a
fixed byte order: TTFT, TTLT and maximum gap per request (uint32, little
endian), the eight counters (int64), the nine percentiles (uint32) and the
status (int32). An instance that failed (a nonzero status, such as a latency
past the 32-bit range) contributes its status alone. Equal digests mean equal outputs, element for element (up to
a 2^-64 collision chance). The stored digests are written by
``make_fullsize_digests.py`` from the CPU oracle alone; the GPU tests compute
the same digests from the HIP path's outputs and compare.
"""
from __future__ import annotations

import hashlib

import numpy as np

DIGEST_BYTES = 8


def instance_digests(ttft, ttlt, tbtmax, counters, pct, status) -> list[str]:
    """Hex digests, one per row (instance) of the output arrays."""
    ttft = np.ascontiguousarray(ttft, "<u4")
    ttlt = np.ascontiguousarray(ttlt, "<u4")
    tbtmax = np.ascontiguousarray(tbtmax, "<u4")
    counters = np.ascontiguousarray(counters, "<i8")
    pct = np.ascontiguousarray(np.asarray(pct).reshape(len(ttft), 9), "<u4")
    status = np.ascontiguousarray(status, "<i4")
    out = []
    for i in range(len(ttft)):
        h = hashlib.blake2b(digest_size=DIGEST_BYTES)
        if status[i] != 0:  # a failed instance: its status is its only defined output
            h.update(b"failed")
            h.update(status[i:i + 1].tobytes())
        else:
            for a in (ttft[i], ttlt[i], tbtmax[i], counters[i], pct[i], status[i:i + 1]):
                h.update(a.tobytes())
        out.append(h.hexdigest())
    return out


def input_digest(w, inst_ids=None) -> str:
    """Digest of a workload's traces, engine and the settings of the chosen
    instances (all by default): detects a drift of the input generator."""
    h = hashlib.blake2b(digest_size=16)
    for a in (w.arrival_us, w.prompt, w.decode):
        h.update(np.ascontiguousarray(a).tobytes())
    if w.cached is not None:
        h.update(np.ascontiguousarray(w.cached).tobytes())
    s = w.settings if inst_ids is None else w.settings[np.asarray(inst_ids)]
    for f in sorted(s.dtype.names):  # field by field: independent of the record layout
        h.update(f.encode())
        h.update(np.ascontiguousarray(s[f]).tobytes())
    e = w.engine
    h.update(repr((e.max_seqs, e.max_tokens, e.chunk, e.kv_blocks, e.block_tokens,
                   e.iter_base_us, e.iter_tok_us, e.iter_ctx_div, e.max_iters,
                   e.tau_us)).encode())
    return h.hexdigest()


def large_sweep_subset(w) -> np.ndarray:
    """The large sweep's checked instances: every 64th instance and every
    setting of four traces spread over the sweep (first, two inner, last)."""
    S = w.meta["n_settings"]
    T = w.n_traces
    pick = set(range(0, w.n_inst, 64))
    for t in (0, T // 3, (2 * T) // 3, T - 1):
        pick.update(range(t * S, (t + 1) * S))
    return np.array(sorted(pick), np.int64)
