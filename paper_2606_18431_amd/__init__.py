"""Tail-aware, prediction-free LLM scheduling (arXiv 2606.18431): the batched,
iteration-level serving simulation on MI355X (gfx950).

The simulation runs in hand-written HIP kernels behind a C ABI
(``include/tas.h``); ``paper_2606_18431_amd.tas`` is the ctypes binding and
``paper_2606_18431_amd.workloads`` draws the seeded synthetic inputs.
"""
