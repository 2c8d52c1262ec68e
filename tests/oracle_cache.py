"""Oracle results of the full-size workloads, computed once per test process.

The fp64 oracle takes tens of seconds on the largest workload; the GPU tests of
both execution modes (and of the output sequence) compare against the same
result, so it is kept here for the process.  Values come from ``oracle`` only.
"""
from __future__ import annotations

import numpy as np

import oracle
import workloads

_STATE = {}
_GRADS = {}


def workload_state(name: str):
    """(h, c) of every row of workload ``name`` (float64 [B, H] each)."""
    if name not in _STATE:
        _STATE[name] = oracle.forward_inputs(workloads.workload_inputs(name))
    return _STATE[name]


def seq_blocks(inp, block: int = 32):
    """The oracle's output sequence in blocks of rows, so that the largest
    workload (8 GB of float64 for all rows at once) is never held whole:
    yields (rows, h, c, seq) with seq float64 [len(rows), T, H].  The final
    states it produces are kept for ``workload_state`` too."""
    for r0 in range(0, inp.B, block):
        rows = list(range(r0, min(inp.B, r0 + block)))
        h, c, seq = oracle.forward_inputs(inp, rows=rows, seq=True)
        yield rows, h, c, seq


def grads(key, fn):
    """Backward-oracle results under ``key``, computed by ``fn()`` once."""
    if key not in _GRADS:
        _GRADS[key] = fn()
    return _GRADS[key]


def spanning_rows(lengths: np.ndarray, n: int) -> list:
    """n rows spread over the length distribution: the longest, the shortest
    and evenly spaced ranks between them (descending length, stable)."""
    order = np.argsort(-lengths, kind="stable")
    picks = np.unique(np.round(np.linspace(0, len(order) - 1, n)).astype(int))
    return sorted(int(order[i]) for i in picks)
