"""Randomised parity sweep of the backward through the C ABI: seeded random
shapes (ragged batch, input and hidden widths, time extents), dtypes, modes
and cells, with and without the output sequence's gradient, each against the
fp64 oracle's gradients at the backward's bar (scaled max-abs error within
1e-5 with fp32 data, 3e-3 with bf16 data).  With bf16 data on persistent
handles, hidden widths that are even and at least 16 take the few-row launch
for their steps with at most 16 rows (cases 30 to 39), and hidden widths that
are multiples of 256 the whole reverse loop in one launch (cases 40 to 149)."""
import numpy as np
import pytest

import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import say
from tests.test_gpu_bwd import GRAD_TOL, compare
from tests.test_gpu_bwd import oracle_grads as lstm_oracle
from tests.test_gpu_bwd import run_train as lstm_run
from tests.test_gpu_bwd_cells import KEYS as CELL_KEYS
from tests.test_gpu_bwd_cells import oracle_grads as cell_oracle
from tests.test_gpu_bwd_cells import run_train as cell_run

pytestmark = pytest.mark.gpu


def _draw(k):
    rng = np.random.default_rng(6000 + k)
    B = int(rng.choice([1, 2, 5, 9, 16, 17, 33, 40]))
    D = int(rng.choice([1, 3, 8, 17, 32, 64, 80]))
    H = int(rng.choice([1, 7, 16, 18, 32, 33, 64, 66, 100, 128, 250, 300]))
    T = int(rng.integers(1, 21))
    dt = str(rng.choice(["f32", "bf16"]))
    mode = str(rng.choice(["persistent", "per_step"]))
    cell = str(rng.choice(["lstm", "gru", "rnn"]))
    seq = bool(rng.integers(0, 2))
    if 30 <= k < 40:  # cases for the few-row launch
        H = int(rng.choice([16, 18, 32, 64, 66, 100, 128, 250, 300]))
        dt, mode = "bf16", "persistent"
    if k >= 40:  # cases for the whole-loop launch
        H = int(rng.choice([256, 512]))
        dt, mode = "bf16", "persistent"
    return B, D, H, T, dt, mode, cell, seq


@pytest.mark.parametrize("k", list(range(150)))
def test_random_backward(k):
    B, D, H, T, dt, mode, cell, seq = _draw(k)
    say(f"case random bwd {k}: B={B} D={D} H={H} T={T} {dt} {mode} {cell} dseq={seq}")
    rng = np.random.default_rng(7000 + k)
    dh = rng.standard_normal((B, H)).astype(np.float32)
    ds = rng.standard_normal((B, T, H)).astype(np.float32) if seq else None
    if cell == "lstm":
        inp = workloads.random_case(8000 + k, B, D, H, T, dtype=dt)
        dc = rng.standard_normal((B, H)).astype(np.float32)
        g, _, _ = lstm_run(inp, mode, dh, dc, ds)
        go = lstm_oracle(inp, dh.astype(np.float64), dc.astype(np.float64),
                         ds.astype(np.float64) if ds is not None else None)
        compare(g, go, GRAD_TOL[dt])
    else:
        inp = workloads.random_cell_case(cell, 8000 + k, B, D, H, T, dtype=dt)
        g, _ = cell_run(inp, mode, dh, ds)
        compare(g, cell_oracle(inp, dh, ds), GRAD_TOL[dt], keys=CELL_KEYS)
    for r in range(B):
        assert not np.any(g["dx"][r, inp.lengths[r]:]), r
