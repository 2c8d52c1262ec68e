"""Randomised parity sweep where a step spans several chunks of row tiles:
129 to 512 rows of bf16 LSTM data on persistent handles, hidden widths 256
and 512 (the whole reverse loop in one launch; above 256 padded rows it keeps
the carried gradients in memory), ragged lengths, with and without the
output sequence's gradient.  The forward for training (final state and
output sequence) and every gradient against the fp64 oracle; the same for
the GRU and tanh RNN cells' gradients."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import max_err, say
from tests.test_gpu_bwd import GRAD_TOL, compare, oracle_grads, run_train
from tests.test_gpu_bwd_cells import KEYS as CELL_KEYS
from tests.test_gpu_bwd_cells import oracle_grads as cell_oracle
from tests.test_gpu_bwd_cells import run_train as cell_run

pytestmark = pytest.mark.gpu

TOL = 3e-3  # the forward's bar with bf16 data


def _draw(k):
    rng = np.random.default_rng(9000 + k)
    B = int(rng.integers(129, 513))
    D = int(rng.choice([8, 24, 40, 64]))
    H = int(rng.choice([256, 512]))
    T = int(rng.integers(2, 25))
    seq = bool(rng.integers(0, 2))
    return B, D, H, T, seq


@pytest.mark.parametrize("k", list(range(12)))
def test_random_large_batch(k):
    B, D, H, T, seq = _draw(k)
    say(f"case random large {k}: B={B} D={D} H={H} T={T} dseq={seq}")
    inp = workloads.random_case(9100 + k, B, D, H, T, dtype="bf16")
    rng = np.random.default_rng(9200 + k)
    dh = rng.standard_normal((B, H)).astype(np.float32)
    dc = rng.standard_normal((B, H)).astype(np.float32)
    ds = rng.standard_normal((B, T, H)).astype(np.float32) if seq else None
    g, fw, m = run_train(inp, "persistent", dh, dc, ds, want_seq=True)
    ho, co, so = oracle.forward_inputs(inp, seq=True)
    eh, ec, es = max_err(fw[0], ho), max_err(fw[1], co), max_err(fw[2], so)
    say(f"  forward max|dh|={eh:.2e} max|dc|={ec:.2e} max|dseq|={es:.2e}")
    assert eh <= TOL and ec <= TOL and es <= TOL
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64),
                      ds.astype(np.float64) if ds is not None else None)
    compare(g, go, GRAD_TOL[workloads.BF16])
    m.close()


@pytest.mark.parametrize("k", list(range(8)))
def test_random_large_batch_cells(k):
    B, D, H, T, seq = _draw(100 + k)
    cell = "gru" if k % 2 == 0 else "rnn"
    say(f"case random large {cell} {k}: B={B} D={D} H={H} T={T} dseq={seq}")
    inp = workloads.random_cell_case(cell, 9300 + k, B, D, H, T, dtype="bf16")
    rng = np.random.default_rng(9400 + k)
    dh = rng.standard_normal((B, H)).astype(np.float32)
    ds = rng.standard_normal((B, T, H)).astype(np.float32) if seq else None
    g, m = cell_run(inp, "persistent", dh, ds)
    compare(g, cell_oracle(inp, dh, ds), GRAD_TOL[workloads.BF16], keys=CELL_KEYS)
    m.close()
