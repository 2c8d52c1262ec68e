"""Randomised parity sweep where a step spans several chunks of row tiles:
129 to 512 rows of bf16 LSTM data on persistent handles, hidden widths 256
and 512 (the whole reverse loop in one launch; above 256 padded rows it keeps
the carried gradients in memory), ragged lengths, with and without the
output sequence's gradient.  The forward for training (final state and
output sequence) and every gradient against the fp64 oracle; the same for
the GRU and tanh RNN cells' gradients.  Also the forward at the widest
hidden layers (bf16 up to 2048, two gate tiles per workgroup above 1024;
fp32 up to 1024), both modes, every row and the output sequence against the
oracle."""
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


def _draw_wide(k):
    # the widest hidden layers each dtype takes (bf16 up to 8 units per CU,
    # fp32 up to 4), each width once; the rest drawn
    rng = np.random.default_rng(9600 + k)
    B = int(rng.integers(17, 301))
    D = int(rng.choice([16, 100]))
    dt = ("bf16", "f32")[k // 4]
    H = ((1024, 1100, 1536, 2048), (513, 777, 1000, 1024))[k // 4][k % 4]
    T = int(rng.integers(2, 13))
    mode = str(rng.choice(["persistent", "per_step"]))
    return B, D, H, T, dt, mode


@pytest.mark.parametrize("k", list(range(8)))
def test_random_wide_forward(k):
    import torch
    from tests.gpu_util import to_device
    import paper_1810_08061_amd as ld
    B, D, H, T, dt, mode = _draw_wide(k)
    say(f"case random wide {k}: B={B} D={D} H={H} T={T} {dt} {mode}")
    inp = workloads.random_case(9650 + k, B, D, H, T, dtype=dt)
    m = ld.LstmDyn(B, D, H, T, dt, mode)
    h, c, seq = m.forward_seq(*to_device(inp))
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    ho, co, so = oracle.forward_inputs(inp, seq=True)
    tol = 1e-5 if dt == "f32" else TOL
    eh, ec, es = max_err(h.cpu().numpy(), ho), max_err(c.cpu().numpy(), co), max_err(seq.cpu().numpy(), so)
    say(f"  max|dh|={eh:.2e} max|dc|={ec:.2e} max|dseq|={es:.2e}")
    assert eh <= tol and ec <= tol and es <= tol
    m.close()
