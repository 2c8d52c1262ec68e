"""Randomised parity sweep of the forward through the C ABI: seeded random
shapes (batch, input and hidden widths, time extent, including ragged sizes
that are multiples of no tile), dtypes, modes and cells, each against the
fp64 oracle at the plain loop's tolerances, with the output sequence."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import max_err, say, to_device
from tests.test_gpu_cells import gru_device

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}


def _draw(k):
    rng = np.random.default_rng(4000 + k)
    B = int(rng.choice([1, 2, 3, 7, 16, 17, 31, 64, 65, 130]))
    D = int(rng.choice([1, 3, 8, 15, 32, 33, 64, 100, 257]))
    H = int(rng.choice([1, 5, 16, 31, 32, 33, 48, 64, 100, 129, 256, 300, 513]))
    T = int(rng.integers(1, 24))
    dt = str(rng.choice(["f32", "bf16"]))
    mode = str(rng.choice(["persistent", "per_step"]))
    cell = str(rng.choice(["lstm", "gru", "rnn"]))
    return B, D, H, T, dt, mode, cell


CASES = list(range(240))


@pytest.mark.parametrize("k", CASES)
def test_random_forward(k):
    import torch
    B, D, H, T, dt, mode, cell = _draw(k)
    say(f"case random {k}: B={B} D={D} H={H} T={T} {dt} {mode} {cell}")
    if cell == "lstm":
        inp = workloads.random_case(5000 + k, B, D, H, T, dtype=dt)
        dev = to_device(inp)
    else:
        inp = workloads.random_cell_case(cell, 5000 + k, B, D, H, T, dtype=dt)
        dev = (*gru_device(inp), None)
    m = ld.LstmDyn(B, D, H, T, dt, mode, cell=cell)
    h, c, seq = m.forward_seq(*dev)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert m.query(ld.Q_STEPS_EXECUTED) == int(inp.lengths.max())
    h, c, seq = h.cpu().numpy(), c.cpu().numpy(), seq.cpu().numpy()
    if cell == "lstm":
        ho, co, so = oracle.forward_inputs(inp, seq=True)
        assert max_err(c, co) <= TOL[dt]
    elif cell == "gru":
        ho, so = oracle.forward_gru_inputs(inp, seq=True)
    else:
        ho, so = oracle.forward_rnn_inputs(inp, seq=True)
    eh, es = max_err(h, ho), max_err(seq, so)
    say(f"  max|dh|={eh:.2e} max|dseq|={es:.2e}")
    assert eh <= TOL[dt] and es <= TOL[dt]
    m.close()
