"""The backward pass of the GRU and tanh RNN cells (lstm_dyn_forward_train +
lstm_dyn_backward on a handle from lstm_dyn_create_cell, through the C ABI)
against the fp64 oracle's ``backward_gru`` / ``backward_rnn``.

Same bar as the LSTM backward: the scaled max-abs error of every gradient,
max|g - g_oracle| / max|g_oracle|, within 1e-5 (fp32 data) or 3e-3 (bf16
data); zero dx on padding and dh0 = d_out_h on length-0 rows bit for bit.
The GRU's bias gradient is [6H]: d b_ih followed by d b_hh."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import say
from tests.test_gpu_bwd import GRAD_TOL, MODES, compare, scaled_err
from tests.test_gpu_cells import gru_device

pytestmark = pytest.mark.gpu

CELLS = ["gru", "rnn"]
KEYS = ("dx", "dW", "dU", "db", "dh0")


def upstream(seed, B, H, T, seq=True):
    rng = np.random.default_rng(seed)
    dh = rng.standard_normal((B, H)).astype(np.float32)
    ds = rng.standard_normal((B, T, H)).astype(np.float32) if seq else None
    return dh, ds


def run_train(inp, mode, dh, ds):
    import torch
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode, cell=inp.cell)
    dev = gru_device(inp)
    m.forward_train(*dev)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda() if a is not None else None
    g = m.backward(*dev, None, t(dh), None, t(ds))
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert "dc0" not in g
    return {k: v.cpu().numpy().astype(np.float64) for k, v in g.items()}, m


def oracle_grads(inp, dh, ds, rows=None):
    x, W, U = inp.as_f32()
    L, h0 = inp.lengths, inp.h0
    if rows is not None:
        x, L, h0, dh = x[rows], L[rows], h0[rows], dh[rows]
        ds = ds[rows] if ds is not None else None
    f64 = lambda a: a.astype(np.float64) if a is not None else None
    if inp.cell == "gru":
        go = oracle.backward_gru(x, L, W, U, inp.b_ih, inp.b_hh, h0, f64(dh), f64(ds))
        go["db"] = np.concatenate([go.pop("db_ih"), go.pop("db_hh")])
        return go
    return oracle.backward_rnn(x, L, W, U, inp.b, h0, f64(dh), f64(ds))


SHAPES = [
    (1, 1, 1, 3, "f32"), (5, 7, 13, 9, "bf16"), (3, 16, 32, 6, "f32"), (17, 24, 32, 11, "bf16"),
    (37, 40, 33, 17, "f32"), (37, 40, 33, 17, "bf16"), (33, 96, 100, 10, "bf16"),
    (16, 8, 260, 5, "f32"), (20, 40, 1100, 5, "bf16"), (272, 24, 1056, 4, "bf16"),
]


@pytest.mark.parametrize("seq", [True, False], ids=["dseq", "final-state"])
@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_cell_backward_small_shapes(shape, mode, cell, seq):
    B, D, H, T, dt = shape
    inp = workloads.random_cell_case(cell, 1500 + B + D + H, B, D, H, T, dtype=dt)
    dh, ds = upstream(2500 + H, B, H, T, seq)
    say(f"case bwd {cell} {shape} {mode} dseq={seq} lengths={inp.lengths.tolist()[:8]}")
    g, _ = run_train(inp, mode, dh, ds)
    compare(g, oracle_grads(inp, dh, ds), GRAD_TOL[dt], keys=KEYS)
    for r in range(B):                              # exact facts
        assert not np.any(g["dx"][r, inp.lengths[r]:]), r
        if inp.lengths[r] == 0:
            assert np.array_equal(g["dh0"][r], dh[r]), r


@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", ["tiny_f32", "lstm256_f32", "lstm512_bf16"])
def test_cell_backward_workloads(name, mode, cell):
    w = workloads.WORKLOADS[name]
    inp = workloads.cell_workload_inputs(cell, name)
    dh, ds = upstream(3500, w.B, w.H, w.T)
    say(f"case bwd {cell} workload {name} {mode}")
    g, _ = run_train(inp, mode, dh, ds)
    compare(g, oracle_grads(inp, dh, ds), GRAD_TOL[w.dtype], keys=KEYS)


@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", ["skewed1024_bf16", "large2048_bf16"])
def test_cell_backward_large_workloads(name, mode, cell):
    """Full-size workloads with the cell's weights: dx and dh0 of a few short
    rows against the oracle on those rows alone; the weight gradients as the
    sums over two halves of the batch, each on its own handle."""
    import torch
    w = workloads.WORKLOADS[name]
    inp = workloads.cell_workload_inputs(cell, name)
    dh, ds = upstream(3501, w.B, w.H, w.T)
    say(f"case bwd {cell} workload {name} {mode}")
    g, m = run_train(inp, mode, dh, ds)
    m.close()
    order = np.argsort(inp.lengths, kind="stable")
    rows = [int(r) for r in order[:3]] + [int(order[len(order) // 8])]
    say(f"  sampled rows {rows} lengths {inp.lengths[rows].tolist()}")
    go = oracle_grads(inp, dh, ds, rows)
    compare({k: g[k][rows] for k in ("dx", "dh0")}, go, GRAD_TOL[w.dtype], keys=("dx", "dh0"))
    half = w.B // 2
    acc = {k: 0.0 for k in ("dW", "dU", "db")}
    for part in (slice(0, half), slice(half, w.B)):
        sub = workloads.CellInputs(x=inp.x[part].copy(), lengths=inp.lengths[part].copy(), W=inp.W,
                                   U=inp.U, b=inp.b, h0=inp.h0[part].copy(), dtype=inp.dtype,
                                   cell=inp.cell)
        gp, mp = run_train(sub, mode, dh[part].copy(), ds[part].copy())
        for k in acc:
            acc[k] = acc[k] + gp[k]
        mp.close()
        torch.cuda.empty_cache()
    add_tol = 1e-5 if w.dtype == workloads.F32 else 1e-3   # as for the LSTM
    for k in acc:
        e = scaled_err(g[k], acc[k])
        say(f"  halves {k}: {e:.2e}")
        assert e <= add_tol, (k, e)


@pytest.mark.parametrize("cell", CELLS)
def test_cell_backward_zero_upstream(cell):
    """Zero upstream gradients give zero gradients everywhere."""
    inp = workloads.random_cell_case(cell, 1602, 9, 20, 48, 14, dtype="bf16")
    g, _ = run_train(inp, "persistent", np.zeros((9, 48), np.float32),
                     np.zeros((9, 14, 48), np.float32))
    for k in KEYS:
        assert np.all(g[k] == 0), k


@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
def test_cell_forward_train_outputs_equal_forward(mode, cell):
    """The forward for training of a GRU or RNN handle gives the plain
    forward's h bit for bit, and its output sequence (rebuilt from the kept
    states) the forward_seq one."""
    import torch
    inp = workloads.random_cell_case(cell, 1603, 37, 40, 100, 17, dtype="bf16")
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode, cell=inp.cell)
    dev = gru_device(inp)
    h1, _, s1 = m.forward_seq(*dev)
    h2, _, s2 = m.forward_train(*dev, with_seq=True)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert torch.equal(h1, h2) and torch.equal(s1, s2)


@pytest.mark.parametrize("cell", CELLS)
def test_cell_backward_one_launch_reverse_loop(cell):
    """The GRU and RNN backward with every step in the one-launch reverse loop
    (bf16 data, at most 16 rows, H even and above 64) against the oracle."""
    B, D, H, T = 9, 20, 96, 40
    inp = workloads.random_cell_case(cell, 1604, B, D, H, T, dtype="bf16", lo=20)
    dh, ds = upstream(2604, B, H, T)
    say(f"case bwd {cell} one-launch loop lengths={inp.lengths.tolist()}")
    g, m = run_train(inp, "persistent", dh, ds)
    assert m.query(ld.Q_LAUNCHES_PER_FORWARD) < 30
    compare(g, oracle_grads(inp, dh, ds), GRAD_TOL["bf16"], keys=KEYS)
