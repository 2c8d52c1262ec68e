"""The fp64 oracle against its pins (closed forms, invariants, brute force,
torch.nn.LSTM in float64), plus argument checks.  CPU only."""
import numpy as np
import pytest

import oracle
import workloads
from tests import oracle_pins


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(oracle.forward)


def test_thread_count_does_not_change_bits():
    inp = workloads.random_case(5, 16, 12, 10, 9)
    x, W, U = inp.as_f32()
    a = oracle.forward(x, inp.lengths, W, U, inp.b, inp.h0, inp.c0, threads=1)
    b = oracle.forward(x, inp.lengths, W, U, inp.b, inp.h0, inp.c0, threads=4)
    assert all(np.array_equal(p, q) for p, q in zip(a, b))


def test_steps_equal_max_length():
    inp = workloads.random_case(6, 5, 3, 4, 10)
    x, W, U = inp.as_f32()
    _, _, steps = oracle.forward(x, inp.lengths, W, U, inp.b, inp.h0, inp.c0,
                                 return_steps=True)
    assert steps == int(inp.lengths.max())


@pytest.mark.parametrize("bad", [-1, 11])
def test_out_of_range_lengths_rejected(bad):
    inp = workloads.random_case(7, 3, 2, 2, 10)
    L = inp.lengths.copy()
    L[1] = bad
    x, W, U = inp.as_f32()
    with pytest.raises(oracle.OracleError):
        oracle.forward(x, L, W, U, inp.b, inp.h0, inp.c0)


def test_shape_mismatch_rejected():
    inp = workloads.random_case(8, 3, 2, 2, 4)
    x, W, U = inp.as_f32()
    with pytest.raises(oracle.OracleError):
        oracle.forward(x, inp.lengths, W.T.copy(), U, inp.b, inp.h0, inp.c0)


def test_bf16_inputs_are_exact_widenings():
    """The bf16 workloads hand the oracle the exact values the bf16 bits denote."""
    inp = workloads.make_inputs(3, 8, 4, 5, workloads.BF16, ("uniform", 1, 5), seed=9)
    x, W, U = inp.as_f32()
    assert np.array_equal(workloads.f32_to_bf16_bits(x), inp.x)
    assert np.all((x.view(np.uint32) & 0xFFFF) == 0)


def test_rows_subset_matches_full_batch():
    inp = workloads.random_case(10, 9, 6, 5, 8)
    h, c = oracle.forward_inputs(inp)
    rows = [7, 0, 4]
    hs, cs = oracle.forward_inputs(inp, rows=rows)
    assert np.array_equal(hs, h[rows]) and np.array_equal(cs, c[rows])


def test_golden_tiny_workload():
    """Generator + oracle reproduce the recorded tiny workload bit for bit."""
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "tiny_f32.json")) as f:
        rec = json.load(f)
    inp = workloads.workload_inputs("tiny_f32")
    assert inp.lengths.tolist() == rec["lengths"]
    h, c = oracle.forward_inputs(inp)
    want_h = np.array([[float.fromhex(v) for v in row] for row in rec["h"]])
    want_c = np.array([[float.fromhex(v) for v in row] for row in rec["c"]])
    assert np.array_equal(h, want_h) and np.array_equal(c, want_c)


@pytest.mark.parametrize("pin", oracle_pins.GRU_PINS, ids=lambda f: f.__name__)
def test_gru_pin(pin):
    pin(oracle.forward_gru)


@pytest.mark.parametrize("pin", oracle_pins.RNN_PINS, ids=lambda f: f.__name__)
def test_rnn_pin(pin):
    pin(oracle.forward_rnn)


@pytest.mark.parametrize("pin", oracle_pins.STOP_PINS, ids=lambda f: f.__name__)
def test_stop_pin(pin):
    pin(oracle.forward_stop)


@pytest.mark.parametrize("pin", oracle_pins.BWD_PINS, ids=lambda f: f.__name__)
def test_backward_pin(pin):
    pin(oracle.backward)


def _cell_bwd(cell, x, L, W, U, b, bhh, h0, dh, ds):
    if cell == "gru":
        return oracle.backward_gru(x, L, W, U, b, bhh, h0, dh, ds)
    return oracle.backward_rnn(x, L, W, U, b, h0, dh, ds)


@pytest.mark.parametrize("pin", oracle_pins.CELL_BWD_PINS, ids=lambda f: f.__name__)
def test_cell_backward_pin(pin):
    pin(_cell_bwd)


@pytest.mark.parametrize("cell", ["lstm", "gru", "rnn"])
def test_backward_thread_count_does_not_change_bits(cell):
    """The backward splits its products by k over threads; every entry is
    still summed by one thread in row, step and k order, so 1, 3 and 8
    threads give the same bits (blocks of rows of different sizes too)."""
    B, D, H, T = 11, 7, 9, 8
    inp = workloads.random_case(21, B, D, H, T, state_var=0.1) if cell == "lstm" else \
        workloads.random_cell_case(cell, 21, B, D, H, T)
    x, W, U = inp.as_f32()
    rng = np.random.default_rng(22)
    dh = rng.standard_normal((B, H))
    dc = rng.standard_normal((B, H))
    ds = rng.standard_normal((B, T, H))
    outs = []
    for th in (1, 3, 8):
        if cell == "lstm":
            outs.append(oracle.backward(x, inp.lengths, W, U, inp.b, inp.h0, inp.c0, dh, dc, ds,
                                        threads=th))
        elif cell == "gru":
            outs.append(oracle.backward_gru(x, inp.lengths, W, U, inp.b_ih, inp.b_hh, inp.h0, dh, ds,
                                            threads=th))
        else:
            outs.append(oracle.backward_rnn(x, inp.lengths, W, U, inp.b, inp.h0, dh, ds, threads=th))
    for o in outs[1:]:
        for k in outs[0]:
            assert np.array_equal(outs[0][k].view(np.uint64), o[k].view(np.uint64)), k
