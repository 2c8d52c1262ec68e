"""Parity of the loop whose termination is computed from the state
(lstm_dyn_forward_stop, through the C ABI) with the fp64 oracle's
``forward_stop``: a row ends after a step that leaves v . h + c > 0; lengths
are caps; the loop leaves once no row runs.

The decision compares a floating-point score with zero, and the GPU forms it
from h in the precision of the recurrent operand, so a score within the error
bound of zero may go either way.  Each row's step count is therefore checked
against the oracle's score trace along the plain loop (the hidden state after
every step up to the cap, which does not depend on any decision): it must be
exactly the oracle's where every score up to it is clear of zero by the bound
delta = |v|_1 * tol, and otherwise a valid choice (no score before it above
+delta, the one after it, unless the cap ended the row, not below -delta).
The state is then compared with the trace at the GPU's step count; the cell
state and the output sequence with the oracle's stopping run where the count
is the oracle's.  Tolerances as for the plain loop."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests import oracle_cache
from tests.gpu_util import max_err, say, to_device
from tests.test_gpu_cells import gru_device

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}
MODES = ["persistent", "per_step"]


def _inputs(cell, inp):
    """(device args without c0, oracle args) for a batch of one cell."""
    x, W, U = inp.as_f32()
    if cell == "lstm":
        dev = to_device(inp)
        return dev[:6], dev[6], dict(x=x, W=W, U=U, b=inp.b, h0=inp.h0, c0=inp.c0, b_hh=None)
    c0 = np.zeros_like(inp.h0)
    b = inp.b_ih if cell == "gru" else inp.b
    return gru_device(inp), None, dict(x=x, W=W, U=U, b=b, h0=inp.h0, c0=c0,
                                        b_hh=inp.b_hh if cell == "gru" else None)


def _plain_trace(cell, o, L, rows):
    """Hidden state after every step up to each row's cap (plain loop, fp64)."""
    sel = (lambda a: a[rows]) if rows is not None else (lambda a: a)
    x, h0, c0 = sel(o["x"]), sel(o["h0"]), sel(o["c0"])
    if cell == "lstm":
        _, _, seq = oracle.forward(x, L, o["W"], o["U"], o["b"], h0, c0, return_seq=True)
    elif cell == "gru":
        _, seq = oracle.forward_gru(x, L, o["W"], o["U"], o["b"], o["b_hh"], h0, return_seq=True)
    else:
        _, seq = oracle.forward_rnn(x, L, o["W"], o["U"], o["b"], h0, return_seq=True)
    return seq


def check_against_oracle(cell, inp, v, c, h, cst, steps, seq, iters, tol, rows=None):
    """The checks described in the module docstring; returns the number of
    rows whose count was a near tie."""
    _, _, o = _inputs(cell, inp)
    Lc = np.clip(inp.lengths, 0, inp.T)
    L = Lc[rows] if rows is not None else Lc
    sel = (lambda a: a[rows]) if rows is not None else (lambda a: a)
    ho, co, so_steps, _, so = oracle.forward_stop(sel(o["x"]), L, o["W"], o["U"], o["b"],
                                                  sel(o["h0"]), sel(o["c0"]), v, c, cell=cell,
                                                  b_hh=o["b_hh"], return_seq=True)
    trace = _plain_trace(cell, o, L, rows)
    score = trace @ v.astype(np.float64) + c                       # [B, T]: after step k+1
    delta = float(np.abs(v).sum()) * tol
    hs, cs_, ss = sel(h), sel(cst), sel(steps)
    ties = 0
    for r in range(len(L)):
        n, no = int(ss[r]), int(so_steps[r])
        clear = np.all(np.abs(score[r, :max(n, no)]) > delta)
        if clear:
            assert n == no, (r, n, no)
        else:
            ties += 1
            assert 0 <= n <= L[r], (r, n)
            assert np.all(score[r, :n - 1] <= delta) if n > 1 else True, (r, n)
            if n < L[r]:
                assert n >= 1 and score[r, n - 1] >= -delta, (r, n)
        want_h = trace[r, n - 1] if n > 0 else sel(o["h0"])[r]
        assert max_err(hs[r], want_h) <= tol, (r, max_err(hs[r], want_h))
        if n == no:
            assert max_err(cs_[r], co[r]) <= tol, r
            if seq is not None:
                assert max_err(sel(seq)[r], so[r]) <= tol, r
        if seq is not None:
            assert not np.any(sel(seq)[r, n:]), r                    # zero from the last step on
    if rows is None:
        assert iters == int(steps.max() if len(steps) else 0)
    return ties


def run_stop(inp, cell, mode, v, c, seq=False, model=None):
    import torch
    m = model or ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode, cell=cell)
    dev, c0, _ = _inputs(cell, inp)
    vd = torch.from_numpy(np.ascontiguousarray(v, np.float32)).cuda()
    out = m.forward_stop(*dev, c0, vd, c, with_seq=seq)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    h, cs, steps = (t.cpu().numpy() for t in out[:3])
    sq = out[3].cpu().numpy() if seq else None
    return h, cs, steps, sq, m.query(ld.Q_STEPS_EXECUTED), m


def _readout(seed, H, c):
    v = np.random.default_rng(seed).standard_normal(H).astype(np.float32) / np.sqrt(H)
    return v, c


def _case(cell, seed, B, D, H, T, dt):
    if cell == "lstm":
        return workloads.random_case(seed, B, D, H, T, dtype=dt)
    return workloads.random_cell_case(cell, seed, B, D, H, T, dtype=dt)


SHAPES = [
    (1, 1, 1, 3, "f32"), (5, 7, 13, 9, "bf16"), (3, 16, 32, 6, "f32"), (17, 24, 32, 11, "bf16"),
    (37, 40, 33, 17, "f32"), (37, 40, 33, 17, "bf16"), (33, 96, 100, 10, "bf16"),
    (16, 8, 260, 5, "f32"), (20, 40, 1100, 5, "bf16"), (272, 24, 1056, 4, "bf16"),
]


@pytest.mark.parametrize("cell", ["lstm", "gru", "rnn"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_stop_small_shapes(shape, mode, cell):
    B, D, H, T, dt = shape
    inp = _case(cell, 700 + B + D + H, B, D, H, T, dt)
    v, c = _readout(800 + H, H, -0.1)
    say(f"case stop {cell} {shape} {mode} caps={inp.lengths.tolist()[:8]}")
    h, cs, steps, seq, iters, m = run_stop(inp, cell, mode, v, c, seq=True)
    ties = check_against_oracle(cell, inp, v, c, h, cs, steps, seq, iters, TOL[dt])
    say(f"  steps={steps.tolist()[:8]} iters={iters} near-ties={ties}")


@pytest.mark.parametrize("cell", ["lstm", "gru", "rnn"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", workloads.ORDER)
def test_stop_workloads(name, mode, cell):
    """The workload shapes; many rows end before their caps, others run to
    them (c chosen so).  large2048_bf16 on 16 rows spread over its lengths."""
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name) if cell == "lstm" else workloads.cell_workload_inputs(cell, name)
    v, c = _readout(900, w.H, -0.5)
    say(f"case stop workload {name} {cell} {mode}")
    h, cs, steps, seq, iters, m = run_stop(inp, cell, mode, v, c, seq=False)
    rows = None
    if name == "large2048_bf16":
        # 16 rows spread over the length range (the oracle's score trace of
        # every row would take 4 GB per cell and mode)
        rows = oracle_cache.spanning_rows(inp.lengths, 16)
    ties = check_against_oracle(cell, inp, v, c, h, cs, steps, None, iters, w.tol, rows=rows)
    early = int((steps < np.clip(inp.lengths, 0, inp.T)).sum())
    say(f"  rows ended early: {early}/{inp.B}, iters={iters} (cap {int(inp.lengths.max())}), near-ties={ties}")
    assert iters == int(steps.max())
    m.close()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_never_stopping_is_the_plain_loop(mode, dt):
    """v = 0 and c <= 0 (a zero score does not end a row): the state is the
    plain forward's bit for bit, every row runs to its cap, the loop runs
    max(L) steps."""
    import torch
    inp = workloads.random_case(81, 37, 40, 33, 17, dtype=dt)
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode)
    hp, cp = m.forward(*to_device(inp))
    torch.cuda.synchronize()
    for c in (-1.0, 0.0):
        h, cs, steps, _, iters, _ = run_stop(inp, "lstm", mode, np.zeros(33, np.float32), c, model=m)
        assert np.array_equal(h.view(np.uint32), hp.cpu().numpy().view(np.uint32))
        assert np.array_equal(cs.view(np.uint32), cp.cpu().numpy().view(np.uint32))
        assert np.array_equal(steps, inp.lengths) and iters == int(inp.lengths.max())


@pytest.mark.parametrize("mode", MODES)
def test_always_stopping_runs_one_step(mode):
    """v = 0, c > 0: every row ends after its first step: steps = min(L, 1),
    one loop step, and the state equals the plain forward with lengths
    min(L, 1) bit for bit."""
    import torch
    inp = workloads.random_case(82, 20, 24, 40, 9, dtype="bf16")
    inp.lengths[3] = 0
    h, cs, steps, _, iters, m = run_stop(inp, "lstm", mode, np.zeros(40, np.float32), 0.5)
    one = inp.lengths.copy()
    one[:] = np.minimum(one, 1)
    assert np.array_equal(steps, one) and iters == 1
    inp1 = workloads.random_case(82, 20, 24, 40, 9, dtype="bf16")
    inp1.lengths[:] = one
    hp, cp = m.forward(*to_device(inp1))
    torch.cuda.synchronize()
    assert np.array_equal(h.view(np.uint32), hp.cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("mode", MODES)
def test_all_caps_zero(mode):
    inp = workloads.random_case(83, 6, 8, 48, 5, dtype="f32")
    inp.lengths[:] = 0
    h, cs, steps, _, iters, _ = run_stop(inp, "lstm", mode, np.ones(48, np.float32), -1.0)
    assert iters == 0 and not steps.any()
    assert np.array_equal(h, inp.h0) and np.array_equal(cs, inp.c0)


@pytest.mark.parametrize("mode", MODES)
def test_early_exit_ends_the_loop(mode):
    """Caps of 200 steps but every row ends within a few: the loop stops at
    the last row's end, far below the cap."""
    inp = workloads.random_case(84, 64, 64, 128, 200, dtype="bf16", lo=200)
    v, c = _readout(85, 128, -0.2)
    v = np.abs(v)                                  # the fp64 oracle ends every row by step 55
    h, cs, steps, seq, iters, m = run_stop(inp, "lstm", mode, v, c, seq=True)
    check_against_oracle("lstm", inp, v, c, h, cs, steps, seq, iters, 3e-3)
    say(f"  iters={iters} steps max={int(steps.max())} min={int(steps.min())}")
    assert iters < 200


@pytest.mark.parametrize("mode", MODES)
def test_stop_poisoned_padding_and_repeat(mode):
    """NaN in x at or after each cap changes nothing; two forwards on one
    handle give the same bits."""
    inp = workloads.random_case(86, 9, 20, 48, 14, dtype="bf16")
    v, c = _readout(87, 48, 0.1)
    h1, c1, s1, q1, i1, m = run_stop(inp, "lstm", mode, v, c, seq=True)
    x = inp.x.copy()
    nan = workloads.f32_to_bf16_bits(np.array([np.nan], np.float32))[0]
    for r in range(inp.B):
        x[r, inp.lengths[r]:] = nan
    inp.x = x
    h2, c2, s2, q2, i2, _ = run_stop(inp, "lstm", mode, v, c, seq=True, model=m)
    assert np.array_equal(h1.view(np.uint32), h2.view(np.uint32))
    assert np.array_equal(c1.view(np.uint32), c2.view(np.uint32))
    assert np.array_equal(s1, s2) and i1 == i2
    assert np.array_equal(q1.view(np.uint32), q2.view(np.uint32))


def test_stop_and_plain_forwards_interleave():
    """A plain forward after a stopping one on the same handle is unaffected."""
    import torch
    inp = workloads.random_case(88, 33, 96, 100, 10, dtype="bf16")
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, "persistent")
    hp, cp = m.forward(*to_device(inp))
    torch.cuda.synchronize()
    hp = hp.cpu().numpy()
    v, c = _readout(89, 100, 0.1)
    run_stop(inp, "lstm", "persistent", v, c, model=m)
    h2, c2 = m.forward(*to_device(inp))
    torch.cuda.synchronize()
    assert np.array_equal(h2.cpu().numpy().view(np.uint32), hp.view(np.uint32))
    assert m.query(ld.Q_STEPS_EXECUTED) == int(inp.lengths.max())
