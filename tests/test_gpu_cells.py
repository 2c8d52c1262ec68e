"""Parity of the GRU and tanh RNN cells (lstm_dyn_create_cell, through the C
ABI) with the fp64 oracle's GRU and RNN: final h and the output sequence, both
execution modes, the small-case shapes and the five workload shapes with that
cell's weights.  Tolerances as for the LSTM: max-abs 1e-5 with fp32 x/W/U,
3e-3 with bf16."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import max_err, say

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}
MODES = ["persistent", "per_step"]
CELLS = ["gru", "rnn"]


def oracle_of(inp, rows=None, seq=False):
    f = oracle.forward_gru_inputs if inp.cell == "gru" else oracle.forward_rnn_inputs
    return f(inp, rows=rows, seq=seq)


def gru_device(inp, device="cuda"):
    import torch
    if inp.dtype == workloads.BF16:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    else:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    L = torch.from_numpy(np.ascontiguousarray(inp.lengths, dtype=np.int32)).to(device)
    return conv(inp.x), L, conv(inp.W), conv(inp.U), f32(inp.b), f32(inp.h0)


def gru_model(inp, mode):
    return ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode, cell=inp.cell)


def run_gru(inp, mode, model=None, seq=False):
    import torch
    m = model or gru_model(inp, mode)
    dev = gru_device(inp)
    out = m.forward_seq(*dev) if seq else m.forward(*dev)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    return (*out, m)


def _check_padding_and_last(seq, h, lengths):
    T = seq.shape[1]
    t = np.arange(T)[None, :, None]
    pad = t >= lengths[:, None, None]
    assert np.all(np.where(pad, seq.view(np.uint32), 0) == 0)
    for r in range(len(lengths)):
        if lengths[r] > 0:
            assert np.array_equal(seq[r, lengths[r] - 1].view(np.uint32), h[r].view(np.uint32)), r


SHAPES = [
    (1, 1, 1, 3, "f32"), (5, 7, 13, 9, "bf16"), (3, 16, 32, 6, "f32"), (17, 24, 32, 11, "bf16"),
    (37, 40, 33, 17, "f32"), (37, 40, 33, 17, "bf16"), (33, 96, 100, 10, "bf16"),
    (16, 8, 260, 5, "f32"), (20, 40, 1100, 5, "bf16"), (272, 24, 1056, 4, "bf16"),
]


@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_cell_small_shapes(shape, mode, cell):
    B, D, H, T, dt = shape
    inp = workloads.random_cell_case(cell, 500 + B + D + H, B, D, H, T, dtype=dt)
    say(f"case {cell} {shape} {mode} lengths={inp.lengths.tolist()[:8]}")
    h, c, seq, m = run_gru(inp, mode, seq=True)
    h, c, seq = h.cpu().numpy(), c.cpu().numpy(), seq.cpu().numpy()
    ho, so = oracle_of(inp, seq=True)
    tol = TOL[dt]
    eh, es = max_err(h, ho), max_err(seq, so)
    say(f"  max|dh|={eh:.3g} max|dseq|={es:.3g}")
    assert eh <= tol and es <= tol
    assert np.all(c.view(np.uint32) == 0)                  # no cell state: out_c = +0.0
    _check_padding_and_last(seq, h, inp.lengths)
    h2, c2, _ = run_gru(inp, mode, model=m)                # plain forward: same h, bit for bit
    assert np.array_equal(h2.cpu().numpy().view(np.uint32), h.view(np.uint32))


SAMPLED = {"large2048_bf16"}


@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", workloads.ORDER)
def test_cell_workloads(name, mode, cell):
    import torch
    w = workloads.WORKLOADS[name]
    inp = workloads.cell_workload_inputs(cell, name)
    say(f"case {cell} workload {name} {mode}")
    h, c, seq, m = run_gru(inp, mode, seq=True)
    assert m.query(ld.Q_STEPS_EXECUTED) == int(inp.lengths.max())
    if name in SAMPLED:
        L = inp.lengths
        order = np.argsort(-L, kind="stable")
        rows = sorted({int(order[0]), int(order[-1]), int(order[len(order) // 2]), 5, 100})
        idx = torch.tensor(rows, device=seq.device)
        seq_s = seq.index_select(0, idx).cpu().numpy()
        h_s = h.cpu().numpy()[rows]
        ho, so = oracle_of(inp, rows=rows, seq=True)
        _check_padding_and_last(seq_s, h_s, L[rows])
        t = torch.arange(inp.T, device=seq.device)[None, :, None]
        Ld = torch.from_numpy(L).to(seq.device)[:, None, None]
        assert int(torch.count_nonzero(torch.where(t >= Ld, seq, torch.zeros_like(seq)))) == 0
        seq, h = seq_s, h_s
    else:
        seq, h = seq.cpu().numpy(), h.cpu().numpy()
        ho, so = oracle_of(inp, seq=True)
        _check_padding_and_last(seq, h, inp.lengths)
    eh, es = max_err(h, ho), max_err(seq, so)
    say(f"  max|dh|={eh:.3g} max|dseq|={es:.3g} tol={w.tol}")
    assert eh <= w.tol and es <= w.tol
    assert int(torch.count_nonzero(c)) == 0
    m.close()


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_rnn_zero_weights_zeroes_state_exactly(mode, dt):
    """W = U = 0 and b = 0: h' = tanh(0) = +0.0 after every step; rows of
    length 0 keep h0 bit for bit; the sequence is zero everywhere."""
    inp = workloads.random_cell_case("rnn", 46, 7, 9, 40, 12, dtype=dt)
    inp.lengths[:] = [0, 1, 2, 5, 12, 7, 3]
    inp.W[:] = 0
    inp.U[:] = 0
    inp.b[:] = 0
    h, c, seq, m = run_gru(inp, mode, seq=True)
    want = np.where(inp.lengths[:, None] > 0, np.float32(0), inp.h0).astype(np.float32)
    assert np.array_equal(np.abs(h.cpu().numpy()), np.abs(want))
    assert np.array_equal(h.cpu().numpy()[0].view(np.uint32), inp.h0[0].view(np.uint32))
    assert int(seq.count_nonzero()) == 0


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_gru_zero_weights_halves_state_exactly(mode, dt):
    """W = U = 0 and zero biases: r = u = 1/2 and n = 0, so every step halves
    h; the kernels' sigmoid(0) and tanh(0) are exact, so h_L = 2**-L h0 bit
    for bit, and rows of length 0 keep h0."""
    inp = workloads.random_gru_case(41, 7, 9, 40, 12, dtype=dt)
    inp.lengths[:] = [0, 1, 2, 5, 12, 7, 3]
    inp.W[:] = 0
    inp.U[:] = 0
    inp.b[:] = 0
    h, c, seq, m = run_gru(inp, mode, seq=True)
    want = np.ldexp(inp.h0, -inp.lengths[:, None]).astype(np.float32)
    assert np.array_equal(h.cpu().numpy().view(np.uint32), want.view(np.uint32))
    s = seq.cpu().numpy()
    for r in range(inp.B):
        for t in range(int(inp.lengths[r])):
            assert np.array_equal(s[r, t], np.ldexp(inp.h0[r], -(t + 1)).astype(np.float32))


@pytest.mark.parametrize("cell", CELLS)
@pytest.mark.parametrize("mode", MODES)
def test_cell_launches_c0_and_poisoned_padding(mode, cell):
    """One pack launch more than the LSTM handle of the same sizes; c0 may be
    None or anything (ignored); NaN in x past each length reaches nothing."""
    import torch
    inp = workloads.random_cell_case(cell, 43, 9, 20, 48, 14, dtype="bf16")
    h1, c1, s1, m = run_gru(inp, mode, seq=True)
    n_gru = m.query(ld.Q_LAUNCHES_PER_FORWARD)
    lstm = workloads.random_case(43, 9, 20, 48, 14, dtype="bf16")
    ml = ld.LstmDyn(lstm.B, lstm.D, lstm.H, lstm.T, lstm.dtype, mode)
    from tests.gpu_util import to_device
    ml.forward_seq(*to_device(lstm))
    torch.cuda.synchronize()
    assert n_gru == ml.query(ld.Q_LAUNCHES_PER_FORWARD) + 1
    ml.close()
    dev = gru_device(inp)
    junk = torch.full((inp.B, inp.H), float("nan"), device="cuda")
    h2, c2, s2 = m.forward_seq(*dev, junk)                 # a c0 full of NaN is ignored
    torch.cuda.synchronize()
    assert torch.equal(h1, h2) and torch.equal(s1, s2) and int(torch.count_nonzero(c2)) == 0
    x = inp.x.copy()
    nan = workloads.f32_to_bf16_bits(np.array([np.nan], np.float32))[0]
    for r in range(inp.B):
        x[r, inp.lengths[r]:] = nan
    inp.x = x
    h3, c3, s3, _ = run_gru(inp, mode, model=m, seq=True)
    assert torch.equal(h1, h3) and torch.equal(s1, s3)


@pytest.mark.parametrize("cell", CELLS)
def test_cell_single_workgroup_kernel(cell):
    """H <= 32: the whole forward is the pack launch plus one."""
    inp = workloads.random_cell_case(cell, 44, 6, 12, 16, 10, dtype="f32")
    h, c, m = run_gru(inp, "persistent")
    assert m.query(ld.Q_GROUPS) == 1 and m.query(ld.Q_LAUNCHES_PER_FORWARD) == 2
    ho = oracle_of(inp)
    assert max_err(h.cpu().numpy(), ho) <= 1e-5


def test_cell_handles_interleave():
    """GRU, RNN and LSTM handles on one stream do not disturb each other's
    results (separate workspaces)."""
    import torch
    from tests.gpu_util import to_device
    g = workloads.random_gru_case(45, 11, 30, 70, 9, dtype="bf16")
    r = workloads.random_cell_case("rnn", 45, 11, 30, 70, 9, dtype="bf16")
    mr = gru_model(r, "persistent")
    hr1, _ = mr.forward(*gru_device(r))
    l = workloads.random_case(45, 11, 30, 70, 9, dtype="bf16")
    mg, ml = gru_model(g, "persistent"), ld.LstmDyn(l.B, l.D, l.H, l.T, l.dtype, "persistent")
    dg, dl = gru_device(g), to_device(l)
    hg1, _ = mg.forward(*dg)
    hl1, cl1 = ml.forward(*dl)
    hg2, _ = mg.forward(*dg)
    torch.cuda.synchronize()
    assert torch.equal(hg1, hg2)
    assert max_err(hg1.cpu().numpy(), oracle.forward_gru_inputs(g)) <= 3e-3
    assert max_err(hr1.cpu().numpy(), oracle.forward_rnn_inputs(r)) <= 3e-3
    ho, co = oracle.forward_inputs(l)
    assert max_err(hl1.cpu().numpy(), ho) <= 3e-3 and max_err(cl1.cpu().numpy(), co) <= 3e-3


@pytest.mark.parametrize("mode", MODES)
def test_recurrent_operand_keeps_fp16_precision(mode):
    """With bf16 data the recurrent product takes h in fp16, not bf16: RNN with
    W = 0, b = 0, U = diag(1/2) and h0 = 1 + 2^-10 (exact in fp16; bf16 rounds
    it to 1) gives after one step tanh((1 + 2^-10) / 2); a bf16 operand would
    give tanh(1/2), 3.9e-4 away."""
    inp = workloads.random_cell_case("rnn", 47, 3, 8, 64, 4, dtype="bf16")
    inp.lengths[:] = 1
    inp.W[:] = 0
    inp.b[:] = 0
    inp.U[:] = 0
    half = workloads.f32_to_bf16_bits(np.array([0.5], np.float32))[0]
    inp.U[np.arange(64), np.arange(64)] = half
    inp.h0[:] = np.float32(1 + 2.0 ** -10)
    h, c, m = run_gru(inp, mode)
    want = np.tanh((1 + 2.0 ** -10) / 2)
    err = float(np.max(np.abs(h.cpu().numpy().astype(np.float64) - want)))
    say(f"  |h - tanh(v/2)| = {err:.3g}")
    assert err <= 2e-6
