"""Parity of the output sequence (lstm_dyn_forward_seq, through the C ABI)
with the fp64 oracle: out_seq[b, t] is the hidden state after step t for
t < L[b] and zero after.  Tolerances as for the final state: max-abs 1e-5
with fp32 x/W/U, 3e-3 with bf16."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests import oracle_cache
from tests.gpu_util import bits, max_err, say, to_device

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}
MODES = ["persistent", "per_step"]


def run_seq(inp, mode, model=None, dev=None):
    import torch
    m = model or ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode)
    dev = dev or to_device(inp)
    h, c, seq = m.forward_seq(*dev)
    torch.cuda.synchronize()
    return h, c, seq, m


def _check_padding_and_last(seq, h, lengths):
    """Zeros (+0.0) past each length, and the last valid step equal to out_h."""
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


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_seq_small_shapes(shape, mode):
    B, D, H, T, dt = shape
    inp = workloads.random_case(300 + B + D + H, B, D, H, T, dtype=dt)
    say(f"case seq {shape} {mode} lengths={inp.lengths.tolist()[:8]}")
    h, c, seq, m = run_seq(inp, mode)
    h, c, seq = h.cpu().numpy(), c.cpu().numpy(), seq.cpu().numpy()
    ho, co, so = oracle.forward_inputs(inp, seq=True)
    tol = TOL[dt]
    assert max_err(h, ho) <= tol and max_err(c, co) <= tol
    assert max_err(seq, so) <= tol, max_err(seq, so)
    _check_padding_and_last(seq, h, inp.lengths)
    # the plain forward gives the same state bit for bit
    import torch
    h2, c2 = m.forward(*to_device(inp))
    torch.cuda.synchronize()
    assert np.array_equal(bits(h2.cpu().numpy()), bits(h)) and np.array_equal(bits(c2.cpu().numpy()), bits(c))


# the largest workload's sequence (2 GB in fp32) is checked in its own test,
# both modes against one blocked pass of the oracle
BLOCKED = {"large2048_bf16"}


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", [n for n in workloads.ORDER if n not in BLOCKED])
def test_seq_workloads(name, mode):
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name)
    say(f"case seq workload {name} {mode}")
    h, c, seq, m = run_seq(inp, mode)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    seq, h, c = seq.cpu().numpy(), h.cpu().numpy(), c.cpu().numpy()
    ho, co, so = oracle.forward_inputs(inp, seq=True)
    _check_padding_and_last(seq, h, inp.lengths)
    es = max_err(seq, so)
    say(f"  max|dseq|={es:.3g} tol={w.tol}")
    assert es <= w.tol and max_err(h, ho) <= w.tol and max_err(c, co) <= w.tol
    m.close()


@pytest.mark.parametrize("name", sorted(BLOCKED))
def test_seq_largest_workload_every_row(name):
    """Every row and step of the output sequence, in both modes, against the
    oracle run on blocks of 32 rows (rows are independent)."""
    import torch
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name)
    got = {}
    for mode in MODES:
        say(f"case seq workload {name} {mode}")
        h, c, seq, m = run_seq(inp, mode)
        assert m.query(ld.Q_LAST_STATUS) == ld.OK
        got[mode] = (h.cpu().numpy(), c.cpu().numpy(), seq.cpu().numpy())
        m.close()
        del h, c, seq
        torch.cuda.empty_cache()
    for mode in MODES:
        _check_padding_and_last(got[mode][2], got[mode][0], inp.lengths)
    worst = {mode: [0.0, 0.0, 0.0] for mode in MODES}
    for rows, ho, co, so in oracle_cache.seq_blocks(inp):
        for mode in MODES:
            h, c, seq = got[mode]
            e = worst[mode]
            e[0] = max(e[0], max_err(seq[rows], so))
            e[1] = max(e[1], max_err(h[rows], ho))
            e[2] = max(e[2], max_err(c[rows], co))
    for mode in MODES:
        es, eh, ec = worst[mode]
        say(f"  {mode}: all {inp.B} rows max|dseq|={es:.3g} max|dh|={eh:.3g} max|dc|={ec:.3g} tol={w.tol}")
        assert es <= w.tol and eh <= w.tol and ec <= w.tol


@pytest.mark.parametrize("mode", MODES)
def test_seq_launches_and_poisoned_padding(mode):
    """One launch more than forward; NaN/Inf in x past each length reach
    neither the state nor the sequence (its padding stays +0.0)."""
    inp = workloads.random_case(31, 9, 20, 48, 14, dtype="bf16")
    h1, c1, s1, m = run_seq(inp, mode)
    n_seq = m.query(ld.Q_LAUNCHES_PER_FORWARD)
    import torch
    m.forward(*to_device(inp))
    torch.cuda.synchronize()
    assert n_seq == m.query(ld.Q_LAUNCHES_PER_FORWARD) + 1
    x = inp.x.copy()
    nan = workloads.f32_to_bf16_bits(np.array([np.nan], np.float32))[0]
    for r in range(inp.B):
        x[r, inp.lengths[r]:] = nan
    inp.x = x
    h2, c2, s2, _ = run_seq(inp, mode, model=m)
    assert torch.equal(h1, h2) and torch.equal(c1, c2) and torch.equal(s1, s2)
    _check_padding_and_last(s2.cpu().numpy(), h2.cpu().numpy(), inp.lengths)


def test_seq_single_workgroup_kernel():
    """H <= 32: the whole forward is one launch; the sequence adds one."""
    inp = workloads.random_case(32, 6, 12, 16, 10, dtype="f32")
    h, c, seq, m = run_seq(inp, "persistent")
    assert m.query(ld.Q_GROUPS) == 1 and m.query(ld.Q_LAUNCHES_PER_FORWARD) == 2
    ho, co, so = oracle.forward_inputs(inp, seq=True)
    assert max_err(seq.cpu().numpy(), so) <= 1e-5
