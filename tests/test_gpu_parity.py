"""Parity of the HIP path (called through the C ABI) with the fp64 oracle.

Tolerances are max-abs over every entry of h and of c: 1e-5 when x, W, U are
fp32 and 3e-3 when they are bf16 (products of bf16 operands accumulated in
fp32, the recurrent operand h rounded to fp16 each step).  Every row of every
workload is compared, the largest included."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests import oracle_cache
from tests.gpu_util import bits, max_err, run, say, to_device

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}
MODES = ["persistent", "per_step"]


def _oracle(inp, rows=None):
    return oracle.forward_inputs(inp, rows=rows)


# ---------------------------------------------------------------- small shapes
SHAPES = [
    # (B, D, H, T, dtype) -- ragged in every dimension, single- and multi-workgroup
    (1, 1, 1, 3, "f32"), (1, 1, 1, 3, "bf16"),
    (9, 5, 40, 1, "f32"), (9, 5, 40, 1, "bf16"),          # one step: lengths 0 or 1
    (5, 7, 13, 9, "f32"), (5, 7, 13, 9, "bf16"),
    (3, 16, 32, 6, "f32"), (17, 24, 32, 11, "bf16"),
    (37, 40, 33, 17, "f32"), (37, 40, 33, 17, "bf16"),   # H just above one workgroup
    (20, 64, 72, 12, "f32"), (33, 96, 100, 10, "bf16"),
    (70, 130, 136, 8, "bf16"), (16, 8, 260, 5, "f32"),
    # the widest variants: fp32 with 64 K-steps per wave, bf16 with two gate
    # tiles per workgroup (H > 1024) at both state capacities
    (8, 16, 700, 4, "f32"), (20, 40, 1100, 5, "bf16"), (272, 24, 1056, 4, "bf16"),
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_small_shapes(shape, mode):
    B, D, H, T, dt = shape
    inp = workloads.random_case(100 + B + D + H, B, D, H, T, dtype=dt)
    say(f"case small {shape} {mode} lengths={inp.lengths.tolist()[:8]}")
    h, c, _ = run(inp, mode)
    ho, co = _oracle(inp)
    tol = TOL[dt]
    assert max_err(h, ho) <= tol and max_err(c, co) <= tol, (max_err(h, ho), max_err(c, co))


# ------------------------------------------------------------ the workloads
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", workloads.ORDER)
def test_workload_parity(name, mode):
    """Every row of the workload against the oracle (its result is computed
    once per process and shared by both modes)."""
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name)
    say(f"case workload {name} {mode}")
    h, c, m = run(inp, mode)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert m.query(ld.Q_STEPS_EXECUTED) == int(inp.lengths.max())
    ho, co = oracle_cache.workload_state(name)
    eh, ec = max_err(h, ho), max_err(c, co)
    say(f"  all {inp.B} rows: max|dh|={eh:.3g} max|dc|={ec:.3g} tol={w.tol}")
    assert eh <= w.tol and ec <= w.tol
    assert np.all(np.abs(h) <= 1.0)
    m.close()


# ------------------------------------------------------------ semantics
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mode", MODES)
def test_length_zero_rows_are_untouched(dt, mode):
    inp = workloads.random_case(5, 9, 12, 40, 7, dtype=dt)
    inp.lengths[[0, 3, 8]] = 0
    h, c, _ = run(inp, mode)
    for r in (0, 3, 8):
        assert np.array_equal(bits(h[r]), bits(inp.h0[r].astype(np.float64)))
        assert np.array_equal(bits(c[r]), bits(inp.c0[r].astype(np.float64)))


@pytest.mark.parametrize("mode", MODES)
def test_all_lengths_zero(mode):
    inp = workloads.random_case(6, 7, 10, 36, 5, dtype="bf16")
    inp.lengths[:] = 0
    h, c, m = run(inp, mode)
    assert np.array_equal(bits(h), bits(inp.h0.astype(np.float64)))
    assert np.array_equal(bits(c), bits(inp.c0.astype(np.float64)))
    assert m.query(ld.Q_STEPS_EXECUTED) == 0


@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("mode", MODES)
def test_poisoned_padding_changes_nothing(dt, mode):
    """x[b, t >= L[b]] and x[:, max_len:] are never read: NaN/Inf there leave
    every output bit unchanged (the select semantics of the paper's loop)."""
    inp = workloads.random_case(7, 21, 18, 70, 12, dtype=dt, hi=9)
    h1, c1, m = run(inp, mode)
    x = inp.x.copy()
    nan = workloads.f32_to_bf16_bits(np.array([np.nan], np.float32))[0] if dt == "bf16" else np.nan
    inf = workloads.f32_to_bf16_bits(np.array([np.inf], np.float32))[0] if dt == "bf16" else np.inf
    for r in range(inp.B):
        x[r, inp.lengths[r]:] = nan
        if inp.lengths[r] + 1 < inp.T:
            x[r, inp.lengths[r] + 1] = inf
    inp.x = x
    h2, c2, _ = run(inp, mode, model=m)
    assert np.array_equal(bits(h1), bits(h2)) and np.array_equal(bits(c1), bits(c2))


@pytest.mark.parametrize("mode", MODES)
def test_repeat_runs_are_bitwise_identical(mode):
    inp = workloads.random_case(8, 48, 64, 130, 25, dtype="bf16")
    import torch
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, "bf16", mode)
    dev = to_device(inp)
    ref = None
    for _ in range(5):
        h, c, _ = run(inp, mode, model=m, dev=dev)
        if ref is None:
            ref = (bits(h), bits(c))
        else:
            assert np.array_equal(ref[0], bits(h)) and np.array_equal(ref[1], bits(c))
    torch.cuda.synchronize()


@pytest.mark.parametrize("mode", MODES)
def test_permutation_equivariance(mode):
    inp = workloads.random_case(9, 30, 20, 96, 14, dtype="bf16")
    h, c, m = run(inp, mode)
    p = np.random.default_rng(1).permutation(inp.B)
    inp2 = workloads.Inputs(x=inp.x[p].copy(), lengths=inp.lengths[p].copy(), W=inp.W, U=inp.U,
                            b=inp.b, h0=inp.h0[p].copy(), c0=inp.c0[p].copy(), dtype=inp.dtype)
    h2, c2, _ = run(inp2, mode, model=m)
    assert np.array_equal(bits(h2), bits(h[p])) and np.array_equal(bits(c2), bits(c[p]))


@pytest.mark.parametrize("mode", MODES)
def test_out_of_range_lengths_are_clamped_and_flagged(mode):
    inp = workloads.random_case(10, 6, 8, 40, 9, dtype="f32")
    bad = inp.lengths.copy()
    bad[1], bad[4] = -3, 50
    good = bad.clip(0, inp.T).astype(np.int32)
    inp.lengths = good
    hg, cg, m = run(inp, mode)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    inp.lengths = bad
    hb, cb, _ = run(inp, mode, model=m)
    assert m.query(ld.Q_LAST_STATUS) == ld.ERR_BAD_LENGTHS
    assert np.array_equal(bits(hg), bits(hb)) and np.array_equal(bits(cg), bits(cb))


def test_launch_counts():
    inp = workloads.random_case(11, 12, 16, 64, 10, dtype="bf16")
    _, _, m = run(inp, "persistent")
    # prep, W transpose (bf16), input projection, loop
    assert m.query(ld.Q_LAUNCHES_PER_FORWARD) == 4
    small = workloads.random_case(11, 12, 16, 32, 10, dtype="bf16")
    _, _, ms = run(small, "persistent")
    assert ms.query(ld.Q_LAUNCHES_PER_FORWARD) == 1 and ms.query(ld.Q_GROUPS) == 1
    _, _, m2 = run(inp, "per_step")
    assert m2.query(ld.Q_LAUNCHES_PER_FORWARD) == 4 + 2 * int(inp.lengths.max())
    assert m.query(ld.Q_TOTAL_ROWS) == int(inp.lengths.sum())


@pytest.mark.parametrize("mode", MODES)
def test_in_place_state_update(mode):
    import torch
    inp = workloads.random_case(12, 10, 14, 48, 8, dtype="f32")
    x, L, W, U, b, h0, c0 = to_device(inp)
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, "f32", mode)
    ref_h, ref_c = m.forward(x, L, W, U, b, h0, c0)
    ref_h, ref_c = ref_h.clone(), ref_c.clone()
    m.forward(x, L, W, U, b, h0, c0, out_h=h0, out_c=c0)
    torch.cuda.synchronize()
    assert torch.equal(h0, ref_h) and torch.equal(c0, ref_c)


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_zero_weights_closed_form(dt):
    """W = U = 0, b = 0: c_L = 2**-L c0 exactly (every gate 1/2, g = 0)."""
    inp = workloads.random_case(13, 7, 9, 36, 11, dtype=dt)
    inp.W[:] = 0
    inp.U[:] = 0
    inp.b[:] = 0
    h, c, _ = run(inp, "persistent")
    want_c = np.ldexp(inp.c0.astype(np.float64), -inp.lengths[:, None])
    assert np.array_equal(bits(c), bits(want_c.astype(np.float32).astype(np.float64)))
    want_h = np.where(inp.lengths[:, None] > 0, 0.5 * np.tanh(want_c), inp.h0)
    assert max_err(h, want_h) <= 1e-6


def test_modes_agree():
    inp = workloads.random_case(14, 40, 48, 200, 30, dtype="bf16")
    h1, c1, _ = run(inp, "persistent")
    h2, c2, _ = run(inp, "per_step")
    assert max_err(h1, h2) <= 3e-3 and max_err(c1, c2) <= 3e-3


def test_many_forwards_on_one_handle():
    """The barrier's arrival values grow across forwards; results stay identical."""
    inp = workloads.random_case(15, 24, 32, 72, 20, dtype="bf16")
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, "bf16", "persistent")
    dev = to_device(inp)
    ref = None
    for _ in range(20):
        h, c, _ = run(inp, model=m, dev=dev)
        if ref is None:
            ref = (bits(h), bits(c))
        assert np.array_equal(ref[0], bits(h)) and np.array_equal(ref[1], bits(c))
    assert m.query(ld.Q_LAST_STATUS) == ld.OK


def test_side_stream():
    import torch
    inp = workloads.random_case(16, 12, 20, 80, 9, dtype="bf16")
    h_ref, c_ref, m = run(inp)
    dev = to_device(inp)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        h, c = m.forward(*dev, stream=s)
    s.synchronize()
    assert np.array_equal(bits(h.cpu().numpy().astype(np.float64)), bits(h_ref))
