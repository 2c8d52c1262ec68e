"""The largest batches the library takes, through the C ABI, against the fp64
oracle: 512 rows (the most the register-resident state of the persistent
variants holds: 8 owned row tiles per wave) on every persistent variant
family, and 8192 rows (the most the length preparation takes) on the
per-step path, which has no register-resident state.  Sampled rows are
checked against the oracle run on those rows alone (rows are independent);
every row of the persistent result against the per-step path's."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import max_err, run, say

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}


def _sample(inp, n=10, seed=11):
    L = inp.lengths
    order = np.argsort(-L, kind="stable")
    picks = {int(order[0]), int(order[-1]), int(order[len(order) // 2])}
    picks |= set(int(v) for v in np.random.default_rng(seed).choice(len(L), size=n, replace=False))
    return sorted(picks)


@pytest.mark.parametrize("shape", [
    (512, 40, 2048, 5, "bf16"),   # two gate tiles per workgroup, eight waves
    (512, 40, 1024, 6, "bf16"),   # one gate tile, four waves
    (512, 24, 256, 7, "f32"),
    (512, 16, 700, 4, "f32"),     # fp32 with 64 K-steps per wave
], ids=lambda s: "x".join(map(str, s)))
def test_largest_persistent_batch(shape):
    B, D, H, T, dt = shape
    inp = workloads.random_case(4000 + H, B, D, H, T, dtype=dt)
    say(f"case limit persistent {shape}")
    h, c, m = run(inp, "persistent")
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    rows = _sample(inp)
    ho, co = oracle.forward_inputs(inp, rows=rows)
    eh, ec = max_err(h[rows], ho), max_err(c[rows], co)
    say(f"  sampled rows: max|dh|={eh:.3g} max|dc|={ec:.3g}")
    assert eh <= TOL[dt] and ec <= TOL[dt]
    hs, cs, ms = run(inp, "per_step")
    e2 = max(max_err(h, hs), max_err(c, cs))
    say(f"  every row against the per-step path: {e2:.3g}")
    assert e2 <= 2 * TOL[dt]
    m.close()
    ms.close()


@pytest.mark.parametrize("mode", ["persistent", "per_step"])
def test_long_sequences(mode):
    """More than 2048 steps: the length preparation hands each wave its steps
    in batches of 64 (one offset per lane), so a bound past 2048 takes three
    batches.  Every row against the oracle; the valid-row count and the steps
    run against the lengths."""
    B, D, H, T = 40, 16, 64, 2600
    inp = workloads.random_case(4050, B, D, H, T, dtype="f32", lo=0, hi=T)
    say(f"case limit long sequences {(B, D, H, T)} {mode} max_len {int(inp.lengths.max())}")
    assert inp.lengths.max() > 2048
    h, c, m = run(inp, mode)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert m.query(ld.Q_TOTAL_ROWS) == int(inp.lengths.sum())
    assert m.query(ld.Q_STEPS_EXECUTED) == int(inp.lengths.max())
    ho, co = oracle.forward_inputs(inp)
    eh, ec = max_err(h, ho), max_err(c, co)
    say(f"  every row: max|dh|={eh:.3g} max|dc|={ec:.3g}")
    assert eh <= TOL["f32"] and ec <= TOL["f32"]
    m.close()


@pytest.mark.parametrize("B", [255, 256, 257, 300, 511, 512, 513, 1000, 1024, 1025, 3001])
def test_length_preparation_batch_sizes(B):
    """The length preparation counts each row's rank on 4, 2 or 1 lanes as B
    is at most 256, 512 or more, and keeps the batch rows of the first 256
    slots in registers (the rest come from LDS): a batch on each side of those
    bounds (the loop kernel up to 512 rows, the per-step path above), lengths
    0..9 with many ties, every row against the oracle and the valid-row
    count."""
    D, H, T = 8, 64, 9
    mode = "persistent" if B <= 512 else "per_step"
    inp = workloads.random_case(4500 + B, B, D, H, T, dtype="f32", lo=0, hi=T)
    say(f"case length preparation B={B} {mode}")
    h, c, m = run(inp, mode)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert m.query(ld.Q_TOTAL_ROWS) == int(inp.lengths.sum())
    ho, co = oracle.forward_inputs(inp)
    eh, ec = max_err(h, ho), max_err(c, co)
    say(f"  every row: max|dh|={eh:.3g} max|dc|={ec:.3g}")
    assert eh <= TOL["f32"] and ec <= TOL["f32"]
    m.close()


def test_one_row_more_needs_the_per_step_path():
    with pytest.raises(ld.LstmDynError) as e:
        ld.LstmDyn(513, 40, 1024, 6, "bf16", "persistent")
    assert e.value.code == ld.ERR_UNSUPPORTED


def test_largest_per_step_batch():
    B, D, H, T = 8192, 8, 32, 3
    inp = workloads.random_case(4100, B, D, H, T, dtype="f32")
    say(f"case limit per_step {(B, D, H, T)}")
    h, c, m = run(inp, "per_step")
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    rows = _sample(inp, n=30)
    ho, co = oracle.forward_inputs(inp, rows=rows)
    eh, ec = max_err(h[rows], ho), max_err(c[rows], co)
    say(f"  sampled rows: max|dh|={eh:.3g} max|dc|={ec:.3g}")
    assert eh <= TOL["f32"] and ec <= TOL["f32"]
    # rows of length 0 keep their initial state exactly
    z = np.flatnonzero(inp.lengths == 0)
    assert z.size > 0
    assert np.array_equal(h[z], inp.h0[z].astype(np.float64)) and np.array_equal(c[z], inp.c0[z].astype(np.float64))
    m.close()


@pytest.mark.parametrize("dt,H", [("bf16", 256), ("f32", 256), ("bf16", 2048)])
def test_largest_persistent_batch_backward(dt, H):
    """The backward at 512 rows, most of them short (steps 3 to 5 have at
    most 16 rows): with bf16 data and H a multiple of 256 the persistent
    handle runs the whole reverse loop in one launch with column blocks of U,
    at its largest batch, with the carried gradients in memory rather than
    LDS (more than 256 padded rows), at the smallest and the largest U block
    per wave (H = 256 and 2048); fewer launches than the per-step handle,
    which runs every step as two launches.  Per-row gradients of sampled rows
    against the oracle run on those rows alone; every gradient against the
    per-step handle's."""
    import torch
    from tests.test_gpu_bwd import GRAD_TOL, compare, oracle_grads, run_train, scaled_err
    B, D, T = 512, 24, 6
    inp = workloads.random_case(4200, B, D, H, T, dtype=dt)
    rng = np.random.default_rng(4201)
    L = rng.integers(1, 4, B).astype(np.int32)
    L[rng.choice(B, size=16, replace=False)[:12]] = 6
    L[np.flatnonzero(L < 4)[:4]] = 5
    inp.lengths = L
    active = [(L > t).sum() for t in range(T)]
    assert active[3] <= 16 and active[4] <= 16 and active[5] <= 16 and active[2] > 16
    dh = rng.standard_normal((B, H)).astype(np.float32)
    dc = rng.standard_normal((B, H)).astype(np.float32)
    ds = rng.standard_normal((B, T, H)).astype(np.float32)
    say(f"case limit backward {(B, D, H, T, dt)} rows per step {active}")
    g, _, m = run_train(inp, "persistent", dh, dc, ds)
    launches = m.query(ld.Q_LAUNCHES_PER_FORWARD)
    rows = _sample(inp) + [int(r) for r in np.flatnonzero(L == 6)[:2]]
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64), ds.astype(np.float64), rows)
    compare({k: g[k][rows] for k in ("dx", "dh0", "dc0")}, go, GRAD_TOL[dt], keys=("dx", "dh0", "dc0"))
    gs, _, ms = run_train(inp, "per_step", dh, dc, ds)
    per_step = ms.query(ld.Q_LAUNCHES_PER_FORWARD)
    say(f"  backward launches: persistent {launches}, per-step {per_step}")
    if dt == "bf16":
        assert launches < per_step
    for k in g:
        e = scaled_err(g[k], gs[k])
        say(f"  {k} against the per-step path: {e:.2e}")
        assert e <= 2 * GRAD_TOL[dt], (k, e)
    m.close()
    ms.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["persistent", "per_step"])
def test_largest_persistent_batch_sequence(mode):
    """The output sequence at 512 rows (the slot-to-row map of the persistent
    loop at its bound): sampled rows against the oracle, zeros past every
    row's length, the last valid step equal to the final h."""
    import torch
    from tests.test_gpu_seq import _check_padding_and_last, run_seq
    B, D, H, T = 512, 40, 2048, 5
    inp = workloads.random_case(4300, B, D, H, T, dtype="bf16")
    say(f"case limit sequence {(B, D, H, T)} {mode}")
    h, c, seq, m = run_seq(inp, mode)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    h, c, seq = h.cpu().numpy(), c.cpu().numpy(), seq.cpu().numpy()
    _check_padding_and_last(seq, h, inp.lengths)
    rows = _sample(inp)
    ho, co, so = oracle.forward_inputs(inp, rows=rows, seq=True)
    es, eh, ec = max_err(seq[rows], so), max_err(h[rows], ho), max_err(c[rows], co)
    say(f"  sampled rows: max|dseq|={es:.3g} max|dh|={eh:.3g} max|dc|={ec:.3g}")
    assert es <= TOL["bf16"] and eh <= TOL["bf16"] and ec <= TOL["bf16"]
    m.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("mode", ["persistent", "per_step"])
def test_largest_persistent_batch_stop_with_sequence(mode):
    """Termination from the state with the output sequence at 512 rows:
    sampled rows checked as in the stop tests (exact step counts away from
    near ties, state and sequence against the oracle)."""
    from tests.test_gpu_stop import _readout, check_against_oracle, run_stop
    B, D, H, T = 512, 40, 2048, 5
    inp = workloads.random_case(4400, B, D, H, T, dtype="bf16")
    v, c = _readout(4401, H, -0.1)
    say(f"case limit stop+sequence {(B, D, H, T)} {mode}")
    h, cs, steps, seq, iters, m = run_stop(inp, "lstm", mode, v, c, seq=True)
    rows = _sample(inp)
    ties = check_against_oracle("lstm", inp, v, c, h, cs, steps, seq, iters, TOL["bf16"], rows=rows)
    early = int((steps < inp.lengths).sum())
    say(f"  rows ended early: {early}/{B}, iters={iters}, near-ties={ties}")
    assert iters == int(steps.max())
    m.close()
