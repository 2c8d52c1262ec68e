"""The backward pass (lstm_dyn_forward_train + lstm_dyn_backward, through the C
ABI) against the fp64 oracle's ``backward``.

Every gradient is compared by its scaled max-abs error,
max|g - g_oracle| / max|g_oracle|, against GRAD_TOL: the forward's tolerances
(1e-5 with fp32 data, 3e-3 with bf16 data, absolute on states of order 1)
taken relative to each gradient's scale.  The gradients flow through the
forward's own values (its pre-activations and states), so they inherit its
error; the backward itself runs in fp32.  Exact facts (zero gradient on
padding, length-0 rows, zero upstream gradient) are checked bit for bit."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests import oracle_cache
from tests.gpu_util import say, to_device

pytestmark = pytest.mark.gpu

GRAD_TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}
MODES = ["persistent", "per_step"]
KEYS = ("dx", "dW", "dU", "db", "dh0", "dc0")


def upstream(seed, B, H, T, seq=True):
    rng = np.random.default_rng(seed)
    dh = rng.standard_normal((B, H)).astype(np.float32)
    dc = rng.standard_normal((B, H)).astype(np.float32)
    ds = rng.standard_normal((B, T, H)).astype(np.float32) if seq else None
    return dh, dc, ds


def run_train(inp, mode, dh, dc, ds, model=None, want_seq=False):
    import torch
    m = model or ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode)
    dev = to_device(inp)
    fw = m.forward_train(*dev, with_seq=want_seq)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda() if a is not None else None
    g = m.backward(*dev, t(dh), t(dc), t(ds))
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    return {k: v.cpu().numpy().astype(np.float64) for k, v in g.items()}, [f.cpu().numpy() for f in fw], m


def oracle_grads(inp, dh, dc, ds, rows=None):
    x, W, U = inp.as_f32()
    L, h0, c0 = inp.lengths, inp.h0, inp.c0
    if rows is not None:
        x, L, h0, c0, dh, dc = x[rows], L[rows], h0[rows], c0[rows], dh[rows], dc[rows]
        ds = ds[rows] if ds is not None else None
    return oracle.backward(x, L, W, U, inp.b, h0, c0, dh, dc, ds)


def scaled_err(g, go):
    den = float(np.max(np.abs(go))) if go.size else 0.0
    return float(np.max(np.abs(g - go))) / den if den > 0 else float(np.max(np.abs(g))) if g.size else 0.0


def compare(g, go, tol, keys=KEYS):
    errs = {k: scaled_err(g[k], go[k]) for k in keys}
    say("  scaled errors " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k in keys:
        assert errs[k] <= tol, (k, errs[k], tol)


SHAPES = [
    (1, 1, 1, 3, "f32"), (5, 7, 13, 9, "bf16"), (3, 16, 32, 6, "f32"), (17, 24, 32, 11, "bf16"),
    (37, 40, 33, 17, "f32"), (37, 40, 33, 17, "bf16"), (33, 96, 100, 10, "bf16"),
    (16, 8, 260, 5, "f32"), (20, 40, 1100, 5, "bf16"), (272, 24, 1056, 4, "bf16"),
    (9, 5, 40, 1, "f32"), (9, 8, 256, 1, "bf16"),   # one step: lengths 0 or 1
]


@pytest.mark.parametrize("seq", [True, False], ids=["dseq", "final-state"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_backward_small_shapes(shape, mode, seq):
    B, D, H, T, dt = shape
    inp = workloads.random_case(1000 + B + D + H, B, D, H, T, dtype=dt)
    dh, dc, ds = upstream(2000 + H, B, H, T, seq)
    say(f"case bwd {shape} {mode} dseq={seq} lengths={inp.lengths.tolist()[:8]}")
    g, _, _ = run_train(inp, mode, dh, dc, ds)
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64),
                      ds.astype(np.float64) if ds is not None else None)
    compare(g, go, GRAD_TOL[dt])
    for r in range(B):                              # exact facts
        assert not np.any(g["dx"][r, inp.lengths[r]:]), r
        if inp.lengths[r] == 0:
            assert np.array_equal(g["dh0"][r], dh[r]) and np.array_equal(g["dc0"][r], dc[r]), r


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", ["tiny_f32", "lstm256_f32", "lstm512_bf16"])
def test_backward_workloads(name, mode):
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name)
    dh, dc, ds = upstream(3000, w.B, w.H, w.T)
    say(f"case bwd workload {name} {mode}")
    g, _, _ = run_train(inp, mode, dh, dc, ds)
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64), ds.astype(np.float64))
    compare(g, go, GRAD_TOL[w.dtype])


@pytest.mark.parametrize("mode", MODES)
def test_backward_skewed_workload_full_batch(mode):
    """skewed1024_bf16, the whole batch: every gradient (dx, dW, dU, db, dh0,
    dc0) against the oracle's (computed once, shared by both modes)."""
    name = "skewed1024_bf16"
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name)
    dh, dc, ds = upstream(3001, w.B, w.H, w.T)
    say(f"case bwd workload {name} {mode} (every row)")
    g, _, _ = run_train(inp, mode, dh, dc, ds)
    go = oracle_cache.grads((name, 3001), lambda: oracle_grads(
        inp, dh.astype(np.float64), dc.astype(np.float64), ds.astype(np.float64)))
    compare(g, go, GRAD_TOL[w.dtype])


@pytest.mark.parametrize("mode", MODES)
def test_backward_large_workload_sub_batch(mode):
    """large2048_bf16 at its full shape (D 1024, H 2048, T_max 1000) on 20 rows
    spread over its length range (the longest, 1000 steps, and the shortest
    included), run on their own handle: every gradient against the oracle.
    On the persistent handle the whole reverse loop is one launch (bf16 data,
    H a multiple of 256), with the carried gradients held in LDS."""
    import torch
    name = "large2048_bf16"
    full = workloads.workload_inputs(name)
    rows = oracle_cache.spanning_rows(full.lengths, 20)
    inp = workloads.Inputs(x=full.x[rows].copy(), lengths=full.lengths[rows].copy(), W=full.W,
                           U=full.U, b=full.b, h0=full.h0[rows].copy(), c0=full.c0[rows].copy(),
                           dtype=full.dtype)
    del full
    dh, dc, ds = upstream(3002, inp.B, inp.H, inp.T)
    say(f"case bwd {name} sub-batch {mode} lengths={sorted(inp.lengths.tolist(), reverse=True)}")
    g, _, m = run_train(inp, mode, dh, dc, ds)
    m.close()
    torch.cuda.empty_cache()
    go = oracle_cache.grads((name, "sub20", 3002), lambda: oracle_grads(
        inp, dh.astype(np.float64), dc.astype(np.float64), ds.astype(np.float64)))
    compare(g, go, GRAD_TOL[inp.dtype])


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("name", ["skewed1024_bf16", "large2048_bf16"])
def test_backward_large_workloads_halves(name, mode):
    """Full-size workloads on the whole batch (beside the oracle checks
    above): the per-row gradients (dx, dh0, dc0) of a few short rows against
    the oracle run on those rows alone (rows are independent); the weight
    gradients against the sums of the gradients of two halves of the batch,
    each run on its own handle."""
    import torch
    w = workloads.WORKLOADS[name]
    inp = workloads.workload_inputs(name)
    dh, dc, ds = upstream(3001, w.B, w.H, w.T)
    say(f"case bwd workload {name} {mode}")
    g, _, _ = run_train(inp, mode, dh, dc, ds)
    order = np.argsort(inp.lengths, kind="stable")
    rows = [int(r) for r in order[:3]] + [int(order[len(order) // 8])]
    say(f"  sampled rows {rows} lengths {inp.lengths[rows].tolist()}")
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64), ds.astype(np.float64), rows)
    gs = {k: g[k][rows] for k in ("dx", "dh0", "dc0")}
    compare(gs, go, GRAD_TOL[w.dtype], keys=("dx", "dh0", "dc0"))
    # weight gradients: the two halves add up to the whole
    half = w.B // 2
    acc = {k: 0.0 for k in ("dW", "dU", "db")}
    for part in (slice(0, half), slice(half, w.B)):
        sub = workloads.Inputs(x=inp.x[part].copy(), lengths=inp.lengths[part].copy(), W=inp.W, U=inp.U,
                               b=inp.b, h0=inp.h0[part].copy(), c0=inp.c0[part].copy(), dtype=inp.dtype)
        gp, _, m = run_train(sub, mode, dh[part].copy(), dc[part].copy(), ds[part].copy())
        for k in acc:
            acc[k] = acc[k] + gp[k]
        m.close()
        torch.cuda.empty_cache()
    # with bf16 data the weight-gradient GEMMs round dz, x and h_prev to fp16
    # under a scale set by each run's largest values, so the halves and the
    # whole round differently: relative 2^-11 per operand, well under 1e-3
    add_tol = 1e-5 if w.dtype == workloads.F32 else 1e-3
    for k in acc:
        e = scaled_err(g[k], acc[k])
        say(f"  halves {k}: {e:.2e}")
        assert e <= add_tol, (k, e)


@pytest.mark.parametrize("mode", MODES)
def test_forward_train_outputs_equal_forward(mode):
    """The forward for training gives the plain forward's state bit for bit,
    and its output sequence the forward_seq one."""
    import torch
    inp = workloads.random_case(1101, 37, 40, 100, 17, dtype="bf16")
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode)
    dev = to_device(inp)
    h1, c1, s1 = m.forward_seq(*dev)
    h2, c2, s2 = m.forward_train(*dev, with_seq=True)
    torch.cuda.synchronize()
    assert torch.equal(h1, h2) and torch.equal(c1, c2) and torch.equal(s1, s2)


@pytest.mark.parametrize("mode", MODES)
def test_backward_exact_facts(mode):
    """Zero upstream gradients give zero gradients everywhere; a backward needs
    a forward for training first, and consumes it."""
    import torch
    inp = workloads.random_case(1102, 9, 20, 48, 14, dtype="bf16")
    z = np.zeros((9, 48), np.float32)
    g, _, m = run_train(inp, mode, z, z, np.zeros((9, 14, 48), np.float32))
    assert all(not np.any(g[k][np.isfinite(g[k])]) and np.all(np.isfinite(g[k])) for k in KEYS)
    dev = to_device(inp)
    zt = torch.zeros((9, 48), device="cuda")
    with pytest.raises(ld.LstmDynError) as e:       # consumed
        m.backward(*dev, zt, zt)
    assert e.value.code == ld.ERR_INVALID
    m.forward(*dev)
    torch.cuda.synchronize()
    with pytest.raises(ld.LstmDynError):            # a plain forward keeps nothing
        m.backward(*dev, zt, zt)


@pytest.mark.parametrize("seq", [True, False], ids=["dseq", "final-state"])
def test_backward_one_launch_reverse_loop(seq):
    """bf16 data, at most 16 rows in every step, H even and above 64 but not
    a multiple of 256: the whole reverse loop is the launch for the steps
    with few rows (dh0 from the launch itself); against the oracle, and
    against the per-step path's launch count."""
    B, D, H, T = 9, 20, 96, 40
    inp = workloads.random_case(1201, B, D, H, T, dtype="bf16", lo=20)
    dh, dc, ds = upstream(2201, B, H, T, seq)
    say(f"case bwd one-launch loop seq={seq} lengths={inp.lengths.tolist()}")
    g, _, m = run_train(inp, "persistent", dh, dc, ds)
    launches = m.query(ld.Q_LAUNCHES_PER_FORWARD)
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64),
                      ds.astype(np.float64) if ds is not None else None)
    compare(g, go, GRAD_TOL["bf16"])
    _, _, mp = run_train(inp, "per_step", dh, dc, ds)
    per_step = mp.query(ld.Q_LAUNCHES_PER_FORWARD)
    say(f"  backward launches: {launches} (per-step path {per_step})")
    assert launches < 30 <= 2 * int(inp.lengths.max()) <= per_step


@pytest.mark.parametrize("seq", [True, False], ids=["dseq", "final-state"])
def test_backward_whole_loop_launch(seq):
    """bf16 data, H a multiple of 256: the whole reverse loop is one
    cooperative launch with column blocks of U, whatever the rows per step
    (up to 96 here); every gradient against the oracle, the launch count
    against the per-step path's, and a second run bit for bit equal to the
    first (the shares of dh and the waves' partial sums are added in a fixed
    order, whatever the order in which the data arrive)."""
    B, D, H, T = 96, 40, 256, 30
    inp = workloads.random_case(1211, B, D, H, T, dtype="bf16")
    dh, dc, ds = upstream(2211, B, H, T, seq)
    L = inp.lengths
    say(f"case bwd whole-loop launch seq={seq} rows per step "
        f"{[int((L > t).sum()) for t in range(0, T, 5)]}")
    g, _, m = run_train(inp, "persistent", dh, dc, ds)
    launches = m.query(ld.Q_LAUNCHES_PER_FORWARD)
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64),
                      ds.astype(np.float64) if ds is not None else None)
    compare(g, go, GRAD_TOL["bf16"])
    g2, _, _ = run_train(inp, "persistent", dh, dc, ds, model=m)
    for k in KEYS:
        assert np.array_equal(g[k], g2[k]), k
    _, _, mp = run_train(inp, "per_step", dh, dc, ds)
    per_step = mp.query(ld.Q_LAUNCHES_PER_FORWARD)
    say(f"  backward launches: {launches} (per-step path {per_step})")
    assert launches < 30 <= 2 * int(L.max()) <= per_step
    m.close()
    mp.close()


@pytest.mark.parametrize("scale", [1e-6, 1e6, 1e12])
@pytest.mark.parametrize("mode", MODES)
def test_backward_upstream_magnitude(scale, mode):
    """Gradients are linear in the upstream gradients: scaled by 1e-6 to 1e12
    they are scaled alike, and the fp16 operands of the bf16 path (powers of
    two per operand, per row and per row block) neither overflow nor lose
    the largest entries.  With H = 100 the persistent handle runs the steps
    with at most 16 rows in one launch and the others on the per-step path."""
    B, D, H, T = 33, 40, 100, 14
    inp = workloads.random_case(1401, B, D, H, T, dtype="bf16")
    dh, dc, ds = upstream(2401, B, H, T)
    dh, dc, ds = dh * np.float32(scale), dc * np.float32(scale), ds * np.float32(scale)
    say(f"case bwd upstream x{scale:g} {mode}")
    g, _, _ = run_train(inp, mode, dh, dc, ds)
    for k in g:
        assert np.all(np.isfinite(g[k])), k
    go = oracle_grads(inp, dh.astype(np.float64), dc.astype(np.float64), ds.astype(np.float64))
    compare(g, go, GRAD_TOL["bf16"])


@pytest.mark.parametrize("mode", MODES)
def test_backward_unaligned_dx(mode):
    """dx need only be 4-byte aligned: a dx 4 bytes past a 16-byte boundary
    (D a multiple of 4, so only the alignment sends its writer to the scalar
    path) receives the same bits as the default 16-byte aligned one, and so
    do the other gradients."""
    import torch
    B, D, H, T = 19, 8, 256, 9
    inp = workloads.random_case(3301, B, D, H, T, dtype="bf16")
    dh, dc, ds = upstream(3302, B, H, T)
    say(f"case bwd unaligned dx {mode}")
    m = ld.LstmDyn(B, D, H, T, inp.dtype, mode)
    dev = to_device(inp)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    m.forward_train(*dev)
    g = m.backward(*dev, t(dh), t(dc), t(ds))
    buf = torch.empty(B * T * D + 4, device="cuda")
    assert buf.data_ptr() % 16 == 0
    out = {k: torch.empty_like(v) for k, v in g.items()}
    out["dx"] = buf[1:1 + B * T * D].view(B, T, D)
    assert out["dx"].data_ptr() % 16 == 4
    m.forward_train(*dev)
    g2 = m.backward(*dev, t(dh), t(dc), t(ds), out=out)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    assert g2 is out
    for k in g:
        assert torch.equal(g[k], g2[k]), k
    m.close()

