"""lstm_dyn_forward_noalloc (the allocation-free entry point, through the C
ABI) against lstm_dyn_forward on a handle with the same sizes: the same
kernels, so the same bits.  Two calls in a row, the second smaller (the
scratch keeps the first call's contents in another layout); the fp32 path, the
single-workgroup path (H <= 32), a clamped length reported through the
status word, and sizes past the scratch rejected before any work."""
import ctypes

import numpy as np
import pytest

import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import say, to_device

pytestmark = pytest.mark.gpu


def _noalloc(inp, dev, status=True):
    import torch
    x, L, W, U, b, h0, c0 = dev
    h = torch.empty((inp.B, inp.H), device="cuda")
    c = torch.empty((inp.B, inp.H), device="cuda")
    st = torch.full((1,), -1, dtype=torch.int32, device="cuda") if status else None
    dt = ld.BF16 if inp.dtype == workloads.BF16 else ld.F32
    ld.lstm_dyn_forward_noalloc(inp.B, inp.D, inp.H, inp.T, dt, x.data_ptr(), L.data_ptr(),
                                W.data_ptr(), U.data_ptr(), b.data_ptr(), h0.data_ptr(),
                                c0.data_ptr(), h.data_ptr(), c.data_ptr(),
                                st.data_ptr() if status else 0,
                                torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return h, c, (int(st.item()) if status else None)


def _handle(inp, dev):
    import torch
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, "persistent")
    h, c = m.forward(*dev)
    torch.cuda.synchronize()
    st = m.query(ld.Q_LAST_STATUS)
    m.close()
    return h, c, st


def _same(a, b):
    import torch
    return torch.equal(a.view(torch.int32), b.view(torch.int32))


CASES = [
    # (seed, B, D, H, T, dtype): each pair runs large then small
    ((6101, 37, 40, 100, 17, "bf16"), (6102, 9, 12, 40, 6, "bf16")),
    ((6103, 64, 512, 512, 200, "bf16"), (6104, 20, 64, 1100, 7, "bf16")),
    ((6105, 32, 256, 256, 100, "f32"), (6106, 5, 7, 13, 9, "f32")),
    ((6107, 6, 12, 16, 10, "f32"), (6108, 3, 5, 8, 4, "bf16")),   # one workgroup (H <= 32)
]


@pytest.mark.parametrize("pair", CASES, ids=lambda p: f"B{p[0][1]}H{p[0][3]}-B{p[1][1]}H{p[1][3]}")
def test_noalloc_matches_handle_forward_twice(pair):
    for spec in pair:
        seed, B, D, H, T, dt = spec
        inp = workloads.random_case(seed, B, D, H, T, dtype=dt)
        dev = to_device(inp)
        say(f"case noalloc {spec}")
        hn, cn, stn = _noalloc(inp, dev)
        hh, ch, sth = _handle(inp, dev)
        say(f"  status {stn} / {sth}, bitwise h {_same(hn, hh)} c {_same(cn, ch)}")
        assert stn == ld.OK and sth == ld.OK
        assert _same(hn, hh) and _same(cn, ch)


def test_noalloc_reports_clamped_lengths():
    inp = workloads.random_case(6201, 11, 16, 48, 9, dtype="bf16")
    inp.lengths[2] = 40
    dev = to_device(inp)
    h, c, st = _noalloc(inp, dev)
    assert st == ld.ERR_BAD_LENGTHS
    inp.lengths[2] = inp.T
    hg, cg, stg = _noalloc(inp, to_device(inp))
    assert stg == ld.OK and _same(h, hg) and _same(c, cg)


def test_noalloc_rejects_sizes_past_its_scratch():
    # the input projection of B * T steps alone needs 16 H B T bytes
    B, D, H, T = 64, 512, 512, 1000
    assert 16 * H * B * T > ld.NOALLOC_SCRATCH_BYTES
    import torch
    x = torch.zeros((B, T, D), dtype=torch.bfloat16, device="cuda")
    L = torch.zeros((B,), dtype=torch.int32, device="cuda")
    W = torch.zeros((D, 4 * H), dtype=torch.bfloat16, device="cuda")
    U = torch.zeros((H, 4 * H), dtype=torch.bfloat16, device="cuda")
    b = torch.zeros((4 * H,), device="cuda")
    s = torch.zeros((B, H), device="cuda")
    o = torch.zeros((B, H), device="cuda")
    oc = torch.zeros((B, H), device="cuda")
    with pytest.raises(ld.LstmDynError) as e:
        ld.lstm_dyn_forward_noalloc(B, D, H, T, ld.BF16, x.data_ptr(), L.data_ptr(), W.data_ptr(),
                                    U.data_ptr(), b.data_ptr(), s.data_ptr(), s.data_ptr(),
                                    o.data_ptr(), oc.data_ptr(), 0, 0)
    assert e.value.code == ld.ERR_TOO_LARGE
    assert "scratch" in ld.lstm_dyn_strerror(ld.ERR_TOO_LARGE)
