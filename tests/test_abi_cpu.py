"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/lstm_dyn.h declares, plans launches as intended and
rejects bad arguments before touching the device."""
import ctypes
import os
import re

import pytest

import paper_1810_08061_amd as ld

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    with open(os.path.join(ROOT, "include", "lstm_dyn.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(lstm_dyn_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert {"lstm_dyn_create", "lstm_dyn_forward", "lstm_dyn_destroy"} <= set(names)
    lib = ctypes.CDLL(ld.library_path())
    for n in names:
        assert hasattr(lib, n), n


def test_strerror_covers_codes():
    for code in range(8):
        assert ld.lstm_dyn_strerror(code) not in ("", "unknown status")
    assert ld.lstm_dyn_strerror(99) == "unknown status"


@pytest.mark.parametrize("B,D,H,T,dt,mt,groups,ksw,kw", [
    (4, 16, 32, 20, ld.F32, 1, 1, 4, 4),          # one workgroup, one launch
    (32, 256, 256, 100, ld.F32, 1, 64, 16, 4),
    (64, 512, 512, 200, ld.BF16, 1, 128, 4, 4),
    (128, 1024, 1024, 500, ld.BF16, 1, 256, 8, 4),
    (256, 1024, 2048, 1000, ld.BF16, 2, 256, 8, 8),
])
def test_plan_of_workloads(B, D, H, T, dt, mt, groups, ksw, kw):
    p = ld.lstm_dyn_plan(B, D, H, T, dt, ld.PERSISTENT, 256)
    assert (p["mt"], p["groups"], p["ksw"], p["kw"]) == (mt, groups, ksw, kw)
    assert p["groups"] <= 256 and (p["single"] or p["groups"] * 4 * p["mt"] >= H)
    kstep = 32 if dt == ld.BF16 else 4
    assert p["hpad"] == p["ksw"] * kstep * p["kw"] and p["hpad"] >= H
    assert p["bpad"] % 16 == 0 and p["bpad"] >= B
    assert p["nstate"] * p["kw"] >= ((B + 15) // 16) * p["mt"]
    assert p["lds_bytes"] <= 160 * 1024
    gx = 16 * H * B * T
    assert p["workspace_bytes"] >= gx
    assert p["single"] == (1 if H <= 32 else 0)
    if p["single"]:
        assert p["groups"] == 1 and p["single_nt"] * 16 >= B


@pytest.mark.parametrize("args", [
    (0, 1, 1, 1, 0, 0), (1, 0, 1, 1, 0, 0), (1, 1, 0, 1, 0, 0), (1, 1, 1, 0, 0, 0),
    (1, 1, 1, 1, 2, 0), (1, 1, 1, 1, 0, 2),
])
def test_plan_rejects_bad_sizes(args):
    with pytest.raises(ld.LstmDynError) as e:
        ld.lstm_dyn_plan(*args, 256)
    assert e.value.code == ld.ERR_INVALID


def test_plan_unsupported_sizes():
    with pytest.raises(ld.LstmDynError) as e:   # fp32 H=4096 needs more K-steps than any variant
        ld.lstm_dyn_plan(8, 8, 4096, 8, ld.F32, ld.PERSISTENT, 256)
    assert e.value.code == ld.ERR_UNSUPPORTED
    # the per-step path has no register-resident state limit
    ld.lstm_dyn_plan(8, 8, 1024, 8, ld.F32, ld.PER_STEP, 256)


def test_create_rejects_bad_sizes_without_device():
    with pytest.raises(ld.LstmDynError) as e:
        ld.lstm_dyn_create(0, 4, 4, 4, ld.F32, ld.PERSISTENT)
    assert e.value.code == ld.ERR_INVALID


def _ptrs(B, D, H, T, e):
    """Disjoint fake device addresses, 256-byte aligned (never dereferenced)."""
    sizes = [B * T * D * e, 4 * B, D * 4 * H * e, H * 4 * H * e, 16 * H, 4 * B * H, 4 * B * H,
             4 * B * H, 4 * B * H]
    out, at = [], 1 << 20
    for s in sizes:
        out.append(at)
        at += (s + 255) // 256 * 256 + 256
    return out


def test_check_args():
    B, D, H, T = 3, 5, 7, 4
    p = _ptrs(B, D, H, T, 4)
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *p) == ld.OK
    for i in range(9):                           # any NULL pointer
        q = list(p)
        q[i] = 0
        assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID
    for i in (0, 2, 3):                          # x, W, U need 16-byte alignment
        q = list(p)
        q[i] += 4
        assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID
    q = list(p)
    q[5] += 2                                    # h0 needs 4-byte alignment
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID
    # exact in-place state update is allowed
    q = list(p)
    q[7], q[8] = q[5], q[6]
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.OK
    # partial overlap of an output with an input is not
    q = list(p)
    q[7] = q[5] + 4
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID
    q = list(p)
    q[8] = q[0]                                  # out_c on top of x
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID
    q = list(p)
    q[8] = q[7]                                  # out_c == out_h
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID
    q = list(p)
    q[7] = q[6]                                  # out_h on c0
    assert ld.lstm_dyn_check_args(B, D, H, T, ld.F32, *q) == ld.ERR_INVALID


def test_check_seq_args():
    B, D, H, T = 3, 5, 7, 4
    p = _ptrs(B, D, H, T, 4)
    seq = p[-1] + (4 * B * H + 255) // 256 * 256 + 512       # after every other buffer
    assert ld.lstm_dyn_check_seq_args(B, D, H, T, ld.F32, *p, seq) == ld.OK
    assert ld.lstm_dyn_check_seq_args(B, D, H, T, ld.F32, *p, 0) == ld.ERR_INVALID
    assert ld.lstm_dyn_check_seq_args(B, D, H, T, ld.F32, *p, seq + 2) == ld.ERR_INVALID
    for i in range(9):                           # out_seq on top of any other argument
        assert ld.lstm_dyn_check_seq_args(B, D, H, T, ld.F32, *p, p[i]) == ld.ERR_INVALID
    q = list(p)
    q[0] = 0                                     # the plain checks still apply
    assert ld.lstm_dyn_check_seq_args(B, D, H, T, ld.F32, *q, seq) == ld.ERR_INVALID


def _gru_ptrs(B, D, H, T, e):
    """Disjoint fake addresses with the GRU's sizes (W, U with 3H columns, b 6H)."""
    sizes = [B * T * D * e, 4 * B, D * 3 * H * e, H * 3 * H * e, 24 * H, 4 * B * H, 4 * B * H,
             4 * B * H, 4 * B * H, 4 * B * T * H]
    out, at = [], 1 << 20
    for s in sizes:
        out.append(at)
        at += (s + 255) // 256 * 256 + 256
    return out


def test_check_cell_args_gru():
    B, D, H, T = 3, 5, 7, 4
    *p, seq = _gru_ptrs(B, D, H, T, 2)
    chk = ld.lstm_dyn_check_cell_args
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p, 0) == ld.OK
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p, seq) == ld.OK
    assert chk(B, D, H, T, ld.BF16, 3, *p, 0) == ld.ERR_INVALID          # unknown cell
    q = list(p)
    q[6] = 0                                      # c0 is ignored by the GRU and may be NULL
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *q, seq) == ld.OK
    assert chk(B, D, H, T, ld.BF16, ld.CELL_LSTM, *q, 0) == ld.ERR_INVALID
    q = list(p)
    q[7] = q[6]                                   # out_h may sit on the ignored c0
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *q, 0) == ld.OK
    for i in (0, 1, 2, 3, 4, 5):                  # but not on a real input
        q = list(p)
        q[7] = q[i] + (4 if i != 5 else 4)
        assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *q, 0) == ld.ERR_INVALID, i
    # the bias is 6H floats (24H bytes): an output 20H bytes past its start overlaps it
    q = list(p)
    q[8] = q[4] + 20 * H
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *q, 0) == ld.ERR_INVALID
    assert chk(B, D, H, T, ld.BF16, ld.CELL_LSTM, *q, 0) == ld.OK        # LSTM bias is 4H
    for i in range(9):                            # out_seq on top of any used argument
        if i == 6:
            continue
        assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p, p[i]) == ld.ERR_INVALID, i


def test_create_cell_rejects_unknown_cell_without_device():
    with pytest.raises(ld.LstmDynError) as e:
        ld.lstm_dyn_create_cell(4, 4, 4, 4, ld.F32, ld.PERSISTENT, 7)
    assert e.value.code == ld.ERR_INVALID


def test_check_cell_args_rnn():
    """The RNN's W [D][H], U [H][H], b [H]: sizes for the overlap checks."""
    B, D, H, T = 3, 5, 7, 4
    sizes = [B * T * D * 4, 4 * B, D * H * 4, H * H * 4, 4 * H, 4 * B * H, 4 * B * H,
             4 * B * H, 4 * B * H]
    p, at = [], 1 << 20
    for s in sizes:
        p.append(at)
        at += s                                   # packed back to back: no slack between
    chk = ld.lstm_dyn_check_cell_args
    p = [v + (-v % 16) for v in p]                # keep the 16-byte alignment of x, W, U
    assert chk(B, D, H, T, ld.F32, ld.CELL_RNN, *p, 0) == ld.OK
    # with the LSTM's sizes (4x wider W and U) the same buffers overlap
    assert chk(B, D, H, T, ld.F32, ld.CELL_LSTM, *p, 0) == ld.ERR_INVALID
    q = list(p)
    q[6] = 0                                      # c0 ignored
    assert chk(B, D, H, T, ld.F32, ld.CELL_RNN, *q, 0) == ld.OK
    q = list(p)
    q[7] = q[4] + 4 * H - 4                       # out_h on the last bias float
    assert chk(B, D, H, T, ld.F32, ld.CELL_RNN, *q, 0) == ld.ERR_INVALID


def test_check_stop_args():
    B, D, H, T = 3, 5, 7, 4
    *p, seq = _gru_ptrs(B, D, H, T, 2)              # GRU-sized buffers; then v and out_steps
    v = seq + (4 * B * T * H + 255) // 256 * 256 + 256
    st = v + 512
    chk = ld.lstm_dyn_check_stop_args
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v, p[7], p[8], st, seq) == ld.OK
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v, p[7], p[8], st, 0) == ld.OK   # no sequence
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], 0, p[7], p[8], st, 0) == ld.ERR_INVALID
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v, p[7], p[8], 0, 0) == ld.ERR_INVALID
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v + 2, p[7], p[8], st, 0) == ld.ERR_INVALID
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v, p[7], p[8], st + 2, 0) == ld.ERR_INVALID
    for i in (0, 1, 2, 3, 4, 5, 7, 8):            # out_steps on any used argument
        q = p[i]
        assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v, p[7], p[8], q, 0) == ld.ERR_INVALID, i
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], v, p[7], p[8], v, 0) == ld.ERR_INVALID
    # v may not lie under an output, but may share memory with an input
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], p[7], p[7], p[8], st, 0) == ld.ERR_INVALID
    assert chk(B, D, H, T, ld.BF16, ld.CELL_GRU, *p[:7], p[5], p[7], p[8], st, 0) == ld.OK


def test_check_backward_args():
    B, D, H, T = 3, 5, 7, 4
    sizes = [B * T * D * 4, 4 * B, D * 4 * H * 4, H * 4 * H * 4, 16 * H, 4 * B * H, 4 * B * H,
             4 * B * H, 4 * B * H, 4 * B * T * H,                                  # inputs
             4 * B * T * D, 16 * D * H, 16 * H * H, 16 * H, 4 * B * H, 4 * B * H]   # outputs
    p, at = [], 1 << 20
    for s in sizes:
        p.append(at)
        at += (s + 255) // 256 * 256 + 256
    chk = lambda *q: ld.lstm_dyn_check_backward_args(B, D, H, T, ld.F32, ld.CELL_LSTM, *q)
    assert chk(*p) == ld.OK
    q = list(p)
    q[9] = 0                                      # d_seq is optional
    assert chk(*q) == ld.OK
    for i in list(range(9)) + list(range(10, 16)):
        q = list(p)
        q[i] = 0
        assert chk(*q) == ld.ERR_INVALID, i
    for i in range(10, 16):                       # an output on an input or on another output
        for j in range(16):
            if j == i:
                continue
            q = list(p)
            q[i] = q[j]
            assert chk(*q) == ld.ERR_INVALID, (i, j)
    q = list(p)
    q[11] += 2                                    # misaligned dW
    assert chk(*q) == ld.ERR_INVALID
    # GRU and RNN: smaller W, U, b; c0, d_out_c and dc0 may be NULL
    for cell in (ld.CELL_GRU, ld.CELL_RNN):
        q = list(p)
        q[6] = q[8] = q[15] = 0
        assert ld.lstm_dyn_check_backward_args(B, D, H, T, ld.F32, cell, *q) == ld.OK, cell
        q[11] = q[2] + 4 * (D * H - 1)            # dW on W's last element (RNN W is [D][H])
        assert ld.lstm_dyn_check_backward_args(B, D, H, T, ld.F32, cell, *q) == ld.ERR_INVALID, cell
    assert ld.lstm_dyn_check_backward_args(B, D, H, T, ld.F32, 5, *p) == ld.ERR_INVALID


@pytest.mark.parametrize("D,H,dt", [(40, 2048, ld.BF16), (40, 1024, ld.BF16), (24, 256, ld.F32),
                                    (16, 700, ld.F32)])
def test_plan_batch_limits(D, H, dt):
    """512 rows is the most the persistent variants hold (8 owned row tiles per
    wave); the per-step path takes up to the length preparation's 8192."""
    p = ld.lstm_dyn_plan(512, D, H, 5, dt, ld.PERSISTENT, 256)
    assert p["nstate"] == 8
    with pytest.raises(ld.LstmDynError) as e:
        ld.lstm_dyn_plan(513, D, H, 5, dt, ld.PERSISTENT, 256)
    assert e.value.code == ld.ERR_UNSUPPORTED
    ld.lstm_dyn_plan(8192, D, H, 5, dt, ld.PER_STEP, 256)
    with pytest.raises(ld.LstmDynError) as e:
        ld.lstm_dyn_plan(8193, D, H, 5, dt, ld.PER_STEP, 256)
    assert e.value.code == ld.ERR_UNSUPPORTED


def test_wait_bound_option_range():
    """Host-side checks of LSTM_DYN_OPT_TIMEOUT_US need no device: a NULL
    handle is refused before the value is looked at."""
    assert ld._load().lstm_dyn_set_option(None, ld.OPT_TIMEOUT_US, 1) == ld.ERR_INVALID
