"""fp64 CPU oracle of the variable-length LSTM time loop.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.  It shares no code
with the HIP library; the only module both sides use is ``workloads`` (seeded
input generation, no arithmetic of the method).

Two independent implementations live here:

* ``forward``  -- plain C in double precision (``lstm_oracle.c``), the
  definition of the masked recurrence of the paper's Section 9 "RNN cells"
  experiment and Appendix A, with the standard LSTM cell.
* ``brute.forward_per_sequence`` -- pure-Python ``math`` loops that run each
  sequence on its own up to its own length, with no masking and no loop bound:
  a brute-force cross-check for tiny cases.

The same loop with the GRU cell (``forward_gru``) and the tanh RNN cell
(``forward_rnn``) is there too: the paper's loop takes the cell as a
parameter.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lstm_oracle.c")
_LIB = os.path.join(_HERE, "liblstm_oracle.so")
_lib = None

OK, BAD_ARGS, BAD_LENGTHS, NOMEM = 0, 1, 2, 3


class OracleError(RuntimeError):
    pass


def build(force: bool = True) -> str:
    """Compile the C oracle into ``oracle/liblstm_oracle.so`` (gcc, OpenMP).

    -ffp-contract=off keeps every multiply and add separately rounded, so the
    result does not depend on the compiler's choice of fused operations.
    """
    stale = not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC)
    if force or stale:
        tmp = _LIB + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O3", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC",
               "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Lib:
    """ctypes view of one build of ``lstm_oracle.c``."""

    def __init__(self, path: str):
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        lib.lstm_oracle_forward.argtypes = [ctypes.c_int] * 4 + [P] * 9 + [
            ctypes.c_int, ctypes.c_int, P]
        lib.lstm_oracle_forward.restype = ctypes.c_int
        lib.lstm_oracle_forward_seq.argtypes = [ctypes.c_int] * 4 + [P] * 9 + [
            ctypes.c_int, ctypes.c_int, P, P]
        lib.lstm_oracle_forward_seq.restype = ctypes.c_int
        lib.lstm_oracle_forward_gru.argtypes = [ctypes.c_int] * 4 + [P] * 10 + [
            ctypes.c_int, ctypes.c_int, P, P]
        lib.lstm_oracle_forward_gru.restype = ctypes.c_int
        lib.lstm_oracle_forward_rnn.argtypes = [ctypes.c_int] * 4 + [P] * 9 + [
            ctypes.c_int, ctypes.c_int, P, P]
        lib.lstm_oracle_forward_rnn.restype = ctypes.c_int
        lib.lstm_oracle_forward_stop.argtypes = [ctypes.c_int] * 4 + [P] * 6 + [ctypes.c_int, P,
                                                 ctypes.c_double] + [P] * 7 + [ctypes.c_int]
        lib.lstm_oracle_forward_stop.restype = ctypes.c_int
        lib.lstm_oracle_backward.argtypes = [ctypes.c_int] * 4 + [P] * 16 + [ctypes.c_int]
        lib.lstm_oracle_backward.restype = ctypes.c_int
        lib.lstm_oracle_backward_cell.argtypes = [ctypes.c_int] * 5 + [P] * 15 + [ctypes.c_int]
        lib.lstm_oracle_backward_cell.restype = ctypes.c_int
        lib.lstm_oracle_max_threads.argtypes = []
        lib.lstm_oracle_max_threads.restype = ctypes.c_int
        self.lib = lib
        self.path = path


def _load():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = _Lib(_LIB)
    return _lib


def compile_variant(src_text: str, out_path: str) -> str:
    """Compile C source text with the oracle's flags (used by the tests that
    plant mistakes in a copy of the oracle to show the pins catch them)."""
    src = out_path + ".c"
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O1", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared", src,
                    "-o", out_path, "-lm"], check=True)
    return out_path


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def forward_with(path: str):
    """A ``forward`` bound to the library at ``path``."""
    lib = _Lib(path)

    def fwd(*args, **kw):
        return forward(*args, _lib_override=lib, **kw)
    return fwd


def max_threads() -> int:
    return _load().lib.lstm_oracle_max_threads()


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def forward(x, lengths, W, U, b, h0, c0, literal: bool = False, threads: int = 0,
            return_steps: bool = False, return_seq: bool = False, _lib_override=None):
    """Final state (h, c) in float64 of the masked LSTM loop.

    With ``return_seq`` also the output sequence [B, T, H] (float64): the
    hidden state of row b after step t for t < L[b], zero for t >= L[b]; it
    is returned after (h, c) and before the step count.

    x [B, T, D], W [D, 4H], U [H, 4H], b [4H]: fp32 values (widen bf16 data
    with ``workloads.bf16_bits_to_f32`` first); h0/c0 [B, H]: fp32 or fp64
    values (held in fp64, so a run can resume from a returned state); lengths int32
    [B] with 0 <= L[b] <= T, otherwise ``OracleError``.
    """
    lib = (_lib_override or _load()).lib
    x, W, U, b = map(_f32, (x, W, U, b))
    h0 = np.ascontiguousarray(h0, dtype=np.float64)
    c0 = np.ascontiguousarray(c0, dtype=np.float64)
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    B, T, D = x.shape
    H = U.shape[0]
    if W.shape != (D, 4 * H) or U.shape != (H, 4 * H) or b.shape != (4 * H,):
        raise OracleError("weight shapes do not match x and U")
    if L.shape != (B,) or h0.shape != (B, H) or c0.shape != (B, H):
        raise OracleError("lengths/state shapes do not match x")
    h = np.empty((B, H), np.float64)
    c = np.empty((B, H), np.float64)
    steps = ctypes.c_int64(0)
    args = (B, T, D, H, x.ctypes.data, L.ctypes.data, W.ctypes.data, U.ctypes.data,
            b.ctypes.data, h0.ctypes.data, c0.ctypes.data, h.ctypes.data, c.ctypes.data,
            int(bool(literal)), int(threads), ctypes.byref(steps))
    seq = None
    if return_seq:
        seq = np.full((B, T, H), np.nan)  # every entry must be written
        rc = lib.lstm_oracle_forward_seq(*args, seq.ctypes.data)
    else:
        rc = lib.lstm_oracle_forward(*args)
    if rc == BAD_LENGTHS:
        raise OracleError("sequence lengths must lie in [0, T]")
    if rc != OK:
        raise OracleError(f"oracle failed with code {rc}")
    out = (h, c) if seq is None else (h, c, seq)
    if return_steps:
        return (*out, int(steps.value))
    return out


def forward_gru(x, lengths, W, U, b_ih, b_hh, h0, literal: bool = False, threads: int = 0,
                return_seq: bool = False, return_steps: bool = False, _lib_override=None):
    """Final hidden state h in float64 of the masked loop with the GRU cell.

    x [B, T, D], W [D, 3H], U [H, 3H] with gate blocks (r, u, n), b_ih, b_hh
    [3H]: fp32 values; h0 [B, H] fp32 or fp64; lengths as for ``forward``.
    With ``return_seq`` also the output sequence [B, T, H] (zeros past each
    length).
    """
    lib = (_lib_override or _load()).lib
    x, W, U, b_ih, b_hh = map(_f32, (x, W, U, b_ih, b_hh))
    h0 = np.ascontiguousarray(h0, dtype=np.float64)
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    B, T, D = x.shape
    H = U.shape[0]
    if W.shape != (D, 3 * H) or U.shape != (H, 3 * H) or b_ih.shape != (3 * H,) or b_hh.shape != (3 * H,):
        raise OracleError("GRU weight shapes do not match x and U")
    if L.shape != (B,) or h0.shape != (B, H):
        raise OracleError("lengths/state shapes do not match x")
    c0 = np.zeros((B, H), np.float64)
    h = np.empty((B, H), np.float64)
    c = np.empty((B, H), np.float64)
    seq = np.full((B, T, H), np.nan) if return_seq else None
    steps = ctypes.c_int64(0)
    rc = lib.lstm_oracle_forward_gru(B, T, D, H, x.ctypes.data, L.ctypes.data, W.ctypes.data,
                                     U.ctypes.data, b_ih.ctypes.data, b_hh.ctypes.data,
                                     h0.ctypes.data, c0.ctypes.data, h.ctypes.data, c.ctypes.data,
                                     int(bool(literal)), int(threads), ctypes.byref(steps),
                                     seq.ctypes.data if seq is not None else None)
    if rc == BAD_LENGTHS:
        raise OracleError("sequence lengths must lie in [0, T]")
    if rc != OK:
        raise OracleError(f"oracle failed with code {rc}")
    out = (h,) if seq is None else (h, seq)
    if return_steps:
        out = (*out, int(steps.value))
    return out[0] if len(out) == 1 else out


def forward_rnn(x, lengths, W, U, b, h0, literal: bool = False, threads: int = 0,
                return_seq: bool = False, return_steps: bool = False, _lib_override=None):
    """Final hidden state h in float64 of the masked loop with the tanh RNN
    cell h' = tanh(x W + h U + b).

    x [B, T, D], W [D, H], U [H, H], b [H]: fp32 values; h0 [B, H] fp32 or
    fp64; lengths as for ``forward``.  With ``return_seq`` also the output
    sequence [B, T, H] (zeros past each length).
    """
    lib = (_lib_override or _load()).lib
    x, W, U, b = map(_f32, (x, W, U, b))
    h0 = np.ascontiguousarray(h0, dtype=np.float64)
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    B, T, D = x.shape
    H = U.shape[0]
    if W.shape != (D, H) or U.shape != (H, H) or b.shape != (H,):
        raise OracleError("RNN weight shapes do not match x and U")
    if L.shape != (B,) or h0.shape != (B, H):
        raise OracleError("lengths/state shapes do not match x")
    c0 = np.zeros((B, H), np.float64)
    h = np.empty((B, H), np.float64)
    c = np.empty((B, H), np.float64)
    seq = np.full((B, T, H), np.nan) if return_seq else None
    steps = ctypes.c_int64(0)
    rc = lib.lstm_oracle_forward_rnn(B, T, D, H, x.ctypes.data, L.ctypes.data, W.ctypes.data,
                                     U.ctypes.data, b.ctypes.data, h0.ctypes.data, c0.ctypes.data,
                                     h.ctypes.data, c.ctypes.data, int(bool(literal)), int(threads),
                                     ctypes.byref(steps),
                                     seq.ctypes.data if seq is not None else None)
    if rc == BAD_LENGTHS:
        raise OracleError("sequence lengths must lie in [0, T]")
    if rc != OK:
        raise OracleError(f"oracle failed with code {rc}")
    out = (h,) if seq is None else (h, seq)
    if return_steps:
        out = (*out, int(steps.value))
    return out[0] if len(out) == 1 else out


def backward(x, lengths, W, U, b, h0, c0, dh_out, dc_out, dseq=None, _lib_override=None,
             threads: int = 0):
    """Gradients of the masked LSTM loop (backpropagation through time): given
    the upstream gradients of the final state (dh_out, dc_out [B, H]) and
    optionally of the output sequence (dseq [B, T, H]), returns a dict of
    float64 arrays dx [B, T, D], dW [D, 4H], dU [H, 4H], db [4H], dh0, dc0
    [B, H].  Layouts as for ``forward``.  ``threads`` (0: all cores) changes
    the schedule only: every thread count gives the same bits."""
    lib = (_lib_override or _load()).lib
    x, W, U, b = map(_f32, (x, W, U, b))
    f64 = lambda a: np.ascontiguousarray(a, dtype=np.float64)
    h0, c0, dh_out, dc_out = map(f64, (h0, c0, dh_out, dc_out))
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    B, T, D = x.shape
    H = U.shape[0]
    if W.shape != (D, 4 * H) or U.shape != (H, 4 * H) or b.shape != (4 * H,):
        raise OracleError("weight shapes do not match x and U")
    for a in (h0, c0, dh_out, dc_out):
        if a.shape != (B, H):
            raise OracleError("state shapes do not match x")
    ds = f64(dseq) if dseq is not None else None
    if ds is not None and ds.shape != (B, T, H):
        raise OracleError("dseq must be [B, T, H]")
    out = {"dx": np.empty((B, T, D)), "dW": np.empty((D, 4 * H)), "dU": np.empty((H, 4 * H)),
           "db": np.empty(4 * H), "dh0": np.empty((B, H)), "dc0": np.empty((B, H))}
    rc = lib.lstm_oracle_backward(B, T, D, H, x.ctypes.data, L.ctypes.data, W.ctypes.data,
                                  U.ctypes.data, b.ctypes.data, h0.ctypes.data, c0.ctypes.data,
                                  dh_out.ctypes.data, dc_out.ctypes.data,
                                  ds.ctypes.data if ds is not None else None,
                                  *(out[k].ctypes.data for k in ("dx", "dW", "dU", "db", "dh0", "dc0")),
                                  int(threads))
    if rc == BAD_LENGTHS:
        raise OracleError("sequence lengths must lie in [0, T]")
    if rc != OK:
        raise OracleError(f"oracle failed with code {rc}")
    return out


def _backward_cell(cell, x, lengths, W, U, b, b_hh, h0, dh_out, dseq, _lib_override, threads=0):
    lib = (_lib_override or _load()).lib
    x, W, U, b = map(_f32, (x, W, U, b))
    bhh = _f32(b_hh) if b_hh is not None else None
    f64 = lambda a: np.ascontiguousarray(a, dtype=np.float64)
    h0, dh_out = f64(h0), f64(dh_out)
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    B, T, D = x.shape
    H = U.shape[0]
    G = 3 * H if cell == 1 else H
    if W.shape != (D, G) or U.shape != (H, G) or b.shape != (G,):
        raise OracleError("weight shapes do not match x, U and the cell")
    if h0.shape != (B, H) or dh_out.shape != (B, H):
        raise OracleError("state shapes do not match x")
    ds = f64(dseq) if dseq is not None else None
    out = {"dx": np.empty((B, T, D)), "dW": np.empty((D, G)), "dU": np.empty((H, G)),
           "db": np.empty(G), "dh0": np.empty((B, H))}
    dbhh = np.empty(G) if cell == 1 else None
    rc = lib.lstm_oracle_backward_cell(B, T, D, H, cell, x.ctypes.data, L.ctypes.data,
                                       W.ctypes.data, U.ctypes.data, b.ctypes.data,
                                       bhh.ctypes.data if bhh is not None else None,
                                       h0.ctypes.data, dh_out.ctypes.data,
                                       ds.ctypes.data if ds is not None else None,
                                       out["dx"].ctypes.data, out["dW"].ctypes.data,
                                       out["dU"].ctypes.data, out["db"].ctypes.data,
                                       dbhh.ctypes.data if dbhh is not None else None,
                                       out["dh0"].ctypes.data, int(threads))
    if rc == BAD_LENGTHS:
        raise OracleError("sequence lengths must lie in [0, T]")
    if rc != OK:
        raise OracleError(f"oracle failed with code {rc}")
    if dbhh is not None:
        out["db_ih"] = out.pop("db")
        out["db_hh"] = dbhh
    return out


def backward_gru(x, lengths, W, U, b_ih, b_hh, h0, dh_out, dseq=None, _lib_override=None,
                 threads: int = 0):
    """Gradients of the masked loop with the GRU cell: dx, dW [D, 3H],
    dU [H, 3H], db_ih, db_hh [3H], dh0 (float64), from the upstream gradient of
    the final h and optionally of the output sequence."""
    return _backward_cell(1, x, lengths, W, U, b_ih, b_hh, h0, dh_out, dseq, _lib_override, threads)


def backward_rnn(x, lengths, W, U, b, h0, dh_out, dseq=None, _lib_override=None,
                 threads: int = 0):
    """Gradients of the masked loop with the tanh RNN cell: dx, dW [D, H],
    dU [H, H], db [H], dh0 (float64)."""
    return _backward_cell(2, x, lengths, W, U, b, None, h0, dh_out, dseq, _lib_override, threads)


_CELL_IDS = {"lstm": 0, "gru": 1, "rnn": 2}


def forward_stop(x, lengths, W, U, b, h0, c0, v, c_stop, cell: str = "lstm", b_hh=None,
                 threads: int = 0, return_seq: bool = False, _lib_override=None):
    """The loop whose termination is computed from the state: row b runs step
    t while t < L[b] (a cap) and it has not terminated; it terminates after a
    step that leaves its halting score v . h + c_stop positive; the loop ends
    at the first step with no running row.

    Returns (h, c, steps, iters) -- float64 [B, H] twice, int32 [B] steps each
    row ran, the loop iterations -- and the output sequence [B, T, H] after
    them with ``return_seq``.  Layouts as for ``forward`` (cell "lstm"),
    ``forward_gru`` (b = b_ih, ``b_hh``) or ``forward_rnn``; v float [H];
    c0 is carried unchanged for GRU and RNN.
    """
    lib = (_lib_override or _load()).lib
    x, W, U, b, v = map(_f32, (x, W, U, b, v))
    bhh = _f32(b_hh) if b_hh is not None else None
    h0 = np.ascontiguousarray(h0, dtype=np.float64)
    c0 = np.ascontiguousarray(c0, dtype=np.float64)
    L = np.ascontiguousarray(lengths, dtype=np.int32)
    B, T, D = x.shape
    H = U.shape[0]
    g = {"lstm": 4, "gru": 3, "rnn": 1}[cell]
    if W.shape != (D, g * H) or U.shape != (H, g * H) or v.shape != (H,):
        raise OracleError("weight shapes do not match x, U and the cell")
    if L.shape != (B,) or h0.shape != (B, H) or c0.shape != (B, H):
        raise OracleError("lengths/state shapes do not match x")
    if cell == "gru" and (bhh is None or bhh.shape != (3 * H,)):
        raise OracleError("the GRU needs b_hh [3H]")
    h = np.empty((B, H), np.float64)
    c = np.empty((B, H), np.float64)
    steps = np.zeros(B, np.int32)
    iters = ctypes.c_int64(0)
    seq = np.full((B, T, H), np.nan) if return_seq else None
    rc = lib.lstm_oracle_forward_stop(B, T, D, H, x.ctypes.data, L.ctypes.data, W.ctypes.data,
                                      U.ctypes.data, b.ctypes.data,
                                      bhh.ctypes.data if bhh is not None else None,
                                      _CELL_IDS[cell], v.ctypes.data, float(c_stop),
                                      h0.ctypes.data, c0.ctypes.data, h.ctypes.data, c.ctypes.data,
                                      steps.ctypes.data, ctypes.byref(iters),
                                      seq.ctypes.data if seq is not None else None, int(threads))
    if rc == BAD_LENGTHS:
        raise OracleError("sequence lengths must lie in [0, T]")
    if rc != OK:
        raise OracleError(f"oracle failed with code {rc}")
    out = (h, c, steps, int(iters.value))
    return (*out, seq) if return_seq else out


def forward_inputs(inp, rows=None, literal: bool = False, threads: int = 0, seq: bool = False):
    """``forward`` on a ``workloads.Inputs`` batch, optionally on a subset of rows.

    Rows are independent in the definition, so running the oracle on rows
    ``rows`` alone gives exactly those rows of the full batch's result.
    """
    x, W, U = inp.as_f32()
    L, h0, c0 = inp.lengths, inp.h0, inp.c0
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        x, L, h0, c0 = x[rows], L[rows], h0[rows], c0[rows]
    return forward(x, L, W, U, inp.b, h0, c0, literal=literal, threads=threads, return_seq=seq)


def forward_gru_inputs(inp, rows=None, literal: bool = False, threads: int = 0, seq: bool = False):
    """``forward_gru`` on a ``workloads.GruInputs`` batch, optionally on a
    subset of rows (rows are independent, as for ``forward_inputs``)."""
    x, W, U = inp.as_f32()
    L, h0 = inp.lengths, inp.h0
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        x, L, h0 = x[rows], L[rows], h0[rows]
    return forward_gru(x, L, W, U, inp.b_ih, inp.b_hh, h0, literal=literal, threads=threads,
                       return_seq=seq)


def forward_rnn_inputs(inp, rows=None, literal: bool = False, threads: int = 0, seq: bool = False):
    """``forward_rnn`` on a ``workloads.CellInputs`` batch of the RNN cell,
    optionally on a subset of rows."""
    x, W, U = inp.as_f32()
    L, h0 = inp.lengths, inp.h0
    if rows is not None:
        rows = np.asarray(rows, dtype=np.int64)
        x, L, h0 = x[rows], L[rows], h0[rows]
    return forward_rnn(x, L, W, U, inp.b, h0, literal=literal, threads=threads, return_seq=seq)
