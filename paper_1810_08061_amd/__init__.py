"""Variable-length LSTM time loop for MI355X (gfx950): Python binding.

A thin ctypes layer over ``liblstm_dyn.so`` (C ABI in ``include/lstm_dyn.h``).
Every step of the computation runs in the library's HIP kernels; torch is used
only to own device memory and to name streams.  Importing this module does not
need a GPU; calling ``lstm_dyn_create`` does.  If the library has not been
built, loading it raises ``ImportError`` -- there is no fallback path.

Functions mirror the C ABI (same names); ``LstmDyn`` wraps a handle for torch
tensors.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "F32", "BF16", "PERSISTENT", "PER_STEP", "LstmDynError", "LstmDyn", "library_path",
    "lstm_dyn_create", "lstm_dyn_forward", "lstm_dyn_destroy", "lstm_dyn_query",
    "lstm_dyn_strerror", "lstm_dyn_plan", "lstm_dyn_check_args", "lstm_dyn_set_option",
    "lstm_dyn_step_trace", "lstm_dyn_forward_seq", "lstm_dyn_check_seq_args",
    "lstm_dyn_create_cell", "lstm_dyn_check_cell_args", "CELL_LSTM", "CELL_GRU", "CELL_RNN",
    "lstm_dyn_forward_stop", "lstm_dyn_check_stop_args", "lstm_dyn_forward_train",
    "lstm_dyn_backward", "lstm_dyn_check_backward_args", "lstm_dyn_forward_noalloc",
    "NOALLOC_SCRATCH_BYTES",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
# LSTM_DYN_LIB may name another build of the library (the timing-stress
# diagnostic build, liblstm_dyn_stress.so); there is no fallback either way
_LIB_PATH = os.environ.get("LSTM_DYN_LIB") or os.path.join(_HERE, "liblstm_dyn.so")

F32, BF16 = 0, 1
PERSISTENT, PER_STEP = 0, 1
CELL_LSTM, CELL_GRU, CELL_RNN = 0, 1, 2
OK, ERR_INVALID, ERR_HIP, ERR_NOMEM, ERR_UNSUPPORTED, ERR_BAD_LENGTHS, ERR_TIMEOUT, \
    ERR_TOO_LARGE = range(8)
NOALLOC_SCRATCH_BYTES = 128 << 20   # LSTM_DYN_NOALLOC_SCRATCH_BYTES
Q_LAST_STATUS, Q_STEPS_EXECUTED, Q_LAUNCHES_PER_FORWARD, Q_GROUPS, Q_WORKSPACE_BYTES, \
    Q_TOTAL_ROWS, Q_TIME_PREP_NS, Q_TIME_INPROJ_NS, Q_TIME_LOOP_NS = range(9)
OPT_TIMING, OPT_STEP_TRACE, OPT_TIMEOUT_US = 0, 1, 2

_DTYPES = {"f32": F32, "fp32": F32, "float32": F32, "bf16": BF16, "bfloat16": BF16}
_MODES = {"persistent": PERSISTENT, "per_step": PER_STEP}
_CELLS = {"lstm": CELL_LSTM, "gru": CELL_GRU, "rnn": CELL_RNN}
_CELL_SHAPES = {CELL_LSTM: (4, 4), CELL_GRU: (3, 6), CELL_RNN: (1, 1)}  # W/U columns, bias, per unit


class LstmDynError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {lstm_dyn_strerror(code)} (status {code})")


class _Plan(ctypes.Structure):
    _fields_ = [("mt", ctypes.c_int), ("groups", ctypes.c_int), ("ksw", ctypes.c_int),
                ("kw", ctypes.c_int), ("hpad", ctypes.c_int), ("bpad", ctypes.c_int),
                ("lds_bytes", ctypes.c_int), ("nstate", ctypes.c_int),
                ("workspace_bytes", ctypes.c_longlong), ("single", ctypes.c_int),
                ("single_kd", ctypes.c_int), ("single_nt", ctypes.c_int)]


_lib = None


def library_path() -> str:
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_1810_08061_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I, LL = ctypes.c_void_p, ctypes.c_int, ctypes.c_longlong
    lib.lstm_dyn_create.argtypes = [ctypes.POINTER(P), I, I, I, I, I, I]
    lib.lstm_dyn_create.restype = I
    lib.lstm_dyn_create_cell.argtypes = [ctypes.POINTER(P), I, I, I, I, I, I, I]
    lib.lstm_dyn_create_cell.restype = I
    lib.lstm_dyn_check_cell_args.argtypes = [I] * 6 + [P] * 10
    lib.lstm_dyn_check_cell_args.restype = I
    lib.lstm_dyn_forward_stop.argtypes = [P] * 9 + [ctypes.c_float] + [P] * 5
    lib.lstm_dyn_forward_stop.restype = I
    lib.lstm_dyn_check_stop_args.argtypes = [I] * 6 + [P] * 12
    lib.lstm_dyn_check_stop_args.restype = I
    lib.lstm_dyn_forward_train.argtypes = [P] * 12
    lib.lstm_dyn_forward_train.restype = I
    lib.lstm_dyn_backward.argtypes = [P] * 18
    lib.lstm_dyn_backward.restype = I
    lib.lstm_dyn_check_backward_args.argtypes = [I] * 6 + [P] * 16
    lib.lstm_dyn_check_backward_args.restype = I
    lib.lstm_dyn_forward.argtypes = [P] * 11
    lib.lstm_dyn_forward_noalloc.argtypes = [I] * 5 + [P] * 11
    lib.lstm_dyn_forward_noalloc.restype = I
    lib.lstm_dyn_forward.restype = I
    lib.lstm_dyn_forward_seq.argtypes = [P] * 12
    lib.lstm_dyn_forward_seq.restype = I
    lib.lstm_dyn_check_seq_args.argtypes = [I] * 5 + [P] * 10
    lib.lstm_dyn_check_seq_args.restype = I
    lib.lstm_dyn_destroy.argtypes = [P]
    lib.lstm_dyn_destroy.restype = I
    lib.lstm_dyn_query.argtypes = [P, I, ctypes.POINTER(LL)]
    lib.lstm_dyn_query.restype = I
    lib.lstm_dyn_set_option.argtypes = [P, I, LL]
    lib.lstm_dyn_set_option.restype = I
    lib.lstm_dyn_step_trace.argtypes = [P, ctypes.POINTER(LL), I, ctypes.POINTER(I), ctypes.POINTER(I)]
    lib.lstm_dyn_step_trace.restype = I
    lib.lstm_dyn_strerror.argtypes = [I]
    lib.lstm_dyn_strerror.restype = ctypes.c_char_p
    lib.lstm_dyn_plan.argtypes = [I] * 7 + [ctypes.POINTER(_Plan)]
    lib.lstm_dyn_plan.restype = I
    lib.lstm_dyn_check_args.argtypes = [I] * 5 + [P] * 9
    lib.lstm_dyn_check_args.restype = I
    _lib = lib
    return lib


# --- C ABI mirrors ----------------------------------------------------------

def lstm_dyn_strerror(code: int) -> str:
    return _load().lstm_dyn_strerror(int(code)).decode()


def lstm_dyn_create(B: int, D: int, H: int, T_max: int, dtype: int, mode: int) -> int:
    h = ctypes.c_void_p()
    rc = _load().lstm_dyn_create(ctypes.byref(h), B, D, H, T_max, dtype, mode)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_create")
    return h.value


def lstm_dyn_create_cell(B: int, D: int, H: int, T_max: int, dtype: int, mode: int,
                         cell: int) -> int:
    h = ctypes.c_void_p()
    rc = _load().lstm_dyn_create_cell(ctypes.byref(h), B, D, H, T_max, dtype, mode, cell)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_create_cell")
    return h.value


def lstm_dyn_forward(handle: int, x: int, lengths: int, W: int, U: int, b: int, h0: int, c0: int,
                     out_h: int, out_c: int, stream: int = 0) -> None:
    rc = _load().lstm_dyn_forward(handle, x, lengths, W, U, b, h0, c0, out_h, out_c, stream)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_forward")


def lstm_dyn_forward_noalloc(B: int, D: int, H: int, T_max: int, dtype: int, x: int, lengths: int,
                             W: int, U: int, b: int, h0: int, c0: int, out_h: int, out_c: int,
                             status: int = 0, stream: int = 0) -> None:
    rc = _load().lstm_dyn_forward_noalloc(B, D, H, T_max, dtype, x, lengths, W, U, b, h0, c0,
                                          out_h, out_c, status, stream)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_forward_noalloc")


def lstm_dyn_forward_seq(handle: int, x: int, lengths: int, W: int, U: int, b: int, h0: int,
                         c0: int, out_h: int, out_c: int, out_seq: int, stream: int = 0) -> None:
    rc = _load().lstm_dyn_forward_seq(handle, x, lengths, W, U, b, h0, c0, out_h, out_c, out_seq,
                                      stream)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_forward_seq")


def lstm_dyn_forward_stop(handle: int, x: int, lengths: int, W: int, U: int, b: int, h0: int,
                          c0: int, stop_v: int, stop_c: float, out_h: int, out_c: int,
                          out_steps: int, out_seq: int = 0, stream: int = 0) -> None:
    rc = _load().lstm_dyn_forward_stop(handle, x, lengths, W, U, b, h0, c0, stop_v,
                                       ctypes.c_float(stop_c), out_h, out_c, out_steps, out_seq,
                                       stream)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_forward_stop")


def lstm_dyn_forward_train(handle: int, x: int, lengths: int, W: int, U: int, b: int, h0: int,
                           c0: int, out_h: int, out_c: int, out_seq: int = 0, stream: int = 0) -> None:
    rc = _load().lstm_dyn_forward_train(handle, x, lengths, W, U, b, h0, c0, out_h, out_c, out_seq,
                                        stream)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_forward_train")


def lstm_dyn_backward(handle: int, x: int, lengths: int, W: int, U: int, b: int, h0: int, c0: int,
                      d_out_h: int, d_out_c: int, d_seq: int, dx: int, dW: int, dU: int, db: int,
                      dh0: int, dc0: int, stream: int = 0) -> None:
    rc = _load().lstm_dyn_backward(handle, x, lengths, W, U, b, h0, c0, d_out_h, d_out_c, d_seq,
                                   dx, dW, dU, db, dh0, dc0, stream)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_backward")


def lstm_dyn_check_backward_args(B: int, D: int, H: int, T_max: int, dtype: int, cell: int,
                                 *ptrs) -> int:
    """Pointers in the order of lstm_dyn_backward: x, lengths, W, U, b, h0, c0,
    d_out_h, d_out_c, d_seq, dx, dW, dU, db, dh0, dc0."""
    return _load().lstm_dyn_check_backward_args(B, D, H, T_max, dtype, cell, *ptrs)


def lstm_dyn_destroy(handle: int) -> None:
    rc = _load().lstm_dyn_destroy(handle)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_destroy")


def lstm_dyn_query(handle: int, what: int) -> int:
    v = ctypes.c_longlong(0)
    rc = _load().lstm_dyn_query(handle, what, ctypes.byref(v))
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_query")
    return int(v.value)


def lstm_dyn_set_option(handle: int, option: int, value: int) -> None:
    rc = _load().lstm_dyn_set_option(handle, option, value)
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_set_option")


def lstm_dyn_step_trace(handle: int, capacity: int):
    """Step timestamps of the last forward (seconds, relative to the first):
    four per step (start, partials done, state done, arrival) and the loop
    end; requires OPT_STEP_TRACE."""
    buf = (ctypes.c_longlong * capacity)()
    n, khz = ctypes.c_int(0), ctypes.c_int(0)
    rc = _load().lstm_dyn_step_trace(handle, buf, capacity, ctypes.byref(n), ctypes.byref(khz))
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_step_trace")
    t = [buf[i] for i in range(n.value)]
    return [(v - t[0]) / (khz.value * 1e3) for v in t] if t else []


def lstm_dyn_plan(B: int, D: int, H: int, T_max: int, dtype: int, mode: int, num_cus: int) -> dict:
    p = _Plan()
    rc = _load().lstm_dyn_plan(B, D, H, T_max, dtype, mode, num_cus, ctypes.byref(p))
    if rc != OK:
        raise LstmDynError(rc, "lstm_dyn_plan")
    return {name: getattr(p, name) for name, _ in _Plan._fields_}


def lstm_dyn_check_args(B: int, D: int, H: int, T_max: int, dtype: int, x: int, lengths: int,
                        W: int, U: int, b: int, h0: int, c0: int, out_h: int, out_c: int) -> int:
    return _load().lstm_dyn_check_args(B, D, H, T_max, dtype, x, lengths, W, U, b, h0, c0,
                                       out_h, out_c)


def lstm_dyn_check_seq_args(B: int, D: int, H: int, T_max: int, dtype: int, x: int, lengths: int,
                            W: int, U: int, b: int, h0: int, c0: int, out_h: int, out_c: int,
                            out_seq: int) -> int:
    return _load().lstm_dyn_check_seq_args(B, D, H, T_max, dtype, x, lengths, W, U, b, h0, c0,
                                           out_h, out_c, out_seq)


def lstm_dyn_check_cell_args(B: int, D: int, H: int, T_max: int, dtype: int, cell: int, x: int,
                             lengths: int, W: int, U: int, b: int, h0: int, c0: int, out_h: int,
                             out_c: int, out_seq: int) -> int:
    return _load().lstm_dyn_check_cell_args(B, D, H, T_max, dtype, cell, x, lengths, W, U, b,
                                            h0, c0, out_h, out_c, out_seq)


def lstm_dyn_check_stop_args(B: int, D: int, H: int, T_max: int, dtype: int, cell: int, x: int,
                             lengths: int, W: int, U: int, b: int, h0: int, c0: int, stop_v: int,
                             out_h: int, out_c: int, out_steps: int, out_seq: int) -> int:
    return _load().lstm_dyn_check_stop_args(B, D, H, T_max, dtype, cell, x, lengths, W, U, b, h0,
                                            c0, stop_v, out_h, out_c, out_steps, out_seq)


# --- torch convenience wrapper ---------------------------------------------

class LstmDyn:
    """One handle of the library for fixed (B, D, H, T_max, dtype, mode, cell).

    ``forward`` takes CUDA (HIP) tensors in the layouts of the C ABI:
    x [B, T_max, D] and W [D, G], U [H, G] in the handle's dtype
    (torch.float32 or torch.bfloat16), lengths int32 [B], b float32,
    h0/c0 float32 [B, H]; it returns (out_h, out_c) float32 [B, H].
    LSTM: G = 4H, b [4H].  GRU: G = 3H, b [6H] = b_ih ++ b_hh.  RNN: G = H,
    b [H].  GRU and RNN: c0 is ignored (may be None) and out_c is zeros.
    """

    def __init__(self, B: int, D: int, H: int, T_max: int, dtype="bf16", mode="persistent",
                 cell="lstm"):
        self.B, self.D, self.H, self.T = B, D, H, T_max
        self.dtype = _DTYPES[dtype] if isinstance(dtype, str) else int(dtype)
        self.mode = _MODES[mode] if isinstance(mode, str) else int(mode)
        self.cell = _CELLS[cell] if isinstance(cell, str) else int(cell)
        self.handle = lstm_dyn_create_cell(B, D, H, T_max, self.dtype, self.mode, self.cell)

    def _check(self, name, t, dtype, shape):
        import torch
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError(f"{name} must be a device tensor")
        if t.dtype != dtype:
            raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")

    def _inputs(self, x, lengths, W, U, b, h0, c0, out_h, out_c, stream):
        """Check the inputs, allocate missing outputs; returns (c0 pointer,
        out_h, out_c, stream handle)."""
        import torch
        B, D, H, T = self.B, self.D, self.H, self.T
        et = torch.bfloat16 if self.dtype == BF16 else torch.float32
        g, nbias = _CELL_SHAPES[self.cell]
        G, nb = g * H, nbias * H
        for name, t, dt, shape in (("x", x, et, (B, T, D)), ("lengths", lengths, torch.int32, (B,)),
                                   ("W", W, et, (D, G)), ("U", U, et, (H, G)),
                                   ("b", b, torch.float32, (nb,)),
                                   ("h0", h0, torch.float32, (B, H))):
            self._check(name, t, dt, shape)
        if c0 is not None or self.cell == CELL_LSTM:
            self._check("c0", c0, torch.float32, (B, H))
        if out_h is None:
            out_h = torch.empty((B, H), dtype=torch.float32, device=x.device)
        if out_c is None:
            out_c = torch.empty((B, H), dtype=torch.float32, device=x.device)
        self._check("out_h", out_h, torch.float32, (B, H))
        self._check("out_c", out_c, torch.float32, (B, H))
        if stream is None:
            stream = torch.cuda.current_stream(x.device)
        s = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        return (c0.data_ptr() if c0 is not None else 0), out_h, out_c, s

    def forward(self, x, lengths, W, U, b, h0, c0=None, out_h=None, out_c=None, stream=None):
        c0p, out_h, out_c, s = self._inputs(x, lengths, W, U, b, h0, c0, out_h, out_c, stream)
        lstm_dyn_forward(self.handle, x.data_ptr(), lengths.data_ptr(), W.data_ptr(),
                         U.data_ptr(), b.data_ptr(), h0.data_ptr(), c0p,
                         out_h.data_ptr(), out_c.data_ptr(), s)
        return out_h, out_c

    __call__ = forward

    def forward_seq(self, x, lengths, W, U, b, h0, c0=None, out_h=None, out_c=None, out_seq=None,
                    stream=None):
        """``forward``, and also the output sequence out_seq float32 [B, T_max, H]:
        the hidden state of row b after step t for t < L[b], zero after.
        Returns (out_h, out_c, out_seq)."""
        import torch
        c0p, out_h, out_c, s = self._inputs(x, lengths, W, U, b, h0, c0, out_h, out_c, stream)
        if out_seq is None:
            out_seq = torch.empty((self.B, self.T, self.H), dtype=torch.float32, device=x.device)
        self._check("out_seq", out_seq, torch.float32, (self.B, self.T, self.H))
        lstm_dyn_forward_seq(self.handle, x.data_ptr(), lengths.data_ptr(), W.data_ptr(),
                             U.data_ptr(), b.data_ptr(), h0.data_ptr(), c0p,
                             out_h.data_ptr(), out_c.data_ptr(), out_seq.data_ptr(), s)
        return out_h, out_c, out_seq

    def forward_stop(self, x, lengths, W, U, b, h0, c0, stop_v, stop_c, out_h=None, out_c=None,
                     out_steps=None, out_seq=None, with_seq=False, stream=None):
        """The loop with its termination computed from the state: row b ends
        after a step that leaves stop_v . h + stop_c > 0 (stop_v float32 [H]);
        lengths are caps.  Returns (out_h, out_c, out_steps) and, with
        ``with_seq`` or a given ``out_seq``, the output sequence after them."""
        import torch
        c0p, out_h, out_c, s = self._inputs(x, lengths, W, U, b, h0, c0, out_h, out_c, stream)
        self._check("stop_v", stop_v, torch.float32, (self.H,))
        if out_steps is None:
            out_steps = torch.empty((self.B,), dtype=torch.int32, device=x.device)
        self._check("out_steps", out_steps, torch.int32, (self.B,))
        if out_seq is None and with_seq:
            out_seq = torch.empty((self.B, self.T, self.H), dtype=torch.float32, device=x.device)
        if out_seq is not None:
            self._check("out_seq", out_seq, torch.float32, (self.B, self.T, self.H))
        lstm_dyn_forward_stop(self.handle, x.data_ptr(), lengths.data_ptr(), W.data_ptr(),
                              U.data_ptr(), b.data_ptr(), h0.data_ptr(), c0p, stop_v.data_ptr(),
                              float(stop_c), out_h.data_ptr(), out_c.data_ptr(),
                              out_steps.data_ptr(),
                              out_seq.data_ptr() if out_seq is not None else 0, s)
        return (out_h, out_c, out_steps) if out_seq is None else (out_h, out_c, out_steps, out_seq)

    def forward_train(self, x, lengths, W, U, b, h0, c0=None, out_h=None, out_c=None, out_seq=None,
                      with_seq=False, stream=None):
        """``forward`` that also keeps what ``backward`` needs.
        Returns (out_h, out_c) and, with ``with_seq`` or a given ``out_seq``,
        the output sequence after them."""
        import torch
        c0p, out_h, out_c, s = self._inputs(x, lengths, W, U, b, h0, c0, out_h, out_c, stream)
        if out_seq is None and with_seq:
            out_seq = torch.empty((self.B, self.T, self.H), dtype=torch.float32, device=x.device)
        if out_seq is not None:
            self._check("out_seq", out_seq, torch.float32, (self.B, self.T, self.H))
        lstm_dyn_forward_train(self.handle, x.data_ptr(), lengths.data_ptr(), W.data_ptr(),
                               U.data_ptr(), b.data_ptr(), h0.data_ptr(), c0p, out_h.data_ptr(),
                               out_c.data_ptr(), out_seq.data_ptr() if out_seq is not None else 0, s)
        return (out_h, out_c) if out_seq is None else (out_h, out_c, out_seq)

    def backward(self, x, lengths, W, U, b, h0, c0, d_out_h, d_out_c=None, d_seq=None,
                 stream=None, out=None):
        """Gradients after ``forward_train`` with the same inputs; returns a
        dict of float32 tensors dx [B, T, D], dW [D, G], dU [H, G], db, dh0
        [B, H] and, for the LSTM, dc0 [B, H] (G and db as the cell's weights:
        LSTM 4H, [4H]; GRU 3H, [6H] = d b_ih ++ d b_hh; RNN H, [H]).  GRU and
        RNN ignore c0 and d_out_c (None allowed).  out: a dict with those keys
        holding caller-owned contiguous tensors of those shapes (4-byte
        aligned), which receive the gradients and are returned."""
        import torch
        B, D, H, T = self.B, self.D, self.H, self.T
        g, nb = _CELL_SHAPES[self.cell]
        lstm = self.cell == CELL_LSTM
        dev = x.device
        self._check("d_out_h", d_out_h, torch.float32, (B, H))
        if lstm or d_out_c is not None:
            self._check("d_out_c", d_out_c, torch.float32, (B, H))
        if d_seq is not None:
            self._check("d_seq", d_seq, torch.float32, (B, T, H))
        shapes = {"dx": (B, T, D), "dW": (D, g * H), "dU": (H, g * H), "db": (nb * H,), "dh0": (B, H)}
        if lstm:
            shapes["dc0"] = (B, H)
        if out is None:
            out = {k: torch.empty(v, device=dev) for k, v in shapes.items()}
        else:
            if sorted(out) != sorted(shapes):
                raise ValueError(f"out must hold exactly {sorted(shapes)}")
            for k, v in shapes.items():
                self._check(k, out[k], torch.float32, v)
        if stream is None:
            stream = torch.cuda.current_stream(dev)
        s = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
        ptr = lambda t: t.data_ptr() if t is not None else 0
        lstm_dyn_backward(self.handle, x.data_ptr(), lengths.data_ptr(), W.data_ptr(), U.data_ptr(),
                          b.data_ptr(), h0.data_ptr(), ptr(c0) if lstm else 0, d_out_h.data_ptr(),
                          ptr(d_out_c) if lstm else 0, ptr(d_seq),
                          *(out[k].data_ptr() for k in ("dx", "dW", "dU", "db", "dh0")),
                          out["dc0"].data_ptr() if lstm else 0, s)
        return out

    def query(self, what: int) -> int:
        return lstm_dyn_query(self.handle, what)

    def set_option(self, option: int, value: int) -> None:
        lstm_dyn_set_option(self.handle, option, value)

    def step_trace(self) -> list:
        return lstm_dyn_step_trace(self.handle, 4 * self.T + 1)

    def close(self):
        if getattr(self, "handle", None):
            lstm_dyn_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
