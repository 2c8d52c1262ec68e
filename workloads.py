"""Seeded synthetic inputs for the variable-length LSTM time loop.

This module is shared by the fp64 oracle (``oracle/``) and by the HIP path's
tests and benchmark.  It draws random numbers and converts storage formats
(fp32 -> bf16 bits and back); it holds none of the method's arithmetic.

The five workloads stand in for the paper's "RNN cells" experiment (Section 9,
Table 1: hidden size 256, batch 32-128, sequence 64/128, fp32, "simple
inputs").  The paper gives no dataset for it; these shapes and distributions
extend that experiment to the sizes a single MI355X is built for.

Recipe (reading of the workload notation):
  * ``N(0, s)`` names the variance: W, U ~ N(0, 1/H) have std H**-0.5, and
    h0, c0 ~ N(0, 0.1) have std sqrt(0.1).
  * Draw order from ``numpy.random.default_rng(seed)``: lengths, x (the full
    [B, T, D] block, padding included), W, U, h0, c0 (the last two only when
    the workload gives them a distribution; otherwise zeros).  A forced length
    is applied to batch index 0 after the draws.
  * Values are drawn in fp64 and cast to fp32; bf16 workloads then round x, W
    and U to bf16 with round-to-nearest-even and keep them as uint16 bit
    patterns.  b = 0 except the forget-gate block b[H:2H] = 1.
  * Geometric lengths use numpy's support {1, 2, ...} with p = 1/mean;
    lognormal lengths use numpy's (mu, sigma) of the underlying normal and are
    rounded half-to-even (``numpy.rint``).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    D: int
    H: int
    T: int
    dtype: str                 # storage/arithmetic type of x, W, U: "f32" or "bf16"
    lengths: tuple             # ("uniform", lo, hi) | ("geometric", mean, lo, hi) | ("lognormal", mu, sigma, lo, hi)
    force: Optional[tuple] = None   # (index, value) applied after the draws
    state_var: float = 0.0     # variance of h0 and c0 (0 -> zeros)
    seed: int = 0
    tol: float = field(default=0.0)  # max-abs tolerance on h and c against the fp64 oracle


WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", B=4, D=16, H=32, T=20, dtype=F32,
                         lengths=("uniform", 0, 20), force=(0, 0), seed=1, tol=1e-5),
    "lstm256_f32": Workload("lstm256_f32", B=32, D=256, H=256, T=100, dtype=F32,
                            lengths=("uniform", 10, 100), state_var=0.1, seed=2, tol=1e-5),
    "lstm512_bf16": Workload("lstm512_bf16", B=64, D=512, H=512, T=200, dtype=BF16,
                             lengths=("uniform", 1, 200), seed=3, tol=3e-3),
    "skewed1024_bf16": Workload("skewed1024_bf16", B=128, D=1024, H=1024, T=500, dtype=BF16,
                                lengths=("geometric", 40.0, 1, 500), force=(0, 500), seed=4, tol=3e-3),
    "large2048_bf16": Workload("large2048_bf16", B=256, D=1024, H=2048, T=1000, dtype=BF16,
                               lengths=("lognormal", 5.0, 0.8, 1, 1000), seed=5, tol=3e-3),
}
ORDER = ["tiny_f32", "lstm256_f32", "lstm512_bf16", "skewed1024_bf16", "large2048_bf16"]


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return uint16 bits."""
    u = np.array(a, dtype=np.float32, copy=True, order="C").view(np.uint32)
    lsb = (u >> 16) & 1
    u += 0x7FFF       # in place; only NaNs with the top payload bits set could wrap
    u += lsb
    u >>= 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to the fp32 values they denote (exact)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def draw_lengths(rng: np.random.Generator, B: int, spec: tuple) -> np.ndarray:
    kind = spec[0]
    if kind == "uniform":
        _, lo, hi = spec
        L = rng.integers(lo, hi + 1, size=B)
    elif kind == "geometric":
        _, mean, lo, hi = spec
        L = np.clip(rng.geometric(1.0 / mean, size=B), lo, hi)
    elif kind == "lognormal":
        _, mu, sigma, lo, hi = spec
        L = np.clip(np.rint(rng.lognormal(mu, sigma, size=B)), lo, hi)
    else:
        raise ValueError(f"unknown length distribution {kind!r}")
    return np.ascontiguousarray(L, dtype=np.int32)


@dataclass
class Inputs:
    """One batch of inputs in the boundary's layouts (all C-contiguous).

    x [B, T, D], W [D, 4H], U [H, 4H]: float32, or uint16 bf16 bits.
    lengths int32 [B]; b float32 [4H]; h0, c0 float32 [B, H].
    Gate blocks along 4H are (i, f, g, o).
    """
    x: np.ndarray
    lengths: np.ndarray
    W: np.ndarray
    U: np.ndarray
    b: np.ndarray
    h0: np.ndarray
    c0: np.ndarray
    dtype: str

    @property
    def B(self):
        return self.x.shape[0]

    @property
    def T(self):
        return self.x.shape[1]

    @property
    def D(self):
        return self.x.shape[2]

    @property
    def H(self):
        return self.U.shape[0]

    def as_f32(self):
        """(x, W, U) as the fp32 values they denote (bf16 widened exactly)."""
        if self.dtype == BF16:
            return bf16_bits_to_f32(self.x), bf16_bits_to_f32(self.W), bf16_bits_to_f32(self.U)
        return self.x, self.W, self.U


def make_inputs(B: int, D: int, H: int, T: int, dtype: str, lengths_spec: tuple,
                seed: int, force: Optional[tuple] = None, state_var: float = 0.0,
                forget_bias: float = 1.0) -> Inputs:
    rng = np.random.default_rng(seed)
    L = draw_lengths(rng, B, lengths_spec)
    x = rng.standard_normal((B, T, D)).astype(np.float32)
    W = (rng.standard_normal((D, 4 * H)) * (1.0 / np.sqrt(H))).astype(np.float32)
    U = (rng.standard_normal((H, 4 * H)) * (1.0 / np.sqrt(H))).astype(np.float32)
    if state_var > 0:
        s = np.sqrt(state_var)
        h0 = (rng.standard_normal((B, H)) * s).astype(np.float32)
        c0 = (rng.standard_normal((B, H)) * s).astype(np.float32)
    else:
        h0 = np.zeros((B, H), np.float32)
        c0 = np.zeros((B, H), np.float32)
    if force is not None:
        L[force[0]] = force[1]
    b = np.zeros(4 * H, np.float32)
    b[H:2 * H] = forget_bias
    if dtype == BF16:
        x, W, U = f32_to_bf16_bits(x), f32_to_bf16_bits(W), f32_to_bf16_bits(U)
    elif dtype != F32:
        raise ValueError(f"unknown dtype {dtype!r}")
    return Inputs(x=x, lengths=L, W=W, U=U, b=b, h0=h0, c0=c0, dtype=dtype)


@dataclass
class CellInputs:
    """One batch for the GRU or the tanh RNN cell in the boundary's layouts
    (C-contiguous).  ``cell`` is "gru" or "rnn"; G = 3H (GRU) or H (RNN).

    x [B, T, D], W [D, G], U [H, G]: float32, or uint16 bf16 bits; GRU gate
    blocks (r, u, n) along 3H.  lengths int32 [B]; h0 float32 [B, H];
    b float32: GRU [6H] = b_ih [3H] followed by b_hh [3H], RNN [H].
    """
    x: np.ndarray
    lengths: np.ndarray
    W: np.ndarray
    U: np.ndarray
    b: np.ndarray
    h0: np.ndarray
    dtype: str
    cell: str = "gru"

    B = Inputs.B
    T = Inputs.T
    D = Inputs.D
    H = Inputs.H
    as_f32 = Inputs.as_f32

    @property
    def b_ih(self):
        return self.b[:3 * self.H]

    @property
    def b_hh(self):
        return self.b[3 * self.H:]


GruInputs = CellInputs
_CELL_COLS = {"gru": (3, 6), "rnn": (1, 1)}   # (columns of W and U, bias entries) per hidden unit
# Variance of W and U times H: 1 for the GRU (as for the LSTM); 1/3 for the tanh
# RNN, the variance of the uniform(-1/sqrt(H), 1/sqrt(H)) initialisation that
# torch.nn.RNN uses by default.  At 1 the plain tanh recurrence sits at the edge
# of chaos (recurrent gain about 1), where any rounding of h, bf16 or fp32,
# grows with the step count instead of dying out.
_CELL_WVAR = {"gru": 1.0, "rnn": 1.0 / 3.0}


def make_cell_inputs(cell: str, B: int, D: int, H: int, T: int, dtype: str, lengths_spec: tuple,
                     seed: int, force: Optional[tuple] = None, state_var: float = 0.0,
                     bias_var: float = 0.1) -> CellInputs:
    """GRU or RNN batch.  Draw order: lengths, x, W, U, b, h0 (h0 only when
    ``state_var`` > 0); W, U ~ N(0, 1/H) (GRU) or N(0, 1/(3H)) (RNN),
    biases ~ N(0, bias_var)."""
    g, nb = _CELL_COLS[cell]
    ws = np.sqrt(_CELL_WVAR[cell] / H)
    rng = np.random.default_rng(seed)
    L = draw_lengths(rng, B, lengths_spec)
    x = rng.standard_normal((B, T, D)).astype(np.float32)
    W = (rng.standard_normal((D, g * H)) * ws).astype(np.float32)
    U = (rng.standard_normal((H, g * H)) * ws).astype(np.float32)
    b = (rng.standard_normal(nb * H) * np.sqrt(bias_var)).astype(np.float32)
    if state_var > 0:
        h0 = (rng.standard_normal((B, H)) * np.sqrt(state_var)).astype(np.float32)
    else:
        h0 = np.zeros((B, H), np.float32)
    if force is not None:
        L[force[0]] = force[1]
    if dtype == BF16:
        x, W, U = f32_to_bf16_bits(x), f32_to_bf16_bits(W), f32_to_bf16_bits(U)
    elif dtype != F32:
        raise ValueError(f"unknown dtype {dtype!r}")
    return CellInputs(x=x, lengths=L, W=W, U=U, b=b, h0=h0, dtype=dtype, cell=cell)


def make_gru_inputs(*args, **kw) -> CellInputs:
    return make_cell_inputs("gru", *args, **kw)


def cell_workload_inputs(cell: str, name: str) -> CellInputs:
    """The GRU or RNN batch of workload ``name``: its shapes, dtype and state
    distribution with that cell's weights; the same seed, so the lengths and
    x are those of the LSTM batch."""
    w = WORKLOADS[name]
    return make_cell_inputs(cell, w.B, w.D, w.H, w.T, w.dtype, w.lengths, w.seed, w.force,
                            w.state_var)


def gru_workload_inputs(name: str) -> CellInputs:
    return cell_workload_inputs("gru", name)


def random_cell_case(cell: str, seed: int, B: int, D: int, H: int, T: int, dtype: str = F32,
                     lo: int = 0, hi: Optional[int] = None, state_var: float = 0.1) -> CellInputs:
    """A small seeded GRU or RNN case with uniform lengths in [lo, hi] (hi
    defaults to T)."""
    return make_cell_inputs(cell, B, D, H, T, dtype, ("uniform", lo, T if hi is None else hi),
                            seed, state_var=state_var)


def random_gru_case(*args, **kw) -> CellInputs:
    return random_cell_case("gru", *args, **kw)


def workload_inputs(name: str) -> Inputs:
    w = WORKLOADS[name]
    return make_inputs(w.B, w.D, w.H, w.T, w.dtype, w.lengths, w.seed, w.force, w.state_var)


def random_case(seed: int, B: int, D: int, H: int, T: int, dtype: str = F32,
                lo: int = 0, hi: Optional[int] = None, state_var: float = 0.1) -> Inputs:
    """A small seeded case with uniform lengths in [lo, hi] (hi defaults to T)."""
    return make_inputs(B, D, H, T, dtype, ("uniform", lo, T if hi is None else hi), seed,
                       state_var=state_var)
