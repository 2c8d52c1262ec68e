"""Helpers for the GPU tests: move seeded inputs to the device, run the HIP
path through the C ABI, compare with the fp64 oracle."""
from __future__ import annotations

import sys

import numpy as np

import paper_1810_08061_amd as ld
import workloads


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_device(inp: workloads.Inputs, device="cuda"):
    import torch
    if inp.dtype == workloads.BF16:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    else:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    return (conv(inp.x), torch.from_numpy(np.ascontiguousarray(inp.lengths, dtype=np.int32)).to(device),
            conv(inp.W), conv(inp.U), f32(inp.b), f32(inp.h0), f32(inp.c0))


def run(inp: workloads.Inputs, mode="persistent", model=None, dev=None, out=None):
    """Forward on the GPU; returns (h, c) as float64 numpy plus the handle."""
    import torch
    m = model or ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, mode)
    dev = dev or to_device(inp)
    kw = {}
    if out is not None:
        kw = {"out_h": out[0], "out_c": out[1]}
    h, c = m.forward(*dev, **kw)
    torch.cuda.synchronize()
    return h.cpu().numpy().astype(np.float64), c.cpu().numpy().astype(np.float64), m


def max_err(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) if np.size(a) else 0.0


def bits(a):
    return np.ascontiguousarray(a, dtype=np.float64).view(np.uint64)
