"""Chunked resume through the C ABI: a forward over steps [0, t1), then a
forward over [t1, T) that starts from the carried state (h, c) with the
remaining lengths max(L - t1, 0) and x shifted by t1, gives the state of one
forward over the whole sequence (the loop's state is all it carries from one
step to the next).  Compared with the single run bit for bit (no kernel's
arithmetic for a row depends on the other rows), and with the oracle within
the workload's tolerance."""
import numpy as np
import pytest

import oracle
import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import bits, max_err, run, say

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.BF16: 3e-3}
MODES = ["persistent", "per_step"]


def _chunks(inp, t1):
    """The two chunks of inp split at step t1 (each padded to T with zeros)."""
    L = inp.lengths
    x1 = inp.x.copy()
    x1[:, t1:] = 0
    x2 = np.zeros_like(inp.x)
    x2[:, :inp.T - t1] = inp.x[:, t1:]
    first = workloads.Inputs(x=x1, lengths=np.minimum(L, t1).astype(np.int32), W=inp.W, U=inp.U,
                             b=inp.b, h0=inp.h0, c0=inp.c0, dtype=inp.dtype)
    second = lambda h, c: workloads.Inputs(x=x2, lengths=np.maximum(L - t1, 0).astype(np.int32),
                                           W=inp.W, U=inp.U, b=inp.b, h0=h, c0=c, dtype=inp.dtype)
    return first, second


CASES = [
    ("random", (5101, 37, 40, 100, 17, "bf16"), 6),
    ("random", (5102, 20, 24, 64, 13, "f32"), 5),
    ("random", (5103, 70, 130, 1100, 9, "bf16"), 4),
    ("workload", "lstm512_bf16", 77),
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0]}-{c[1] if c[0] == 'workload' else c[1][0]}")
def test_chunked_resume_equals_one_run(case, mode):
    kind, spec, t1 = case
    if kind == "workload":
        inp = workloads.workload_inputs(spec)
    else:
        seed, B, D, H, T, dt = spec
        inp = workloads.random_case(seed, B, D, H, T, dtype=dt)
    tol = TOL[inp.dtype]
    say(f"case resume {kind} {spec} t1={t1} {mode}")
    h_full, c_full, m = run(inp, mode)
    first, second = _chunks(inp, t1)
    h1, c1, _ = run(first, mode, model=m)
    h2, c2, _ = run(second(h1.astype(np.float32), c1.astype(np.float32)), mode, model=m)
    eh, ec = max_err(h2, h_full), max_err(c2, c_full)
    same = np.array_equal(bits(h2), bits(h_full)) and np.array_equal(bits(c2), bits(c_full))
    say(f"  resumed vs one run: max|dh|={eh:.3g} max|dc|={ec:.3g} bitwise={same}")
    # every kernel computes a row the same way whatever the other rows, and
    # the carried state is the loop's own fp32 state: the same bits
    assert same, (eh, ec)
    ho, co = oracle.forward_inputs(inp)
    assert max_err(h2, ho) <= tol and max_err(c2, co) <= tol
    # rows that end within the first chunk are untouched by the second
    done = inp.lengths <= t1
    assert np.array_equal(bits(h2[done]), bits(h1[done])) and np.array_equal(bits(c2[done]), bits(c1[done]))
    m.close()
