"""Failure handling of the bounded waits, forced from the host: with the wait
bound (LSTM_DYN_OPT_TIMEOUT_US) set to 1 microsecond, the cooperative
kernels give up at a wait that lasts longer than that, report
LSTM_DYN_ERR_TIMEOUT through LSTM_DYN_Q_LAST_STATUS and exit normally; with
the default bound restored, the same handle computes what a fresh handle
computes, bit for bit."""
import numpy as np
import pytest

import paper_1810_08061_amd as ld
import workloads
from tests.gpu_util import say, to_device

pytestmark = pytest.mark.gpu


def test_forward_wait_bound():
    import torch
    inp = workloads.random_case(1301, 64, 32, 512, 120, dtype="bf16", lo=60)
    dev = to_device(inp)
    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, "persistent")
    m.set_option(ld.OPT_TIMEOUT_US, 1)
    say("case forward with a 1 us wait bound")
    m.forward(*dev)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.ERR_TIMEOUT
    m.set_option(ld.OPT_TIMEOUT_US, 0)
    h, c = m.forward(*dev)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    f = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, "persistent")
    h2, c2 = f.forward(*dev)
    torch.cuda.synchronize()
    assert torch.equal(h, h2) and torch.equal(c, c2)
    m.close()
    f.close()


@pytest.mark.parametrize("B,H", [(256, 2048), (16, 96)], ids=["whole-loop-launch", "few-row-launch"])
def test_backward_wait_bound(B, H):
    """The reverse loop's cooperative launches (bf16 data): the whole loop
    with column blocks of U (H a multiple of 256), and the launch for the
    steps with at most 16 rows (other H).  Past the bound the launch stops
    with ERR_TIMEOUT; with the bound restored the gradients equal a fresh
    handle's bit for bit.  The whole-loop launch has no grid barrier: its
    waits are those of one workgroup for another's data, which at a few rows
    end within a microsecond; at 256 rows of H = 2048 a workgroup waits
    several microseconds for its siblings in every step."""
    import torch
    inp = workloads.random_case(1302, B, 32, H, 40, dtype="bf16", lo=20)
    dev = to_device(inp)
    rng = np.random.default_rng(1303)
    dh = torch.from_numpy(rng.standard_normal((inp.B, inp.H)).astype(np.float32)).cuda()
    dc = torch.from_numpy(rng.standard_normal((inp.B, inp.H)).astype(np.float32)).cuda()

    def grads(m):
        m.forward_train(*dev)
        g = m.backward(*dev, dh, dc)
        torch.cuda.synchronize()
        return g

    m = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, "persistent")
    m.forward_train(*dev)
    torch.cuda.synchronize()
    m.set_option(ld.OPT_TIMEOUT_US, 1)
    say("case backward with a 1 us wait bound")
    m.backward(*dev, dh, dc)
    torch.cuda.synchronize()
    assert m.query(ld.Q_LAST_STATUS) == ld.ERR_TIMEOUT
    m.set_option(ld.OPT_TIMEOUT_US, 0)
    g = grads(m)
    assert m.query(ld.Q_LAST_STATUS) == ld.OK
    f = ld.LstmDyn(inp.B, inp.D, inp.H, inp.T, inp.dtype, "persistent")
    g2 = grads(f)
    for k in g:
        assert torch.equal(g[k], g2[k]), k
    m.close()
    f.close()
