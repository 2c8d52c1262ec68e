"""Pins of the fp64 oracle to facts that do not come from the oracle itself.

Each ``pin_*`` takes a ``forward`` callable with the signature of
``oracle.forward`` and raises AssertionError when the implementation disagrees
with what the definition (AutoGraph Section 9 "RNN cells", Appendix A) or the
mathematics fixes.  ``test_oracle.py`` runs every pin on the real oracle;
``test_oracle_mutants.py`` runs them on copies of the oracle with planted
mistakes and checks that each mistake is caught by at least one pin.
"""
from __future__ import annotations

import math

import numpy as np

import workloads
import oracle
from oracle import brute


def _case(seed, B, D, H, T, lo=0, hi=None, state_var=0.1):
    inp = workloads.random_case(seed, B, D, H, T, lo=lo, hi=hi, state_var=state_var)
    return inp.x.copy(), inp.lengths.copy(), inp.W.copy(), inp.U.copy(), inp.b.copy(), \
        inp.h0.copy(), inp.c0.copy()


def _bits_equal(a, b):
    return np.array_equal(np.asarray(a).view(np.uint64), np.asarray(b).view(np.uint64))


def pin_zero_weights_closed_form(fwd):
    """W = U = 0, b = 0: every sigmoid gate is exactly 1/2 and g = tanh(0) = 0,
    so c after L steps is 2**-L * c0 (exact in binary floating point) and
    h = tanh(c) / 2; a row of length 0 keeps (h0, c0)."""
    B, D, H, T = 6, 5, 7, 9
    x, L, W, U, b, h0, c0 = _case(11, B, D, H, T)
    L[:] = [0, 1, 2, 5, 9, 3]
    W[:] = 0
    U[:] = 0
    b[:] = 0
    h, c = fwd(x, L, W, U, b, h0, c0)
    c0d = c0.astype(np.float64)
    for r in range(B):
        n = int(L[r])
        if n == 0:
            assert _bits_equal(c[r], c0d[r]) and _bits_equal(h[r], h0[r].astype(np.float64))
            continue
        want_c = np.ldexp(c0d[r], -n)
        assert _bits_equal(c[r], want_c), (r, c[r], want_c)
        want_h = np.array([0.5 * math.tanh(v) for v in want_c])
        assert np.max(np.abs(h[r] - want_h)) <= 1e-16


def pin_forget_bias_closed_form(fwd):
    """W = U = 0 and a forget-gate bias beta (gate blocks i, f, g, o): i = o = 1/2,
    g = 0, f = logistic(beta), so c_L = logistic(beta)**L * c0, h = tanh(c_L) / 2."""
    B, D, H, T = 4, 3, 5, 12
    x, L, W, U, b, h0, c0 = _case(12, B, D, H, T)
    L[:] = [12, 7, 1, 4]
    W[:] = 0
    U[:] = 0
    b[:] = 0
    beta = 1.0
    b[H:2 * H] = beta
    h, c = fwd(x, L, W, U, b, h0, c0)
    f = 1.0 / (1.0 + math.exp(-beta))
    for r in range(B):
        want_c = c0[r].astype(np.float64) * f ** int(L[r])
        assert np.max(np.abs(c[r] - want_c)) <= 1e-15 * max(1.0, np.max(np.abs(c0[r])))
        want_h = 0.5 * np.tanh(want_c)
        assert np.max(np.abs(h[r] - want_h)) <= 1e-15


def pin_constant_input_geometric_series(fwd):
    """U = 0 and x[b, t] the same vector at every step: the pre-activation
    z = x W + b is constant per row, so the gates are constant and the cell
    update c <- f c + i g is an affine recurrence with the closed form
        c_L = f**L c0 + i g (1 - f**L) / (1 - f),   h_L = o tanh(c_L).
    z is formed with numpy's matrix product; each gate block (i, f, g, o) gets
    a different bias so a permuted gate order, a transposed W or a sign error
    changes the result."""
    B, D, H, T = 5, 4, 3, 10
    x, L, W, U, b, h0, c0 = _case(13, B, D, H, T, lo=1)
    L[:] = [10, 1, 3, 6, 8]
    x[:] = x[:, :1, :]
    U[:] = 0
    b[:] = np.concatenate([np.full(H, 0.3), np.full(H, -0.7), np.full(H, 0.45), np.full(H, -0.2)])
    b = b.astype(np.float32)
    h, c = fwd(x, L, W, U, b, h0, c0)
    z = x[:, 0, :].astype(np.float64) @ W.astype(np.float64) + b.astype(np.float64)
    sig = lambda v: 1.0 / (1.0 + np.exp(-v))
    gi, gf, gg, go = sig(z[:, :H]), sig(z[:, H:2 * H]), np.tanh(z[:, 2 * H:3 * H]), sig(z[:, 3 * H:])
    n = L.astype(np.float64)[:, None]
    fL = gf ** n
    want_c = fL * c0.astype(np.float64) + gi * gg * (1.0 - fL) / (1.0 - gf)
    want_h = go * np.tanh(want_c)
    assert np.max(np.abs(c - want_c)) <= 1e-13
    assert np.max(np.abs(h - want_h)) <= 1e-13


def pin_length_zero(fwd):
    """A row of length 0 never runs the cell: it returns (h0, c0) exactly."""
    x, L, W, U, b, h0, c0 = _case(14, 5, 6, 4, 7)
    L[:] = [0, 7, 0, 3, 0]
    h, c = fwd(x, L, W, U, b, h0, c0)
    for r in (0, 2, 4):
        assert _bits_equal(h[r], h0[r].astype(np.float64))
        assert _bits_equal(c[r], c0[r].astype(np.float64))
    assert not np.array_equal(h[1], h0[1].astype(np.float64))


def pin_all_lengths_zero(fwd):
    """All lengths 0: the loop bound is 0 and the state is returned unchanged."""
    x, L, W, U, b, h0, c0 = _case(15, 3, 4, 5, 6)
    L[:] = 0
    h, c = fwd(x, L, W, U, b, h0, c0)
    assert _bits_equal(h, h0.astype(np.float64)) and _bits_equal(c, c0.astype(np.float64))


def pin_freeze_poisoned_padding(fwd):
    """Steps at t >= L[b] must not touch row b: NaN and Inf written into
    x[b, t >= L[b]] leave every output bit unchanged (a select, not a blend)."""
    x, L, W, U, b, h0, c0 = _case(16, 6, 5, 4, 9, lo=0)
    L[:] = [9, 0, 4, 1, 7, 2]
    h1, c1 = fwd(x, L, W, U, b, h0, c0)
    xp = x.copy()
    for r in range(len(L)):
        xp[r, L[r]:, :] = np.nan
        if L[r] + 1 < x.shape[1]:
            xp[r, L[r] + 1, :] = np.inf
    h2, c2 = fwd(xp, L, W, U, b, h0, c0)
    assert _bits_equal(h1, h2) and _bits_equal(c1, c2)
    assert np.isfinite(h2).all() and np.isfinite(c2).all()


def pin_early_exit(fwd):
    """Nothing at t >= max(L) is read: poisoning x[:, max_len:] changes nothing."""
    x, L, W, U, b, h0, c0 = _case(17, 4, 3, 5, 12)
    L[:] = [3, 5, 2, 0]
    h1, c1 = fwd(x, L, W, U, b, h0, c0)
    xp = x.copy()
    xp[:, 5:, :] = np.nan
    h2, c2 = fwd(xp, L, W, U, b, h0, c0)
    assert _bits_equal(h1, h2) and _bits_equal(c1, c2)


def pin_row_equals_own_run(fwd):
    """Row b of a batch equals a batch of one holding x[b, :L[b]] alone."""
    x, L, W, U, b, h0, c0 = _case(18, 5, 6, 5, 8, lo=1)
    h, c = fwd(x, L, W, U, b, h0, c0)
    for r in range(len(L)):
        n = int(L[r])
        hr, cr = fwd(x[r:r + 1, :n], L[r:r + 1], W, U, b, h0[r:r + 1], c0[r:r + 1])
        assert _bits_equal(hr[0], h[r]) and _bits_equal(cr[0], c[r])


def pin_permutation(fwd):
    """Permuting the rows of (x, L, h0, c0) permutes the rows of the result."""
    x, L, W, U, b, h0, c0 = _case(19, 7, 4, 6, 10)
    h, c = fwd(x, L, W, U, b, h0, c0)
    p = np.random.default_rng(0).permutation(len(L))
    hp, cp = fwd(x[p], L[p], W, U, b, h0[p], c0[p])
    assert _bits_equal(hp, h[p]) and _bits_equal(cp, c[p])


def pin_chunked_resume(fwd):
    """Running steps [0, t1) and then [t1, T) from the carried state, with
    lengths min(L, t1) and max(L - t1, 0), equals the whole run."""
    x, L, W, U, b, h0, c0 = _case(20, 6, 5, 4, 11)
    h, c = fwd(x, L, W, U, b, h0, c0)
    t1 = 4
    ha, ca = fwd(x[:, :t1], np.minimum(L, t1), W, U, b, h0, c0)
    hb, cb = fwd(x[:, t1:], np.maximum(L - t1, 0), W, U, b, ha, ca)
    assert _bits_equal(hb, h) and _bits_equal(cb, c)


def pin_brute_force(fwd, seeds=range(30)):
    """Agreement (<= 1e-12) with running each sequence alone in pure Python,
    on exhaustive-random tiny shapes B <= 4, D, H <= 3, T <= 6."""
    for s in seeds:
        rng = np.random.default_rng(1000 + s)
        B, D, H, T = (int(rng.integers(1, 5)), int(rng.integers(1, 4)), int(rng.integers(1, 4)),
                      int(rng.integers(1, 7)))
        x, L, W, U, b, h0, c0 = _case(2000 + s, B, D, H, T)
        b = (np.random.default_rng(s).standard_normal(4 * H) * 0.5).astype(np.float32)
        h, c = fwd(x, L, W, U, b, h0, c0)
        hb, cb = brute.forward_per_sequence(x, L, W, U, b, h0, c0)
        assert np.max(np.abs(h - np.array(hb))) <= 1e-12, (s, B, D, H, T)
        assert np.max(np.abs(c - np.array(cb))) <= 1e-12, (s, B, D, H, T)


def pin_torch_lstm(fwd, shapes=((3, 4, 5, 6), (8, 24, 16, 12), (5, 1, 1, 9))):
    """Agreement (<= 1e-12) with torch.nn.LSTM in float64 on packed sequences.

    torch's LSTM computes the same cell with gate order (i, f, g, o) and
    weights stored transposed: weight_ih = W^T, weight_hh = U^T, bias_ih = b,
    bias_hh = 0.  Packing requires L >= 1."""
    import torch
    from torch.nn.utils.rnn import pack_padded_sequence
    for k, (B, D, H, T) in enumerate(shapes):
        x, L, W, U, b, h0, c0 = _case(3000 + k, B, D, H, T, lo=1)
        b = (np.random.default_rng(k).standard_normal(4 * H) * 0.5).astype(np.float32)
        h, c = fwd(x, L, W, U, b, h0, c0)
        m = torch.nn.LSTM(D, H, batch_first=True).double()
        with torch.no_grad():
            m.weight_ih_l0.copy_(torch.from_numpy(W.astype(np.float64).T))
            m.weight_hh_l0.copy_(torch.from_numpy(U.astype(np.float64).T))
            m.bias_ih_l0.copy_(torch.from_numpy(b.astype(np.float64)))
            m.bias_hh_l0.zero_()
            packed = pack_padded_sequence(torch.from_numpy(x.astype(np.float64)),
                                          torch.from_numpy(L.astype(np.int64)),
                                          batch_first=True, enforce_sorted=False)
            _, (hn, cn) = m(packed, (torch.from_numpy(h0.astype(np.float64))[None],
                                     torch.from_numpy(c0.astype(np.float64))[None]))
        assert np.max(np.abs(h - hn[0].numpy())) <= 1e-12, (B, D, H, T)
        assert np.max(np.abs(c - cn[0].numpy())) <= 1e-12, (B, D, H, T)


def pin_literal_equals_skip(fwd):
    """Computing every row and selecting equals skipping finished rows, bitwise."""
    x, L, W, U, b, h0, c0 = _case(21, 7, 6, 5, 10)
    h1, c1 = fwd(x, L, W, U, b, h0, c0, literal=False)
    h2, c2 = fwd(x, L, W, U, b, h0, c0, literal=True)
    assert _bits_equal(h1, h2) and _bits_equal(c1, c2)


def pin_bounds(fwd):
    """|h| <= 1 always, and |c_L| <= |c0| + L (each step adds i g with |i g| < 1
    to f c with 0 < f < 1)."""
    x, L, W, U, b, h0, c0 = _case(22, 8, 6, 7, 15)
    x *= 4.0
    h, c = fwd(x, L, W, U, b, h0, c0)
    assert np.all(np.abs(h) <= 1.0)
    assert np.all(np.abs(c) <= np.abs(c0) + L[:, None] + 1e-12)


def pin_seq_ends_and_padding(fwd):
    """The output sequence holds the final state at the last step of each
    sequence (bitwise) and zeros at every later step; a row of length 0 is all
    zeros."""
    x, L, W, U, b, h0, c0 = _case(23, 6, 4, 5, 9)
    L[:] = [9, 0, 4, 1, 6, 2]
    h, c, seq = fwd(x, L, W, U, b, h0, c0, return_seq=True)
    assert seq.shape == (6, 9, 5)
    for r in range(len(L)):
        n = int(L[r])
        if n:
            assert _bits_equal(seq[r, n - 1], h[r])
        assert np.all(seq[r, n:] == 0.0) and not np.signbit(seq[r, n:]).any()
    h2, c2 = fwd(x, L, W, U, b, h0, c0)
    assert _bits_equal(h, h2) and _bits_equal(c, c2)


def pin_seq_prefixes(fwd):
    """Step t of the output sequence equals the final hidden state of the run
    whose lengths are cut to min(L, t + 1), for every row still active at t
    (bitwise: the same steps in the same order)."""
    x, L, W, U, b, h0, c0 = _case(24, 5, 3, 4, 7)
    _, _, seq = fwd(x, L, W, U, b, h0, c0, return_seq=True)
    for t in range(x.shape[1]):
        ht, _ = fwd(x, np.minimum(L, t + 1).astype(np.int32), W, U, b, h0, c0)
        for r in range(len(L)):
            if t < L[r]:
                assert _bits_equal(seq[r, t], ht[r]), (t, r)


def pin_seq_brute_force(fwd, seeds=range(12)):
    """Agreement (<= 1e-12) of the output sequence with each sequence run
    alone in pure Python, padded with zeros past its length."""
    for s in seeds:
        rng = np.random.default_rng(4000 + s)
        B, D, H, T = (int(rng.integers(1, 5)), int(rng.integers(1, 4)), int(rng.integers(1, 4)),
                      int(rng.integers(1, 7)))
        x, L, W, U, b, h0, c0 = _case(5000 + s, B, D, H, T)
        b = (np.random.default_rng(s).standard_normal(4 * H) * 0.5).astype(np.float32)
        _, _, seq = fwd(x, L, W, U, b, h0, c0, return_seq=True)
        want = np.array(brute.sequence_per_sequence(x, L, W, U, b, h0, c0))
        assert np.max(np.abs(seq - want)) <= 1e-12, (s, B, D, H, T)


def pin_seq_torch_lstm(fwd, shapes=((3, 4, 5, 6), (6, 10, 8, 9))):
    """Agreement (<= 1e-12) with torch.nn.LSTM in float64 on packed sequences,
    unpacked with zero padding to the full extent T."""
    import torch
    from torch.nn.utils.rnn import pack_padded_sequence, pad_packed_sequence
    for k, (B, D, H, T) in enumerate(shapes):
        x, L, W, U, b, h0, c0 = _case(6000 + k, B, D, H, T, lo=1)
        b = (np.random.default_rng(k).standard_normal(4 * H) * 0.5).astype(np.float32)
        _, _, seq = fwd(x, L, W, U, b, h0, c0, return_seq=True)
        m = torch.nn.LSTM(D, H, batch_first=True).double()
        with torch.no_grad():
            m.weight_ih_l0.copy_(torch.from_numpy(W.astype(np.float64).T))
            m.weight_hh_l0.copy_(torch.from_numpy(U.astype(np.float64).T))
            m.bias_ih_l0.copy_(torch.from_numpy(b.astype(np.float64)))
            m.bias_hh_l0.zero_()
            packed = pack_padded_sequence(torch.from_numpy(x.astype(np.float64)),
                                          torch.from_numpy(L.astype(np.int64)),
                                          batch_first=True, enforce_sorted=False)
            out, _ = m(packed, (torch.from_numpy(h0.astype(np.float64))[None],
                                torch.from_numpy(c0.astype(np.float64))[None]))
            out, _ = pad_packed_sequence(out, batch_first=True, total_length=T)
        assert np.max(np.abs(seq - out.numpy())) <= 1e-12, (B, D, H, T)


PINS = [
    pin_zero_weights_closed_form,
    pin_forget_bias_closed_form,
    pin_constant_input_geometric_series,
    pin_length_zero,
    pin_all_lengths_zero,
    pin_freeze_poisoned_padding,
    pin_early_exit,
    pin_row_equals_own_run,
    pin_permutation,
    pin_chunked_resume,
    pin_brute_force,
    pin_torch_lstm,
    pin_literal_equals_skip,
    pin_bounds,
    pin_seq_ends_and_padding,
    pin_seq_prefixes,
    pin_seq_brute_force,
    pin_seq_torch_lstm,
]


# ---------------------------------------------------------------------------
# The loop with the GRU cell (gate blocks r, u, n; biases b_ih, b_hh).  Each
# pin takes a callable with the signature of ``oracle.forward_gru``.

def _gru_case(seed, B, D, H, T, lo=0):
    inp = workloads.random_case(seed, B, D, H, T, lo=lo)
    rng = np.random.default_rng(seed + 7)
    W = (rng.standard_normal((D, 3 * H)) / math.sqrt(H)).astype(np.float32)
    U = (rng.standard_normal((H, 3 * H)) / math.sqrt(H)).astype(np.float32)
    bih = (rng.standard_normal(3 * H) * 0.5).astype(np.float32)
    bhh = (rng.standard_normal(3 * H) * 0.5).astype(np.float32)
    return inp.x.copy(), inp.lengths.copy(), W, U, bih, bhh, inp.h0.copy()


def gpin_zero_weights_closed_form(fwd):
    """W = U = 0 and zero biases: r = u = 1/2 and n = tanh(0) = 0, so each
    step halves h: h_L = 2**-L h0, exactly."""
    x, L, W, U, bih, bhh, h0 = _gru_case(40, 5, 4, 6, 8)
    L[:] = [0, 1, 3, 8, 5]
    W[:] = 0
    U[:] = 0
    bih[:] = 0
    bhh[:] = 0
    h = fwd(x, L, W, U, bih, bhh, h0)
    assert _bits_equal(h, np.ldexp(h0.astype(np.float64), -L[:, None]))


def gpin_constant_input_closed_form(fwd):
    """U = 0 and x[b, t] constant per row: r, u and n are constant per row
    (n = tanh(x W_n + b_in + r b_hn)), so h' = (1 - u) n + u h is affine with
    h_L = u**L h0 + n (1 - u**L).  Every gate block and both biases of every
    block take different values, so a swapped block, a reset gate applied to
    the input part, or a misplaced bias changes the result."""
    x, L, W, U, bih, bhh, h0 = _gru_case(41, 5, 3, 4, 9, lo=1)
    L[:] = [9, 1, 4, 6, 2]
    x[:] = x[:, :1, :]
    U[:] = 0
    H = 4
    bih[:] = np.concatenate([np.full(H, 0.4), np.full(H, -0.3), np.full(H, 0.25)]).astype(np.float32)
    bhh[:] = np.concatenate([np.full(H, -0.1), np.full(H, 0.6), np.full(H, -0.8)]).astype(np.float32)
    h = fwd(x, L, W, U, bih, bhh, h0)
    zx = x[:, 0, :].astype(np.float64) @ W.astype(np.float64) + bih.astype(np.float64)
    zh = np.broadcast_to(bhh.astype(np.float64), zx.shape)
    sig = lambda v: 1.0 / (1.0 + np.exp(-v))
    r = sig(zx[:, :H] + zh[:, :H])
    u = sig(zx[:, H:2 * H] + zh[:, H:2 * H])
    n = np.tanh(zx[:, 2 * H:] + r * zh[:, 2 * H:])
    uL = u ** L.astype(np.float64)[:, None]
    want = uL * h0.astype(np.float64) + n * (1.0 - uL)
    assert np.max(np.abs(h - want)) <= 1e-13


def gpin_length_zero_and_poisoned_padding(fwd):
    """A row of length 0 keeps h0 exactly, and NaN/Inf in x past each length
    changes no bit of the result or of the output sequence."""
    x, L, W, U, bih, bhh, h0 = _gru_case(42, 6, 5, 4, 9)
    L[:] = [9, 0, 4, 1, 7, 0]
    h1, s1 = fwd(x, L, W, U, bih, bhh, h0, return_seq=True)
    for r in (1, 5):
        assert _bits_equal(h1[r], h0[r].astype(np.float64))
    xp = x.copy()
    for r in range(len(L)):
        xp[r, L[r]:, :] = np.nan
        if L[r] + 1 < x.shape[1]:
            xp[r, L[r] + 1, :] = np.inf
    h2, s2 = fwd(xp, L, W, U, bih, bhh, h0, return_seq=True)
    assert _bits_equal(h1, h2) and _bits_equal(s1, s2)


def gpin_row_equals_own_run(fwd):
    """Each row of a batch equals a batch of one holding that row alone."""
    x, L, W, U, bih, bhh, h0 = _gru_case(43, 5, 4, 5, 7, lo=1)
    h = fwd(x, L, W, U, bih, bhh, h0)
    for r in range(len(L)):
        hr = fwd(x[r:r + 1, :int(L[r])], L[r:r + 1], W, U, bih, bhh, h0[r:r + 1])
        assert _bits_equal(hr[0], h[r])


def gpin_brute_force(fwd, seeds=range(20)):
    """Agreement (<= 1e-12) of h and of the output sequence with each sequence
    run alone in pure Python."""
    for s in seeds:
        rng = np.random.default_rng(7000 + s)
        B, D, H, T = (int(rng.integers(1, 5)), int(rng.integers(1, 4)), int(rng.integers(1, 4)),
                      int(rng.integers(1, 7)))
        x, L, W, U, bih, bhh, h0 = _gru_case(8000 + s, B, D, H, T)
        h, seq = fwd(x, L, W, U, bih, bhh, h0, return_seq=True)
        hb, sb = brute.gru_per_sequence(x, L, W.tolist(), U.tolist(), bih.tolist(), bhh.tolist(),
                                        h0.tolist())
        assert np.max(np.abs(h - np.array(hb))) <= 1e-12, (s, B, D, H, T)
        assert np.max(np.abs(seq - np.array(sb))) <= 1e-12, (s, B, D, H, T)


def gpin_torch_gru(fwd, shapes=((3, 4, 5, 6), (7, 12, 9, 10))):
    """Agreement (<= 1e-12) with torch.nn.GRU in float64 on packed sequences:
    torch's gate order is (r, z, n) with z the update gate, weight_ih = W^T,
    weight_hh = U^T, bias_ih = b_ih, bias_hh = b_hh; the output sequence is
    unpacked with zero padding."""
    import torch
    from torch.nn.utils.rnn import pack_padded_sequence, pad_packed_sequence
    for k, (B, D, H, T) in enumerate(shapes):
        x, L, W, U, bih, bhh, h0 = _gru_case(9000 + k, B, D, H, T, lo=1)
        h, seq = fwd(x, L, W, U, bih, bhh, h0, return_seq=True)
        m = torch.nn.GRU(D, H, batch_first=True).double()
        with torch.no_grad():
            m.weight_ih_l0.copy_(torch.from_numpy(W.astype(np.float64).T))
            m.weight_hh_l0.copy_(torch.from_numpy(U.astype(np.float64).T))
            m.bias_ih_l0.copy_(torch.from_numpy(bih.astype(np.float64)))
            m.bias_hh_l0.copy_(torch.from_numpy(bhh.astype(np.float64)))
            packed = pack_padded_sequence(torch.from_numpy(x.astype(np.float64)),
                                          torch.from_numpy(L.astype(np.int64)),
                                          batch_first=True, enforce_sorted=False)
            out, hn = m(packed, torch.from_numpy(h0.astype(np.float64))[None])
            out, _ = pad_packed_sequence(out, batch_first=True, total_length=T)
        assert np.max(np.abs(h - hn[0].numpy())) <= 1e-12, (B, D, H, T)
        assert np.max(np.abs(seq - out.numpy())) <= 1e-12, (B, D, H, T)


GRU_PINS = [
    gpin_zero_weights_closed_form,
    gpin_constant_input_closed_form,
    gpin_length_zero_and_poisoned_padding,
    gpin_row_equals_own_run,
    gpin_brute_force,
    gpin_torch_gru,
]


# ---------------------------------------------------------------------------
# The loop with the tanh RNN cell h' = tanh(x W + h U + b).  Each pin takes a
# callable with the signature of ``oracle.forward_rnn``.

def _rnn_case(seed, B, D, H, T, lo=0):
    inp = workloads.random_case(seed, B, D, H, T, lo=lo)
    rng = np.random.default_rng(seed + 11)
    W = (rng.standard_normal((D, H)) / math.sqrt(H)).astype(np.float32)
    U = (rng.standard_normal((H, H)) / math.sqrt(H)).astype(np.float32)
    b = (rng.standard_normal(H) * 0.5).astype(np.float32)
    return inp.x.copy(), inp.lengths.copy(), W, U, b, inp.h0.copy()


def rpin_no_recurrence_closed_form(fwd):
    """U = 0: each step's output depends on its own input only,
    out[b, t] = tanh(x[b, t] W + b) for t < L[b] and zero after, and the final
    state is the last of them (h0 for length 0).  Pins W's orientation, the
    bias, the non-linearity, the time index and the padding."""
    x, L, W, U, b, h0 = _rnn_case(60, 5, 4, 6, 8)
    L[:] = [0, 1, 3, 8, 5]
    U[:] = 0
    h, seq = fwd(x, L, W, U, b, h0, return_seq=True)
    want = np.tanh(x.astype(np.float64) @ W.astype(np.float64) + b.astype(np.float64))
    t = np.arange(x.shape[1])[None, :, None]
    want = np.where(t < L[:, None, None], want, 0.0)
    assert np.max(np.abs(seq - want)) <= 1e-15
    for r in range(len(L)):
        last = want[r, L[r] - 1] if L[r] > 0 else h0[r].astype(np.float64)
        assert np.max(np.abs(h[r] - last)) <= 1e-15


def rpin_one_hot_state_reads_a_row_of_U(fwd):
    """W = 0, b = 0 and h0 = e_k: one step gives tanh(e_k U) = tanh(U[k, :]),
    the k-th ROW of U (a transposed U gives its column instead)."""
    x, L, W, U, b, h0 = _rnn_case(61, 5, 3, 5, 4)
    L[:] = 1
    W[:] = 0
    b[:] = 0
    h0[:] = 0
    for r in range(5):
        h0[r, r] = 1.0
    h = fwd(x, L, W, U, b, h0)
    want = np.array([[math.tanh(float(u)) for u in row] for row in U])  # libm's tanh, as the C
    assert _bits_equal(h, want)


def rpin_diagonal_recurrence(fwd):
    """W = 0, b = 0, U = diag(a): every unit follows its own scalar map
    h <- tanh(a_v h), iterated L[b] times in plain Python."""
    x, L, W, U, b, h0 = _rnn_case(62, 4, 3, 5, 9, lo=0)
    L[:] = [9, 0, 4, 7]
    W[:] = 0
    b[:] = 0
    a = np.array([1.5, -0.7, 0.3, 2.0, -1.2], np.float32)
    U[:] = np.diag(a)
    h = fwd(x, L, W, U, b, h0)
    for r in range(4):
        for v in range(5):
            s = float(h0[r, v])
            for _ in range(int(L[r])):
                s = math.tanh(float(a[v]) * s)
            assert h[r, v] == s, (r, v)


def rpin_length_zero_and_poisoned_padding(fwd):
    """A row of length 0 keeps h0 exactly, and NaN/Inf in x past each length
    changes no bit of the result or of the output sequence."""
    x, L, W, U, b, h0 = _rnn_case(63, 6, 5, 4, 9)
    L[:] = [9, 0, 4, 1, 7, 0]
    h1, s1 = fwd(x, L, W, U, b, h0, return_seq=True)
    for r in (1, 5):
        assert _bits_equal(h1[r], h0[r].astype(np.float64))
    xp = x.copy()
    for r in range(len(L)):
        xp[r, L[r]:, :] = np.nan
        if L[r] + 1 < x.shape[1]:
            xp[r, L[r] + 1, :] = np.inf
    h2, s2 = fwd(xp, L, W, U, b, h0, return_seq=True)
    assert _bits_equal(h1, h2) and _bits_equal(s1, s2)


def rpin_brute_force(fwd, seeds=range(20)):
    """Agreement (<= 1e-12) of h and of the output sequence with each sequence
    run alone in pure Python."""
    for s in seeds:
        rng = np.random.default_rng(7100 + s)
        B, D, H, T = (int(rng.integers(1, 5)), int(rng.integers(1, 4)), int(rng.integers(1, 5)),
                      int(rng.integers(1, 7)))
        x, L, W, U, b, h0 = _rnn_case(8100 + s, B, D, H, T)
        h, seq = fwd(x, L, W, U, b, h0, return_seq=True)
        hb, sb = brute.rnn_per_sequence(x, L, W.tolist(), U.tolist(), b.tolist(), h0.tolist())
        assert np.max(np.abs(h - np.array(hb))) <= 1e-12, (s, B, D, H, T)
        assert np.max(np.abs(seq - np.array(sb))) <= 1e-12, (s, B, D, H, T)


def rpin_torch_rnn(fwd, shapes=((3, 4, 5, 6), (7, 12, 9, 10))):
    """Agreement (<= 1e-12) with torch.nn.RNN (tanh) in float64 on packed
    sequences: weight_ih = W^T, weight_hh = U^T, bias_ih = b, bias_hh = 0;
    the output sequence is unpacked with zero padding."""
    import torch
    from torch.nn.utils.rnn import pack_padded_sequence, pad_packed_sequence
    for k, (B, D, H, T) in enumerate(shapes):
        x, L, W, U, b, h0 = _rnn_case(9100 + k, B, D, H, T, lo=1)
        h, seq = fwd(x, L, W, U, b, h0, return_seq=True)
        m = torch.nn.RNN(D, H, nonlinearity="tanh", batch_first=True).double()
        with torch.no_grad():
            m.weight_ih_l0.copy_(torch.from_numpy(W.astype(np.float64).T))
            m.weight_hh_l0.copy_(torch.from_numpy(U.astype(np.float64).T))
            m.bias_ih_l0.copy_(torch.from_numpy(b.astype(np.float64)))
            m.bias_hh_l0.zero_()
            packed = pack_padded_sequence(torch.from_numpy(x.astype(np.float64)),
                                          torch.from_numpy(L.astype(np.int64)),
                                          batch_first=True, enforce_sorted=False)
            out, hn = m(packed, torch.from_numpy(h0.astype(np.float64))[None])
            out, _ = pad_packed_sequence(out, batch_first=True, total_length=T)
        assert np.max(np.abs(h - hn[0].numpy())) <= 1e-12, (B, D, H, T)
        assert np.max(np.abs(seq - out.numpy())) <= 1e-12, (B, D, H, T)


RNN_PINS = [
    rpin_no_recurrence_closed_form,
    rpin_one_hot_state_reads_a_row_of_U,
    rpin_diagonal_recurrence,
    rpin_length_zero_and_poisoned_padding,
    rpin_brute_force,
    rpin_torch_rnn,
]


# ---------------------------------------------------------------------------
# The loop with termination computed from the state (halting score
# v . h + c_stop > 0 after a step ends a row; lengths are caps).  Each pin
# takes a callable with the signature of ``oracle.forward_stop``.

def _stop_case(seed, B, D, H, T, lo=0):
    inp = workloads.random_case(seed, B, D, H, T, lo=lo)
    x, W, U = inp.as_f32()
    return x.copy(), inp.lengths.copy(), W, U, inp.b.copy(), inp.h0.copy(), inp.c0.copy()


def spin_never_stopping_equals_plain_loop(fwd):
    """v = 0, c_stop < 0 (and c_stop = 0: the score must be positive): no row
    ever terminates, so the result is the plain masked loop's bit for bit,
    every row runs to its cap and the loop runs max(L) iterations."""
    x, L, W, U, b, h0, c0 = _stop_case(70, 6, 5, 7, 9)
    h, c, steps, iters = fwd(x, L, W, U, b, h0, c0, np.zeros(7, np.float32), -1.0)
    hp, cp = oracle.forward(x, L, W, U, b, h0, c0)
    assert _bits_equal(h, hp) and _bits_equal(c, cp)
    assert np.array_equal(steps, L) and iters == int(L.max())
    # a score of exactly zero does not end a row (the rule is score > 0)
    h0s, _, steps0, _ = fwd(x, L, W, U, b, h0, c0, np.zeros(7, np.float32), 0.0)
    assert np.array_equal(steps0, L) and _bits_equal(h0s, hp)


def spin_always_stopping_runs_one_step(fwd):
    """v = 0, c_stop > 0: every row terminates after its first step: steps =
    min(L, 1), the state is the plain loop's with lengths min(L, 1), and the
    loop runs one iteration (none if every cap is 0)."""
    x, L, W, U, b, h0, c0 = _stop_case(71, 6, 5, 7, 9)
    L[2] = 0
    h, c, steps, iters = fwd(x, L, W, U, b, h0, c0, np.zeros(7, np.float32), 0.5)
    L1 = np.minimum(L, 1)
    hp, cp = oracle.forward(x, L1, W, U, b, h0, c0)
    assert _bits_equal(h, hp) and _bits_equal(c, cp)
    assert np.array_equal(steps, L1) and iters == 1
    _, _, steps0, iters0 = fwd(x, np.zeros_like(L), W, U, b, h0, c0, np.zeros(7, np.float32), 0.5)
    assert iters0 == 0 and not steps0.any()


def spin_zero_weights_stopping_step(fwd):
    """W = U = 0, b = 0: every gate is 1/2, so c_t = 2^-t c0 and h_t = tanh(c_t)/2
    exactly.  With v = -e_0 and c_stop = thr a row terminates after the first
    step t >= 1 with tanh(2^-t c0[0])/2 < thr; the step is found by a plain
    Python loop over t and thresholds sit between consecutive values (no ties)."""
    x, L, W, U, b, h0, c0 = _stop_case(72, 5, 3, 4, 12)
    W[:] = 0
    U[:] = 0
    b[:] = 0
    L[:] = [12, 12, 3, 12, 0]
    c0[:, 0] = [6.0, 3.0, 6.0, -2.0, 5.0]
    v = np.zeros(4, np.float32)
    v[0] = -1.0
    thr = 0.5 * (0.5 * math.tanh(6.0 / 2 ** 4) + 0.5 * math.tanh(6.0 / 2 ** 5))  # between t = 4 and 5
    h, c, steps, iters = fwd(x, L, W, U, b, h0, c0, v, thr)
    want = []
    for r in range(5):
        n = 0
        for t in range(1, int(L[r]) + 1):
            n = t
            if -0.5 * math.tanh(float(c0[r, 0]) / 2 ** t) + thr > 0:
                break
        want.append(n)
    assert steps.tolist() == want, (steps.tolist(), want)
    assert want[0] == 5 and want[2] == 3 and want[3] == 1 and want[4] == 0
    assert iters == max(want)
    for r in range(5):
        assert _bits_equal(c[r], np.ldexp(c0[r].astype(np.float64), -want[r]))


def spin_consistent_with_plain_loop_trace(fwd):
    """A random read-out that ends most rows early: (1) the state equals the
    plain loop run with lengths = steps, bit for bit; (2) along the plain loop's
    output sequence (caps as lengths) the halting score is <= 0 after every
    step before a row's last and > 0 after its last unless it reached its cap;
    (3) the loop ran max(steps) iterations."""
    x, L, W, U, b, h0, c0 = _stop_case(73, 12, 6, 10, 16, lo=8)
    rng = np.random.default_rng(74)
    v = rng.standard_normal(10).astype(np.float32)
    h, c, steps, iters = fwd(x, L, W, U, b, h0, c0, v, -0.6)
    assert (steps < L).sum() >= 4                        # the read-out does end rows early
    hp, cp = oracle.forward(x, steps, W, U, b, h0, c0)
    assert _bits_equal(h, hp) and _bits_equal(c, cp)
    _, _, seq = oracle.forward(x, L, W, U, b, h0, c0, return_seq=True)
    score = seq @ v.astype(np.float64) - 0.6            # [B, T]
    for r in range(len(L)):
        n = int(steps[r])
        assert np.all(score[r, :n - 1] <= 1e-12), r
        if n < L[r]:
            assert n >= 1 and score[r, n - 1] > -1e-12, r
    assert iters == int(steps.max())


def spin_brute_force(fwd, seeds=range(12)):
    """Agreement with each sequence run alone in pure Python under the same
    stopping rule, for the three cells: steps exactly, states <= 1e-12."""
    for s in seeds:
        rng = np.random.default_rng(7300 + s)
        B, D, H, T = (int(rng.integers(1, 5)), int(rng.integers(1, 4)), int(rng.integers(1, 4)),
                      int(rng.integers(1, 8)))
        cell = ("lstm", "gru", "rnn")[s % 3]
        g = {"lstm": 4, "gru": 3, "rnn": 1}[cell]
        x, L, _, _, _, h0, c0 = _stop_case(8300 + s, B, D, H, T)
        W = (rng.standard_normal((D, g * H)) / math.sqrt(H)).astype(np.float32)
        U = (rng.standard_normal((H, g * H)) / math.sqrt(H)).astype(np.float32)
        b = (rng.standard_normal(g * H) * 0.5).astype(np.float32)
        bhh = (rng.standard_normal(3 * H) * 0.5).astype(np.float32) if cell == "gru" else None
        if cell != "lstm":
            c0 = np.zeros_like(c0)
        v = rng.standard_normal(H).astype(np.float32)
        cs = float(rng.standard_normal() * 0.3)
        h, c, steps, iters = fwd(x, L, W, U, b, h0, c0, v, cs, cell=cell, b_hh=bhh)
        hb, cb, sb = brute.stop_per_sequence(x, L, W, U, b, h0, c0, v, cs, cell=cell, b_hh=bhh)
        assert steps.tolist() == sb, (s, cell, steps.tolist(), sb)
        assert np.max(np.abs(h - np.array(hb))) <= 1e-12, (s, cell)
        assert np.max(np.abs(c - np.array(cb))) <= 1e-12, (s, cell)
        assert iters == (max(sb) if sb else 0)


def spin_other_cells_match_their_plain_loops(fwd):
    """GRU and RNN under the stopping rule equal their plain loops run with
    lengths = steps, bit for bit, and their output sequences agree on the
    steps run (zero after)."""
    for cell in ("gru", "rnn"):
        inp = workloads.random_cell_case(cell, 75, 8, 5, 9, 12, lo=6)
        x, W, U = inp.as_f32()
        rng = np.random.default_rng(76)
        v = rng.standard_normal(9).astype(np.float32)
        c0 = np.zeros_like(inp.h0)
        bias = inp.b_ih if cell == "gru" else inp.b
        h, c, steps, iters, seq = fwd(x, inp.lengths, W, U, bias, inp.h0, c0, v, -0.3, cell=cell,
                                      b_hh=inp.b_hh if cell == "gru" else None, return_seq=True)
        assert (steps < inp.lengths).any(), cell
        if cell == "gru":
            hp, sp = oracle.forward_gru(x, steps, W, U, inp.b_ih, inp.b_hh, inp.h0, return_seq=True)
        else:
            hp, sp = oracle.forward_rnn(x, steps, W, U, inp.b, inp.h0, return_seq=True)
        assert _bits_equal(h, hp) and _bits_equal(seq, sp), cell


STOP_PINS = [
    spin_never_stopping_equals_plain_loop,
    spin_always_stopping_runs_one_step,
    spin_zero_weights_stopping_step,
    spin_consistent_with_plain_loop_trace,
    spin_brute_force,
    spin_other_cells_match_their_plain_loops,
]


# ---------------------------------------------------------------------------
# The backward pass of the masked LSTM loop.  Each pin takes a callable with
# the signature of ``oracle.backward``.  The loss whose gradients these are is
#   loss = sum(dh_out * h_final) + sum(dc_out * c_final) + sum(dseq * seq)
# with seq the output sequence (zero past each length).

def _bwd_case(seed, B, D, H, T, lo=0):
    x, L, W, U, b, h0, c0 = _stop_case(seed, B, D, H, T, lo=lo)
    rng = np.random.default_rng(seed + 13)
    b = (b + rng.standard_normal(b.shape) * 0.3).astype(np.float32)   # every gate's bias non-zero
    dh = rng.standard_normal((B, H))
    dc = rng.standard_normal((B, H))
    ds = rng.standard_normal((B, T, H))
    return x, L, W, U, b, h0.astype(np.float64), c0.astype(np.float64), dh, dc, ds


def _loss(x, L, W, U, b, h0, c0, dh, dc, ds):
    h, c, seq = oracle.forward(x, L, W, U, b, h0, c0, return_seq=True)
    return float(np.sum(dh * h) + np.sum(dc * c) + np.sum(ds * seq))


def bpin_finite_differences(bwd):
    """Central differences of the loss, entry by entry, for x (valid steps and
    padding), W, U, b, h0 and c0.  x, W, U, b are fp32, so each is moved to
    the neighbouring fp32 values v(1 +- 2^-10) and the difference quotient
    uses the exact distance between them; agreement to 2e-6 relative."""
    x, L, W, U, b, h0, c0, dh, dc, ds = _bwd_case(90, 3, 2, 3, 4)
    L[:] = [4, 2, 0]
    g = bwd(x, L, W, U, b, h0, c0, dh, dc, ds)

    def check(name, arr, grad, f32):
        flat = arr.reshape(-1)
        for i in range(flat.size):
            v = float(flat[i])
            if f32:
                step = max(abs(v), 0.05) * 2.0 ** -10
                vp, vm = np.float32(v + step), np.float32(v - step)
            else:
                step = max(abs(v), 0.05) * 1e-5
                vp, vm = v + step, v - step
            flat[i] = vp
            lp = _loss(x, L, W, U, b, h0, c0, dh, dc, ds)
            flat[i] = vm
            lm = _loss(x, L, W, U, b, h0, c0, dh, dc, ds)
            flat[i] = v
            fd = (lp - lm) / (float(vp) - float(vm))
            gi = float(grad.reshape(-1)[i])
            assert abs(fd - gi) <= 2e-6 * max(1.0, abs(gi)), (name, i, fd, gi)

    check("x", x, g["dx"], True)
    check("W", W, g["dW"], True)
    check("U", U, g["dU"], True)
    check("b", b, g["db"], True)
    check("h0", h0, g["dh0"], False)
    check("c0", c0, g["dc0"], False)


def bpin_torch_autograd(bwd, shapes=((3, 4, 5, 6), (7, 12, 9, 10))):
    """Agreement (<= 1e-11) with torch.nn.LSTM's autograd in float64 on packed
    sequences (weight_ih = W^T, weight_hh = U^T, bias_ih = b, bias_hh = 0),
    for the same loss: the gradients of the weights (dW = weight_ih.grad^T
    etc., db = bias_ih.grad), of the padded input, of h0 and of c0."""
    import torch
    from torch.nn.utils.rnn import pack_padded_sequence, pad_packed_sequence
    for k, (B, D, H, T) in enumerate(shapes):
        x, L, W, U, b, h0, c0, dh, dc, ds = _bwd_case(9200 + k, B, D, H, T, lo=1)
        g = bwd(x, L, W, U, b, h0, c0, dh, dc, ds)
        m = torch.nn.LSTM(D, H, batch_first=True).double()
        with torch.no_grad():
            m.weight_ih_l0.copy_(torch.from_numpy(W.astype(np.float64).T))
            m.weight_hh_l0.copy_(torch.from_numpy(U.astype(np.float64).T))
            m.bias_ih_l0.copy_(torch.from_numpy(b.astype(np.float64)))
            m.bias_hh_l0.zero_()
        xt = torch.from_numpy(x.astype(np.float64)).requires_grad_()
        h0t = torch.from_numpy(h0).requires_grad_()
        c0t = torch.from_numpy(c0).requires_grad_()
        packed = pack_padded_sequence(xt, torch.from_numpy(L.astype(np.int64)), batch_first=True,
                                      enforce_sorted=False)
        out, (hn, cn) = m(packed, (h0t[None], c0t[None]))
        out, _ = pad_packed_sequence(out, batch_first=True, total_length=T)
        loss = (torch.from_numpy(dh) * hn[0]).sum() + (torch.from_numpy(dc) * cn[0]).sum() + \
               (torch.from_numpy(ds) * out).sum()
        loss.backward()
        pairs = [("dW", m.weight_ih_l0.grad.T), ("dU", m.weight_hh_l0.grad.T),
                 ("db", m.bias_ih_l0.grad), ("dx", xt.grad), ("dh0", h0t.grad), ("dc0", c0t.grad)]
        for name, ref in pairs:
            err = np.max(np.abs(g[name] - ref.numpy()))
            assert err <= 1e-11 * max(1.0, float(np.max(np.abs(ref.numpy())))), (k, name, err)


def bpin_masking_facts(bwd):
    """Padding gets no gradient (dx = 0 exactly at t >= L[b]); a row of length
    0 passes its upstream gradients to (dh0, dc0) bit for bit and adds nothing
    to the weight gradients; dseq past a length has no effect."""
    x, L, W, U, b, h0, c0, dh, dc, ds = _bwd_case(91, 5, 3, 4, 7)
    L[:] = [7, 0, 3, 5, 0]
    g = bwd(x, L, W, U, b, h0, c0, dh, dc, ds)
    for r in range(5):
        assert not np.any(g["dx"][r, L[r]:]), r
    for r in (1, 4):
        assert _bits_equal(g["dh0"][r], dh[r]) and _bits_equal(g["dc0"][r], dc[r])
    ds2 = ds.copy()
    for r in range(5):
        ds2[r, L[r]:] = 1e3
    g2 = bwd(x, L, W, U, b, h0, c0, dh, dc, ds2)
    assert all(_bits_equal(g[k], g2[k]) for k in g)
    keep = [0, 2, 3]                              # the rows of length 0 contribute nothing
    g3 = bwd(x[keep], L[keep], W, U, b, h0[keep], c0[keep], dh[keep], dc[keep], ds[keep])
    for k in ("dW", "dU", "db"):
        assert np.max(np.abs(g[k] - g3[k])) <= 1e-13 * max(1.0, np.max(np.abs(g[k]))), k


def bpin_linear_in_upstream(bwd):
    """The gradients are linear in the upstream gradients:
    grad(a g1 + g2) = a grad(g1) + grad(g2)."""
    x, L, W, U, b, h0, c0, dh, dc, ds = _bwd_case(92, 4, 3, 5, 6)
    rng = np.random.default_rng(93)
    dh2, dc2, ds2 = rng.standard_normal(dh.shape), rng.standard_normal(dc.shape), rng.standard_normal(ds.shape)
    a = -1.75
    g1 = bwd(x, L, W, U, b, h0, c0, dh, dc, ds)
    g2 = bwd(x, L, W, U, b, h0, c0, dh2, dc2, ds2)
    g = bwd(x, L, W, U, b, h0, c0, a * dh + dh2, a * dc + dc2, a * ds + ds2)
    for k in g:
        ref = a * g1[k] + g2[k]
        assert np.max(np.abs(g[k] - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref))), k


def bpin_rows_add_up(bwd):
    """The weight gradients of a batch are the sums of its rows' gradients,
    and each row's (dx, dh0, dc0) is the batch-of-one result."""
    x, L, W, U, b, h0, c0, dh, dc, ds = _bwd_case(94, 4, 3, 4, 6, lo=1)
    g = bwd(x, L, W, U, b, h0, c0, dh, dc, ds)
    acc = {k: 0.0 for k in ("dW", "dU", "db")}
    for r in range(4):
        s = slice(r, r + 1)
        gr = bwd(x[s], L[s], W, U, b, h0[s], c0[s], dh[s], dc[s], ds[s])
        for k in acc:
            acc[k] = acc[k] + gr[k]
        for k in ("dx", "dh0", "dc0"):
            assert _bits_equal(gr[k][0], g[k][r]), (k, r)
    for k in acc:
        assert np.max(np.abs(g[k] - acc[k])) <= 1e-13 * max(1.0, np.max(np.abs(acc[k]))), k


BWD_PINS = [
    bpin_finite_differences,
    bpin_torch_autograd,
    bpin_masking_facts,
    bpin_linear_in_upstream,
    bpin_rows_add_up,
]


# ---------------------------------------------------------------------------
# The backward pass with the GRU and tanh RNN cells.  Each pin takes a
# callable bwd(cell, x, L, W, U, b, b_hh, h0, dh, ds) returning the gradient
# dict of ``oracle.backward_gru`` / ``oracle.backward_rnn``.

def _cell_bwd_case(cell, seed, B, D, H, T, lo=0):
    x, L, _, _, _, h0, _ = _stop_case(seed, B, D, H, T, lo=lo)
    rng = np.random.default_rng(seed + 17)
    g = 3 if cell == "gru" else 1
    W = (rng.standard_normal((D, g * H)) / math.sqrt(H)).astype(np.float32)
    U = (rng.standard_normal((H, g * H)) / math.sqrt(H)).astype(np.float32)
    b = (rng.standard_normal(g * H) * 0.4).astype(np.float32)
    bhh = (rng.standard_normal(g * H) * 0.4).astype(np.float32) if cell == "gru" else None
    dh = rng.standard_normal((B, H))
    ds = rng.standard_normal((B, T, H))
    return x, L, W, U, b, bhh, h0.astype(np.float64), dh, ds


def _cell_loss(cell, x, L, W, U, b, bhh, h0, dh, ds):
    if cell == "gru":
        h, seq = oracle.forward_gru(x, L, W, U, b, bhh, h0, return_seq=True)
    else:
        h, seq = oracle.forward_rnn(x, L, W, U, b, h0, return_seq=True)
    return float(np.sum(dh * h) + np.sum(ds * seq))


def cbpin_finite_differences(bwd):
    """Central differences of the loss entry by entry (x, W, U, both biases,
    h0), for both cells; fp32 parameters moved to neighbouring fp32 values and
    divided by their exact distance; agreement to 2e-6 relative."""
    for cell in ("gru", "rnn"):
        x, L, W, U, b, bhh, h0, dh, ds = _cell_bwd_case(cell, 95, 3, 2, 3, 4)
        L[:] = [4, 2, 0]
        g = bwd(cell, x, L, W, U, b, bhh, h0, dh, ds)
        names = [("x", x, "dx", True), ("W", W, "dW", True), ("U", U, "dU", True),
                 ("h0", h0, "dh0", False)]
        names += [("b_ih", b, "db_ih", True), ("b_hh", bhh, "db_hh", True)] if cell == "gru" else \
                 [("b", b, "db", True)]
        for name, arr, key, f32 in names:
            flat = arr.reshape(-1)
            for i in range(flat.size):
                v = float(flat[i])
                if f32:
                    step = max(abs(v), 0.05) * 2.0 ** -10
                    vp, vm = np.float32(v + step), np.float32(v - step)
                else:
                    step = max(abs(v), 0.05) * 1e-5
                    vp, vm = v + step, v - step
                flat[i] = vp
                lp = _cell_loss(cell, x, L, W, U, b, bhh, h0, dh, ds)
                flat[i] = vm
                lm = _cell_loss(cell, x, L, W, U, b, bhh, h0, dh, ds)
                flat[i] = v
                fd = (lp - lm) / (float(vp) - float(vm))
                gi = float(g[key].reshape(-1)[i])
                assert abs(fd - gi) <= 2e-6 * max(1.0, abs(gi)), (cell, name, i, fd, gi)


def cbpin_torch_autograd(bwd, shapes=((3, 4, 5, 6), (7, 12, 9, 10))):
    """Agreement (<= 1e-11) with torch.nn.GRU / torch.nn.RNN (tanh) autograd in
    float64 on packed sequences, for the same loss (the RNN's bias_hh fixed at
    zero, its bias_ih = b)."""
    import torch
    from torch.nn.utils.rnn import pack_padded_sequence, pad_packed_sequence
    for cell in ("gru", "rnn"):
        for k, (B, D, H, T) in enumerate(shapes):
            x, L, W, U, b, bhh, h0, dh, ds = _cell_bwd_case(cell, 9300 + k, B, D, H, T, lo=1)
            g = bwd(cell, x, L, W, U, b, bhh, h0, dh, ds)
            m = (torch.nn.GRU(D, H, batch_first=True) if cell == "gru" else
                 torch.nn.RNN(D, H, nonlinearity="tanh", batch_first=True)).double()
            with torch.no_grad():
                m.weight_ih_l0.copy_(torch.from_numpy(W.astype(np.float64).T))
                m.weight_hh_l0.copy_(torch.from_numpy(U.astype(np.float64).T))
                m.bias_ih_l0.copy_(torch.from_numpy(b.astype(np.float64)))
                if cell == "gru":
                    m.bias_hh_l0.copy_(torch.from_numpy(bhh.astype(np.float64)))
                else:
                    m.bias_hh_l0.zero_()
            xt = torch.from_numpy(x.astype(np.float64)).requires_grad_()
            h0t = torch.from_numpy(h0).requires_grad_()
            packed = pack_padded_sequence(xt, torch.from_numpy(L.astype(np.int64)), batch_first=True,
                                          enforce_sorted=False)
            out, hn = m(packed, h0t[None])
            out, _ = pad_packed_sequence(out, batch_first=True, total_length=T)
            loss = (torch.from_numpy(dh) * hn[0]).sum() + (torch.from_numpy(ds) * out).sum()
            loss.backward()
            pairs = [("dW", m.weight_ih_l0.grad.T), ("dU", m.weight_hh_l0.grad.T),
                     ("dx", xt.grad), ("dh0", h0t.grad)]
            if cell == "gru":
                pairs += [("db_ih", m.bias_ih_l0.grad), ("db_hh", m.bias_hh_l0.grad)]
            else:
                pairs += [("db", m.bias_ih_l0.grad)]
            for name, ref in pairs:
                err = np.max(np.abs(g[name] - ref.numpy()))
                assert err <= 1e-11 * max(1.0, float(np.max(np.abs(ref.numpy())))), (cell, k, name, err)


def cbpin_masking_facts(bwd):
    """No gradient on padding; a length-0 row passes dh to dh0 bit for bit."""
    for cell in ("gru", "rnn"):
        x, L, W, U, b, bhh, h0, dh, ds = _cell_bwd_case(cell, 96, 5, 3, 4, 7)
        L[:] = [7, 0, 3, 5, 0]
        g = bwd(cell, x, L, W, U, b, bhh, h0, dh, ds)
        for r in range(5):
            assert not np.any(g["dx"][r, L[r]:]), (cell, r)
        for r in (1, 4):
            assert _bits_equal(g["dh0"][r], dh[r]), (cell, r)


CELL_BWD_PINS = [
    cbpin_finite_differences,
    cbpin_torch_autograd,
    cbpin_masking_facts,
]
