"""Brute-force cross-check of the oracle for tiny cases (pure Python, ``math``).

TEST INFRASTRUCTURE ONLY.  It runs every sequence on its own, for exactly its
own number of steps (Section 9 "RNN cells": a sequence's state stops changing
once its length is reached), with no batch, no mask, no select and no loop
bound shared across rows.  It shares no code with ``lstm_oracle.c``; the cell
is the standard LSTM (gate blocks i, f, g, o along 4H, one bias vector).
"""
from __future__ import annotations

import math


def _logistic(v: float) -> float:
    return 1.0 / (1.0 + math.exp(-v))


def run_sequence(xs, W, U, b, h, c, outputs=None):
    """Run the cell over the rows of ``xs`` (a list of length-D lists).

    W is D x 4H, U is H x 4H (nested lists), b has 4H entries; h, c have H.
    Returns the final (h, c) as lists of floats; if ``outputs`` is a list, the
    hidden state after each step is appended to it.
    """
    H = len(h)
    h = [float(v) for v in h]
    c = [float(v) for v in c]
    for xt in xs:
        pre = []
        for j in range(4 * H):
            acc = 0.0
            for k, xk in enumerate(xt):
                acc += float(xk) * float(W[k][j])
            for k in range(H):
                acc += h[k] * float(U[k][j])
            pre.append(acc + float(b[j]))
        new_c = []
        new_h = []
        for u in range(H):
            gi = _logistic(pre[u])
            gf = _logistic(pre[H + u])
            gg = math.tanh(pre[2 * H + u])
            go = _logistic(pre[3 * H + u])
            cu = gf * c[u] + gi * gg
            new_c.append(cu)
            new_h.append(go * math.tanh(cu))
        h, c = new_h, new_c
        if outputs is not None:
            outputs.append(list(h))
    return h, c


def forward_per_sequence(x, lengths, W, U, b, h0, c0):
    """Final (h, c) of each sequence run alone for its own length.

    Arguments are numpy arrays or nested lists with the oracle's layouts;
    returns two lists of B lists of H floats.
    """
    Wl = [list(map(float, row)) for row in W]
    Ul = [list(map(float, row)) for row in U]
    bl = list(map(float, b))
    hs, cs = [], []
    for r in range(len(lengths)):
        n = int(lengths[r])
        xs = [list(map(float, x[r][t])) for t in range(n)]
        h, c = run_sequence(xs, Wl, Ul, bl, list(h0[r]), list(c0[r]))
        hs.append(h)
        cs.append(c)
    return hs, cs


def sequence_per_sequence(x, lengths, W, U, b, h0, c0):
    """Output sequence of each sequence run alone: out[r][t] is its hidden
    state after step t for t < L[r] and H zeros for the remaining steps up to
    the padded extent T (the padding convention of the output sequence)."""
    Wl = [list(map(float, row)) for row in W]
    Ul = [list(map(float, row)) for row in U]
    bl = list(map(float, b))
    T, H = len(x[0]), len(h0[0])
    out = []
    for r in range(len(lengths)):
        n = int(lengths[r])
        xs = [list(map(float, x[r][t])) for t in range(n)]
        steps = []
        run_sequence(xs, Wl, Ul, bl, list(h0[r]), list(c0[r]), outputs=steps)
        out.append(steps + [[0.0] * H for _ in range(T - n)])
    return out


def run_sequence_gru(xs, W, U, b_ih, b_hh, h, outputs=None):
    """GRU cell over the rows of ``xs``: W is D x 3H, U is H x 3H (gate blocks
    r, u, n), b_ih and b_hh have 3H entries each, h has H.  Returns the final
    h; if ``outputs`` is a list, h after each step is appended to it."""
    H = len(h)
    h = [float(v) for v in h]
    for xt in xs:
        ax = [sum(float(xk) * float(W[k][j]) for k, xk in enumerate(xt)) + float(b_ih[j]) for j in range(3 * H)]
        ah = [sum(h[k] * float(U[k][j]) for k in range(H)) + float(b_hh[j]) for j in range(3 * H)]
        new_h = []
        for v in range(H):
            r = _logistic(ax[v] + ah[v])
            u = _logistic(ax[H + v] + ah[H + v])
            n = math.tanh(ax[2 * H + v] + r * ah[2 * H + v])
            new_h.append((1.0 - u) * n + u * h[v])
        h = new_h
        if outputs is not None:
            outputs.append(list(h))
    return h


def gru_per_sequence(x, lengths, W, U, b_ih, b_hh, h0):
    """Final h and the zero-padded output sequence of each sequence run alone
    with the GRU cell."""
    T, H = len(x[0]), len(h0[0])
    hs, seqs = [], []
    for r in range(len(lengths)):
        n = int(lengths[r])
        steps = []
        h = run_sequence_gru([list(map(float, x[r][t])) for t in range(n)], W, U, b_ih, b_hh,
                             list(h0[r]), outputs=steps)
        hs.append(h)
        seqs.append(steps + [[0.0] * H for _ in range(T - n)])
    return hs, seqs


def run_sequence_rnn(xs, W, U, b, h, outputs=None):
    """tanh RNN cell over the rows of ``xs``: W is D x H, U is H x H, b has H
    entries, h has H.  Returns the final h; if ``outputs`` is a list, h after
    each step is appended to it."""
    H = len(h)
    h = [float(v) for v in h]
    for xt in xs:
        new_h = []
        for v in range(H):
            acc = sum(float(xk) * float(W[k][v]) for k, xk in enumerate(xt))
            acc += sum(h[k] * float(U[k][v]) for k in range(H))
            new_h.append(math.tanh(acc + float(b[v])))
        h = new_h
        if outputs is not None:
            outputs.append(list(h))
    return h


def rnn_per_sequence(x, lengths, W, U, b, h0):
    """Final h and the zero-padded output sequence of each sequence run alone
    with the tanh RNN cell."""
    T, H = len(x[0]), len(h0[0])
    hs, seqs = [], []
    for r in range(len(lengths)):
        n = int(lengths[r])
        steps = []
        h = run_sequence_rnn([list(map(float, x[r][t])) for t in range(n)], W, U, b,
                             list(h0[r]), outputs=steps)
        hs.append(h)
        seqs.append(steps + [[0.0] * H for _ in range(T - n)])
    return hs, seqs


def stop_per_sequence(x, lengths, W, U, b, h0, c0, v, c_stop, cell="lstm", b_hh=None):
    """Each sequence run alone, one step at a time, until its cap L[r] or the
    first step after which v . h + c_stop > 0.  Returns (hs, cs, steps):
    final states as lists and the number of steps each sequence ran."""
    Wl = [list(map(float, row)) for row in W]
    Ul = [list(map(float, row)) for row in U]
    bl = list(map(float, b))
    vl = list(map(float, v))
    bhl = list(map(float, b_hh)) if b_hh is not None else None
    hs, cs, steps = [], [], []
    for r in range(len(lengths)):
        h = [float(a) for a in h0[r]]
        c = [float(a) for a in c0[r]]
        n = 0
        for t in range(int(lengths[r])):
            xt = [list(map(float, x[r][t]))]
            if cell == "lstm":
                h, c = run_sequence(xt, Wl, Ul, bl, h, c)
            elif cell == "gru":
                h = run_sequence_gru(xt, Wl, Ul, bl, bhl, h)
            else:
                h = run_sequence_rnn(xt, Wl, Ul, bl, h)
            n = t + 1
            if sum(vk * hk for vk, hk in zip(vl, h)) + float(c_stop) > 0.0:
                break
        hs.append(h)
        cs.append(c)
        steps.append(n)
    return hs, cs, steps
