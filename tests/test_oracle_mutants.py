"""Plant plausible mistakes in copies of the C oracle and check that at least
one pin catches each of them.  This shows the pins constrain every part of the
definition: the input and recurrent products, the bias, the gate order and
non-linearities, the cell update, the masking select and the loop bound.
CPU only; the copies are compiled with gcc into a temporary directory."""
import numpy as np
import pytest

import oracle
from tests import oracle_pins

MUTANTS = {
    "drop_bias": ("z[j] += (double)bias[j];", "(void)bias[j];"),
    "drop_recurrent_term": ("z[j] += hk * (double)uk[j];", "(void)(hk + uk[j]);"),
    "drop_input_term": ("z[j] += xk * (double)wk[j];", "(void)(xk + wk[j]);"),
    "transposed_W": ("z[j] += xk * (double)wk[j];", "z[j] += xk * (double)W[(size_t)j * D + k];"),
    "transposed_U": ("z[j] += hk * (double)uk[j];", "z[j] += hk * (double)U[(size_t)j * H + k];"),
    "swap_input_forget_gates": ("const double ig = sig(z[u]);\n        const double fg = sig(z[H + u]);",
                                "const double ig = sig(z[H + u]);\n        const double fg = sig(z[u]);"),
    "swap_cell_output_gates": ("const double gg = tanh(z[2 * H + u]);\n        const double og = sig(z[3 * H + u]);",
                               "const double gg = tanh(z[3 * H + u]);\n        const double og = sig(z[2 * H + u]);"),
    "sigmoid_sign": ("return 1.0 / (1.0 + exp(-v));", "return 1.0 / (1.0 + exp(v));"),
    "output_gate_tanh": ("const double og = sig(z[3 * H + u]);", "const double og = tanh(z[3 * H + u]);"),
    "cell_uses_output_gate": ("const double cc = fg * c[u] + ig * gg;", "const double cc = fg * c[u] + og * gg;"),
    "forget_sign": ("const double cc = fg * c[u] + ig * gg;", "const double cc = -fg * c[u] + ig * gg;"),
    "h_from_old_cell": ("hn[u] = og * tanh(cc);", "hn[u] = og * tanh(c[u]);"),
    "mask_inclusive": ("if (t < L[b]) {", "if (t <= L[b]) {"),
    "no_select": ("if (t < L[b]) {", "if (1) {"),
    "loop_bound_short": ("for (int t = 0; t < max_len; ++t) {", "for (int t = 0; t < max_len - 1; ++t) {"),
    "ignore_initial_cell": ("c[i] = c0[i];", "c[i] = 0.0; (void)c0[i];"),
    "ignore_initial_hidden": ("h[i] = h0[i];", "h[i] = 0.0; (void)h0[i];"),
    "gx_row_stride": ("const float* xt = x + ((size_t)b * T + t) * D;",
                      "const float* xt = x + ((size_t)t * B + b) * D;"),
    # the output sequence
    "seq_holds_cell_state": ("memcpy(seq_out + ((size_t)b * T + t) * H, h + (size_t)b * H,",
                             "memcpy(seq_out + ((size_t)b * T + t) * H, c + (size_t)b * H,"),
    "seq_time_major": ("memcpy(seq_out + ((size_t)b * T + t) * H,", "memcpy(seq_out + ((size_t)t * B + b) * H,"),
    "seq_padding_not_zeroed": ("if (seq_out) memset(seq_out, 0, BH", "if (seq_out) memset(seq_out, 0, 0 * BH"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.compile_variant(src.replace(old, new), str(tmp_path / f"mut_{name}.so"))
    fwd = oracle.forward_with(lib)
    caught = []
    for pin in oracle_pins.PINS:
        try:
            with np.errstate(all="ignore"):
                pin(fwd)
        except (AssertionError, oracle.OracleError):
            caught.append(pin.__name__)
            break
    assert caught, f"no pin caught mutant {name}"


GRU_MUTANTS = {
    "gru_reset_on_input_part": ("const double ng = tanh(zx[2 * H + v] + rg * zh[2 * H + v]);",
                                "const double ng = tanh(rg * zx[2 * H + v] + zh[2 * H + v]);"),
    "gru_update_swapped": ("hn[v] = (1.0 - ug) * ng + ug * h[v];", "hn[v] = ug * ng + (1.0 - ug) * h[v];"),
    "gru_gates_swapped": ("const double rg = sig(zx[v] + zh[v]);\n        const double ug = sig(zx[H + v] + zh[H + v]);",
                          "const double rg = sig(zx[H + v] + zh[H + v]);\n        const double ug = sig(zx[v] + zh[v]);"),
    "gru_hidden_bias_outside_reset": ("zh[j] += (double)bhh[j];", "zx[j] += (double)bhh[j];"),
    "gru_no_recurrent_term": ("for (int j = 0; j < G; ++j) zh[j] += hk * (double)uk[j];",
                              "for (int j = 0; j < G; ++j) (void)(hk + uk[j]);"),
}


@pytest.mark.parametrize("name", sorted(GRU_MUTANTS))
def test_gru_pins_catch_planted_mistake(name, tmp_path):
    old, new = GRU_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.compile_variant(src.replace(old, new), str(tmp_path / f"mut_{name}.so"))
    low = oracle._Lib(lib)

    def fwd(*args, **kw):
        return oracle.forward_gru(*args, _lib_override=low, **kw)
    caught = []
    for pin in oracle_pins.GRU_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(fwd)
        except (AssertionError, oracle.OracleError):
            caught.append(pin.__name__)
            break
    assert caught, f"no pin caught mutant {name}"


RNN_MUTANTS = {
    "rnn_transposed_U": ("a[v] += hv * (double)urow[v];", "a[v] += hv * (double)U[(size_t)v * H + k];"),
    "rnn_transposed_W": ("a[v] += xv * (double)wrow[v];", "a[v] += xv * (double)W[(size_t)v * D + k];"),
    "rnn_no_recurrent_term": ("a[v] += hv * (double)urow[v];", "(void)(hv + urow[v]);"),
    "rnn_drop_bias": ("hn[v] = tanh(a[v] + (double)bias[v]);", "hn[v] = tanh(a[v]);"),
    "rnn_sigmoid_instead_of_tanh": ("hn[v] = tanh(a[v] + (double)bias[v]);", "hn[v] = sig(a[v] + (double)bias[v]);"),
}


@pytest.mark.parametrize("name", sorted(RNN_MUTANTS))
def test_rnn_pins_catch_planted_mistake(name, tmp_path):
    old, new = RNN_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.compile_variant(src.replace(old, new), str(tmp_path / f"mut_{name}.so"))
    low = oracle._Lib(lib)

    def fwd(*args, **kw):
        return oracle.forward_rnn(*args, _lib_override=low, **kw)
    caught = []
    for pin in oracle_pins.RNN_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(fwd)
        except (AssertionError, oracle.OracleError):
            caught.append(pin.__name__)
            break
    assert caught, f"no pin caught mutant {name}"


STOP_MUTANTS = {
    # the score of the state before a step decides whether the row runs it
    "stop_tested_before_the_step": [("            if (!(t < L[b]) || done[b]) continue;\n            int tid = 0;",
                                     "            if (!(t < L[b]) || done[b]) continue;\n            { double s0 = c_stop; for (int k = 0; k < H; ++k) s0 += (double)v[k] * h[(size_t)b * H + k]; if (t > 0 && s0 > 0.0) { done[b] = 1; continue; } }\n            int tid = 0;"),
                                    ("if (score > 0.0) done[b] = 1;", "(void)score;")],
    "stop_on_zero_score": ("if (score > 0.0) done[b] = 1;", "if (score >= 0.0) done[b] = 1;"),
    "stop_without_bias": ("            score += c_stop;\n", ""),
    "loop_ends_when_any_row_ends": ("for (int b = 0; b < B; ++b) any |= (t < L[b]) && !done[b];",
                                    "for (int b = 0; b < B; ++b) any |= 1; for (int b = 0; b < B; ++b) if (done[b]) any = 0;"),
    "terminated_rows_keep_running": ("            if (!(t < L[b]) || done[b]) continue;\n            memcpy(h + (size_t)b * H",
                                     "            if (!(t < L[b])) continue;\n            memcpy(h + (size_t)b * H"),
    "steps_count_from_zero": ("            steps_out[b] = t + 1;", "            steps_out[b] = t;"),
}


@pytest.mark.parametrize("name", sorted(STOP_MUTANTS))
def test_stop_pins_catch_planted_mistake(name, tmp_path):
    edits = STOP_MUTANTS[name]
    src = oracle.source_text()
    for old, new in (edits if isinstance(edits, list) else [edits]):
        assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
        src = src.replace(old, new)
    lib = oracle.compile_variant(src, str(tmp_path / f"mut_{name}.so"))
    low = oracle._Lib(lib)

    def fwd(*args, **kw):
        return oracle.forward_stop(*args, _lib_override=low, **kw)
    caught = []
    for pin in oracle_pins.STOP_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(fwd)
        except (AssertionError, oracle.OracleError):
            caught.append(pin.__name__)
            break
    assert caught, f"no pin caught mutant {name}"


BWD_MUTANTS = {
    "bwd_cell_gradient_not_carried": ("                dc[u] = dct * fg;\n", "                dc[u] = dct;\n"),
    "bwd_tanh_derivative_sign": ("const double dct = dc[u] + dh[u] * og * (1.0 - tc * tc);",
                                 "const double dct = dc[u] + dh[u] * og * (1.0 + tc * tc);"),
    "bwd_sequence_gradient_ignored": ("for (int u = 0; u < H; ++u) dh[u] += dseq[((size_t)b * T + t) * H + u];",
                                      "for (int u = 0; u < H; ++u) (void)dseq[((size_t)b * T + t) * H + u];"),
    "bwd_dU_uses_new_state": ("const double* hprev = hs + (size_t)t * H;", "const double* hprev = hs + (size_t)(t + 1) * H;"),
    "bwd_forget_gate_uses_new_cell": ("dz[H + u] = dct * cprev[u] * fg * (1.0 - fg);", "dz[H + u] = dct * cnew[u] * fg * (1.0 - fg);"),
    "bwd_starts_at_padded_end": ("for (int t = n - 1; t >= 0; --t) {", "for (int t = (n > 0 ? T : 0) - 1; t >= 0; --t) {"),
    "bwd_output_gate_without_derivative": ("dz[3 * H + u] = d_o * og * (1.0 - og);", "dz[3 * H + u] = d_o;"),
}


@pytest.mark.parametrize("name", sorted(BWD_MUTANTS))
def test_backward_pins_catch_planted_mistake(name, tmp_path):
    old, new = BWD_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.compile_variant(src.replace(old, new), str(tmp_path / f"mut_{name}.so"))
    low = oracle._Lib(lib)

    def bwd(*args, **kw):
        return oracle.backward(*args, _lib_override=low, **kw)
    caught = []
    for pin in oracle_pins.BWD_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(bwd)
        except (AssertionError, oracle.OracleError):
            caught.append(pin.__name__)
            break
    assert caught, f"no pin caught mutant {name}"


CELL_BWD_MUTANTS = {
    "gru_bwd_no_direct_path": ("nh[v] = dh[v] * ug;       /* h reaches h' directly through u */",
                               "nh[v] = 0.0;"),
    "gru_bwd_reset_on_input_side": ("da[2 * H + v] = dzn;      de[2 * H + v] = dzn * rg;",
                                    "da[2 * H + v] = dzn * rg; de[2 * H + v] = dzn;"),
    "gru_bwd_update_sign": ("const double du = dh[v] * (hp[v] - ng);", "const double du = dh[v] * (ng - hp[v]);"),
    "rnn_bwd_derivative": ("da[v] = dh[v] * (1.0 - hn * hn);", "da[v] = dh[v] * (1.0 + hn * hn);"),
}


@pytest.mark.parametrize("name", sorted(CELL_BWD_MUTANTS))
def test_cell_backward_pins_catch_planted_mistake(name, tmp_path):
    old, new = CELL_BWD_MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    lib = oracle.compile_variant(src.replace(old, new), str(tmp_path / f"mut_{name}.so"))
    low = oracle._Lib(lib)

    def bwd(cell, x, L, W, U, b, bhh, h0, dh, ds):
        if cell == "gru":
            return oracle.backward_gru(x, L, W, U, b, bhh, h0, dh, ds, _lib_override=low)
        return oracle.backward_rnn(x, L, W, U, b, h0, dh, ds, _lib_override=low)
    caught = []
    for pin in oracle_pins.CELL_BWD_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(bwd)
        except (AssertionError, oracle.OracleError):
            caught.append(pin.__name__)
            break
    assert caught, f"no pin caught mutant {name}"
