/*
 * lstm_oracle.c -- fp64 CPU oracle of the variable-length LSTM time loop.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline do.  It shares no code, header or constant with the HIP library.
 *
 * What it computes (AutoGraph paper, Section 9 "RNN cells", and the
 * hand-written graph form of the same loop in Appendix A):
 *
 *   The state (h, c) starts at (h0, c0).  The loop bound is the largest
 *   sequence length in the batch, max_len.  At step t = 0 .. max_len-1 every
 *   row b with t < L[b] replaces its state by the cell applied to x[b, t] and
 *   that state; every row with t >= L[b] keeps its state.  The masking is a
 *   per-row select, not an arithmetic blend, so nothing computed for a
 *   finished row can reach its state.  The result is the final state, which
 *   for row b is the state after its own L[b] steps.
 *
 * The paper leaves rnn_cell abstract.  The cell here is the standard LSTM with
 * one bias vector and gate blocks (i, f, g, o) along 4H:
 *
 *   z     = x_t W + h U + b          W [D][4H], U [H][4H], b [4H]
 *   i = sig(z_i)  f = sig(z_f)  g = tanh(z_g)  o = sig(z_o)
 *   c'    = f c + i g
 *   h'    = o tanh(c')
 *   sig(v) = 1 / (1 + exp(-v))
 *
 * Each dot product is summed in increasing k: the x part, then the h part,
 * then the bias, so results do not depend on the thread count.
 *
 * Optionally the per-step output sequence is returned as well: out_seq[b][t]
 * is the hidden state row b holds after step t, i.e. the cell's output at
 * that step, for t < L[b], and zero for t >= L[b] (the listings append the
 * cell output at every step; no value is defined past a sequence's length,
 * and zero is the padding convention chosen for it).
 *
 * The same loop with a GRU cell (the paper's rnn_cell is a parameter) is
 * lstm_oracle_forward_gru: W [D][3H], U [H][3H] with gate blocks (r, u, n)
 * and biases b_ih, b_hh [3H] each,
 *
 *   r  = sig(x_t W_r + b_ir + h U_r + b_hr)
 *   u  = sig(x_t W_u + b_iu + h U_u + b_hu)
 *   n  = tanh(x_t W_n + b_in + r * (h U_n + b_hn))
 *   h' = (1 - u) n + u h
 *
 * and no cell state (c is carried unchanged).
 *
 * And with the plain tanh RNN cell, lstm_oracle_forward_rnn: W [D][H],
 * U [H][H], one bias b [H],
 *
 *   h' = tanh(x_t W + h U + b)
 *
 * again with no cell state.
 *
 * Two forms of the masking are provided:
 *   literal = 1 : every row runs the cell at every step and the new state is
 *                 then selected per row.
 *   literal = 0 : rows with t >= L[b] are skipped; the value the
 *                 select would discard is never read, so the result is
 *                 bitwise the same.
 *
 * x, W, U and b are fp32 (bf16 data is widened to fp32 exactly by the caller)
 * and are widened to double here; the state is double; all arithmetic is in
 * double.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Return codes. */
#define ORACLE_OK 0
#define ORACLE_BAD_ARGS 1
#define ORACLE_BAD_LENGTHS 2
#define ORACLE_NOMEM 3

/* Cells. */
#define CELL_LSTM 0
#define CELL_GRU 1
#define CELL_RNN 2

static double sig(double v) { return 1.0 / (1.0 + exp(-v)); }

/* One application of the LSTM cell to one row.
 * xt: [D] input at this step; h, c: [H] current state (fp64);
 * z: [4H] scratch; hn, cn: [H] new state. */
static void lstm_cell_row(int D, int H, const float* xt, const float* W, const float* U,
                          const float* bias, const double* h, const double* c,
                          double* z, double* hn, double* cn) {
    const int G = 4 * H;
    for (int j = 0; j < G; ++j) z[j] = 0.0;
    for (int k = 0; k < D; ++k) {              /* x_t W */
        const double xk = (double)xt[k];
        const float* wk = W + (size_t)k * G;
        for (int j = 0; j < G; ++j) z[j] += xk * (double)wk[j];
    }
    for (int k = 0; k < H; ++k) {              /* + h U */
        const double hk = h[k];
        const float* uk = U + (size_t)k * G;
        for (int j = 0; j < G; ++j) z[j] += hk * (double)uk[j];
    }
    for (int j = 0; j < G; ++j) z[j] += (double)bias[j];   /* + b */
    for (int u = 0; u < H; ++u) {
        const double ig = sig(z[u]);
        const double fg = sig(z[H + u]);
        const double gg = tanh(z[2 * H + u]);
        const double og = sig(z[3 * H + u]);
        const double cc = fg * c[u] + ig * gg;
        cn[u] = cc;
        hn[u] = og * tanh(cc);
    }
}

/* One application of the GRU cell to one row.  W [D][3H], U [H][3H],
 * bih, bhh [3H]; zx, zh: [3H] scratch (input and recurrent parts, each with
 * its bias); hn: [H] new hidden state. */
static void gru_cell_row(int D, int H, const float* xt, const float* W, const float* U,
                         const float* bih, const float* bhh, const double* h, double* zx,
                         double* zh, double* hn) {
    const int G = 3 * H;
    for (int j = 0; j < G; ++j) {
        zx[j] = 0.0;
        zh[j] = 0.0;
    }
    for (int k = 0; k < D; ++k) {              /* x_t W */
        const double xk = (double)xt[k];
        const float* wk = W + (size_t)k * G;
        for (int j = 0; j < G; ++j) zx[j] += xk * (double)wk[j];
    }
    for (int k = 0; k < H; ++k) {              /* h U */
        const double hk = h[k];
        const float* uk = U + (size_t)k * G;
        for (int j = 0; j < G; ++j) zh[j] += hk * (double)uk[j];
    }
    for (int j = 0; j < G; ++j) {
        zx[j] += (double)bih[j];
        zh[j] += (double)bhh[j];
    }
    for (int v = 0; v < H; ++v) {
        const double rg = sig(zx[v] + zh[v]);
        const double ug = sig(zx[H + v] + zh[H + v]);
        const double ng = tanh(zx[2 * H + v] + rg * zh[2 * H + v]);
        hn[v] = (1.0 - ug) * ng + ug * h[v];
    }
}

/* One application of the tanh RNN cell to one row.  W [D][H], U [H][H],
 * bias [H]; a: [H] scratch; hn: [H] new hidden state. */
static void rnn_cell_row(int D, int H, const float* xt, const float* W, const float* U,
                         const float* bias, const double* h, double* a, double* hn) {
    for (int v = 0; v < H; ++v) a[v] = 0.0;
    for (int k = 0; k < D; ++k) {              /* x_t W */
        const double xv = (double)xt[k];
        const float* wrow = W + (size_t)k * H;
        for (int v = 0; v < H; ++v) a[v] += xv * (double)wrow[v];
    }
    for (int k = 0; k < H; ++k) {              /* + h U */
        const double hv = h[k];
        const float* urow = U + (size_t)k * H;
        for (int v = 0; v < H; ++v) a[v] += hv * (double)urow[v];
    }
    for (int v = 0; v < H; ++v) hn[v] = tanh(a[v] + (double)bias[v]);   /* + b, tanh */
}

/*
 * forward_impl (exported as lstm_oracle_forward and lstm_oracle_forward_seq
 * with cell = CELL_LSTM; as lstm_oracle_forward_gru with cell = CELL_GRU,
 * where W, U are [D][3H], [H][3H], bias is b_ih [3H] and bhh is b_hh [3H];
 * as lstm_oracle_forward_rnn with cell = CELL_RNN, where W, U are [D][H],
 * [H][H] and bias is [H])
 *   B, T, D, H   : batch, padded time extent, input width, hidden width (> 0)
 *   x            : [B][T][D] fp32
 *   L            : [B] int32 sequence lengths, each in [0, T]
 *   W, U         : [D][4H], [H][4H] fp32
 *   bias         : [4H] fp32
 *   h0, c0       : [B][H] fp64 initial state (fp32 data widened exactly; fp64
 *                  lets a run resume bitwise from a state this function wrote)
 *   h_out, c_out : [B][H] fp64 final state (written)
 *   literal      : 1 = compute every row then select, 0 = skip finished rows
 *   nthreads     : OpenMP threads over the rows of one step (<= 0: default)
 *   steps_out    : if non-NULL, receives the number of loop iterations run
 *   seq_out      : if non-NULL, [B][T][H] fp64 output sequence (written)
 * Returns ORACLE_OK, or an error code with the outputs untouched.
 */
static int forward_impl(int B, int T, int D, int H, const float* x, const int32_t* L,
                        const float* W, const float* U, const float* bias,
                        const double* h0, const double* c0, double* h_out, double* c_out,
                        int literal, int nthreads, int64_t* steps_out, double* seq_out,
                        int cell, const float* bhh) {
    if (B <= 0 || T < 0 || D <= 0 || H <= 0 || !x || !L || !W || !U || !bias || !h0 || !c0 ||
        !h_out || !c_out)
        return ORACLE_BAD_ARGS;
    int max_len = 0;
    for (int b = 0; b < B; ++b) {
        if (L[b] < 0 || L[b] > T) return ORACLE_BAD_LENGTHS;
        if (L[b] > max_len) max_len = L[b];
    }
    const size_t BH = (size_t)B * H;
    double* h = (double*)malloc(BH * sizeof(double));
    double* c = (double*)malloc(BH * sizeof(double));
    double* hn = (double*)malloc(BH * sizeof(double));
    double* cn = (double*)malloc(BH * sizeof(double));
    int nt = 1;
#ifdef _OPENMP
    nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#endif
    double* zs = (double*)malloc((size_t)nt * 6 * H * sizeof(double));  /* 4H (LSTM) or 2 x 3H (GRU) */
    if (!h || !c || !hn || !cn || !zs) {
        free(h); free(c); free(hn); free(cn); free(zs);
        return ORACLE_NOMEM;
    }
    for (size_t i = 0; i < BH; ++i) {            /* initial state */
        h[i] = h0[i];
        c[i] = c0[i];
    }
    if (seq_out) memset(seq_out, 0, BH * (size_t)T * sizeof(double));  /* zero past each length */
    for (int t = 0; t < max_len; ++t) {          /* t < max_len: the loop bound */
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(dynamic, 1)
#endif
        for (int b = 0; b < B; ++b) {
            const int active = t < L[b];
            if (!active && !literal) continue;
            int tid = 0;
#ifdef _OPENMP
            tid = omp_get_thread_num();
#endif
            double* z = zs + (size_t)tid * 6 * H;
            const float* xt = x + ((size_t)b * T + t) * D;
            if (cell == CELL_GRU) {
                gru_cell_row(D, H, xt, W, U, bias, bhh, h + (size_t)b * H, z, z + 3 * H,
                             hn + (size_t)b * H);
                memcpy(cn + (size_t)b * H, c + (size_t)b * H, (size_t)H * sizeof(double));
            } else if (cell == CELL_RNN) {
                rnn_cell_row(D, H, xt, W, U, bias, h + (size_t)b * H, z, hn + (size_t)b * H);
                memcpy(cn + (size_t)b * H, c + (size_t)b * H, (size_t)H * sizeof(double));
            } else {
                lstm_cell_row(D, H, xt, W, U, bias, h + (size_t)b * H, c + (size_t)b * H, z,
                              hn + (size_t)b * H, cn + (size_t)b * H);
            }
        }
        /* Per-row select: rows with t < L[b] take the new state, the others
         * keep theirs.  Commits happen after every row of the step is done. */
        for (int b = 0; b < B; ++b) {
            if (t < L[b]) {
                memcpy(h + (size_t)b * H, hn + (size_t)b * H, (size_t)H * sizeof(double));
                memcpy(c + (size_t)b * H, cn + (size_t)b * H, (size_t)H * sizeof(double));
                if (seq_out)                     /* the cell's output at step t */
                    memcpy(seq_out + ((size_t)b * T + t) * H, h + (size_t)b * H, (size_t)H * sizeof(double));
            }
        }
    }
    memcpy(h_out, h, BH * sizeof(double));
    memcpy(c_out, c, BH * sizeof(double));
    if (steps_out) *steps_out = max_len;
    free(h); free(c); free(hn); free(cn); free(zs);
    return ORACLE_OK;
}

int lstm_oracle_forward(int B, int T, int D, int H, const float* x, const int32_t* L,
                        const float* W, const float* U, const float* bias,
                        const double* h0, const double* c0, double* h_out, double* c_out,
                        int literal, int nthreads, int64_t* steps_out) {
    return forward_impl(B, T, D, H, x, L, W, U, bias, h0, c0, h_out, c_out, literal, nthreads,
                        steps_out, NULL, CELL_LSTM, NULL);
}

/* As lstm_oracle_forward, and also the output sequence seq_out [B][T][H]. */
int lstm_oracle_forward_seq(int B, int T, int D, int H, const float* x, const int32_t* L,
                            const float* W, const float* U, const float* bias,
                            const double* h0, const double* c0, double* h_out, double* c_out,
                            int literal, int nthreads, int64_t* steps_out, double* seq_out) {
    if (!seq_out) return ORACLE_BAD_ARGS;
    return forward_impl(B, T, D, H, x, L, W, U, bias, h0, c0, h_out, c_out, literal, nthreads,
                        steps_out, seq_out, CELL_LSTM, NULL);
}

/* The loop with the GRU cell: W [D][3H], U [H][3H], bih = b_ih [3H],
 * bhh = b_hh [3H]; c0 is carried to c_out unchanged; seq_out may be NULL. */
int lstm_oracle_forward_gru(int B, int T, int D, int H, const float* x, const int32_t* L,
                            const float* W, const float* U, const float* bih, const float* bhh,
                            const double* h0, const double* c0, double* h_out, double* c_out,
                            int literal, int nthreads, int64_t* steps_out, double* seq_out) {
    if (!bhh) return ORACLE_BAD_ARGS;
    return forward_impl(B, T, D, H, x, L, W, U, bih, h0, c0, h_out, c_out, literal, nthreads,
                        steps_out, seq_out, CELL_GRU, bhh);
}

/* The loop with the tanh RNN cell: W [D][H], U [H][H], bias [H]; c0 is
 * carried to c_out unchanged; seq_out may be NULL. */
int lstm_oracle_forward_rnn(int B, int T, int D, int H, const float* x, const int32_t* L,
                            const float* W, const float* U, const float* bias,
                            const double* h0, const double* c0, double* h_out, double* c_out,
                            int literal, int nthreads, int64_t* steps_out, double* seq_out) {
    return forward_impl(B, T, D, H, x, L, W, U, bias, h0, c0, h_out, c_out, literal, nthreads,
                        steps_out, seq_out, CELL_RNN, NULL);
}

/*
 * lstm_oracle_forward_stop: the loop with its termination computed from the
 * state.  The paper's decoders (beam search and seq2seq, Appendix D) leave the
 * loop once every candidate sequence has terminated; here a row terminates
 * when a linear read-out of its state, the halting score
 *
 *   s = (sum over k of v[k] h[k]) + c_stop,      summed in increasing k,
 *
 * is positive after one of its steps.  L[b] caps the steps of row b (x holds
 * data for t < L[b]).  At step t a row is running if t < L[b] and it has not
 * terminated; the loop stops at the first step with no running row.  Running
 * rows take the cell's new state, the others keep theirs.
 *   cell        : CELL_LSTM, CELL_GRU (bias = b_ih, bhh = b_hh) or CELL_RNN
 *   v [H], c_stop: the read-out
 *   steps_out   : [B] int32, the steps row b ran
 *   iters_out   : loop iterations run (= the largest entry of steps_out)
 *   seq_out     : if non-NULL, [B][T][H] hidden state after each step a row
 *                 ran, zero after its last
 * Returns ORACLE_OK or an error code.
 */
int lstm_oracle_forward_stop(int B, int T, int D, int H, const float* x, const int32_t* L,
                             const float* W, const float* U, const float* bias, const float* bhh,
                             int cell, const float* v, double c_stop, const double* h0,
                             const double* c0, double* h_out, double* c_out, int32_t* steps_out,
                             int64_t* iters_out, double* seq_out, int nthreads) {
    if (B <= 0 || T < 0 || D <= 0 || H <= 0 || !x || !L || !W || !U || !bias || !v || !h0 ||
        !c0 || !h_out || !c_out || !steps_out || (cell == CELL_GRU && !bhh))
        return ORACLE_BAD_ARGS;
    if (cell != CELL_LSTM && cell != CELL_GRU && cell != CELL_RNN) return ORACLE_BAD_ARGS;
    int max_len = 0;
    for (int b = 0; b < B; ++b) {
        if (L[b] < 0 || L[b] > T) return ORACLE_BAD_LENGTHS;
        if (L[b] > max_len) max_len = L[b];
    }
    const size_t BH = (size_t)B * H;
    double* h = (double*)malloc(BH * sizeof(double));
    double* c = (double*)malloc(BH * sizeof(double));
    double* hn = (double*)malloc(BH * sizeof(double));
    double* cn = (double*)malloc(BH * sizeof(double));
    unsigned char* done = (unsigned char*)calloc((size_t)B, 1);
    int nt = 1;
#ifdef _OPENMP
    nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#endif
    double* zs = (double*)malloc((size_t)nt * 6 * H * sizeof(double));
    if (!h || !c || !hn || !cn || !done || !zs) {
        free(h); free(c); free(hn); free(cn); free(done); free(zs);
        return ORACLE_NOMEM;
    }
    memcpy(h, h0, BH * sizeof(double));          /* initial state */
    memcpy(c, c0, BH * sizeof(double));
    for (int b = 0; b < B; ++b) steps_out[b] = 0;
    if (seq_out) memset(seq_out, 0, (size_t)T * BH * sizeof(double));  /* zero after each row's last step */
    int64_t iters = 0;
    for (int t = 0; t < max_len; t++) {
        int any = 0;                             /* leave the loop once no row runs */
        for (int b = 0; b < B; ++b) any |= (t < L[b]) && !done[b];
        if (!any) break;
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(dynamic, 1)
#endif
        for (int b = 0; b < B; ++b) {
            if (!(t < L[b]) || done[b]) continue;
            int tid = 0;
#ifdef _OPENMP
            tid = omp_get_thread_num();
#endif
            double* z = zs + (size_t)tid * 6 * H;
            const float* xrow = x + ((size_t)b * T + t) * D;
            double* hb = h + (size_t)b * H;
            if (cell == CELL_GRU) {
                gru_cell_row(D, H, xrow, W, U, bias, bhh, hb, z, z + 3 * H, hn + (size_t)b * H);
                memcpy(cn + (size_t)b * H, c + (size_t)b * H, (size_t)H * sizeof(double));
            } else if (cell == CELL_RNN) {
                rnn_cell_row(D, H, xrow, W, U, bias, hb, z, hn + (size_t)b * H);
                memcpy(cn + (size_t)b * H, c + (size_t)b * H, (size_t)H * sizeof(double));
            } else {
                lstm_cell_row(D, H, xrow, W, U, bias, hb, c + (size_t)b * H, z, hn + (size_t)b * H,
                              cn + (size_t)b * H);
            }
        }
        for (int b = 0; b < B; ++b) {            /* commit the running rows, then test them */
            if (!(t < L[b]) || done[b]) continue;
            memcpy(h + (size_t)b * H, hn + (size_t)b * H, (size_t)H * sizeof(double));
            memcpy(c + (size_t)b * H, cn + (size_t)b * H, (size_t)H * sizeof(double));
            steps_out[b] = t + 1;
            if (seq_out)                         /* the row's output at step t */
                memcpy(&seq_out[((size_t)b * T + t) * H], &h[(size_t)b * H], (size_t)H * sizeof(double));
            double score = 0.0;
            for (int k = 0; k < H; ++k) score += (double)v[k] * h[(size_t)b * H + k];
            score += c_stop;
            if (score > 0.0) done[b] = 1;       /* terminated after this step */
        }
        iters = t + 1;
    }
    memcpy(h_out, h, BH * sizeof(double));
    memcpy(c_out, c, BH * sizeof(double));
    if (iters_out) *iters_out = iters;
    free(h); free(c); free(hn); free(cn); free(done); free(zs);
    return ORACLE_OK;
}

/*
 * lstm_oracle_backward: gradients of the masked LSTM loop (backpropagation
 * through time; the paper trains its staged models in-graph, Section 9).
 * Given the upstream gradients of the final state (dh_out, dc_out [B][H])
 * and, optionally, of the output sequence (dseq [B][T][H], may be NULL;
 * entries at t >= L[b] have no effect), it returns the gradients of the loss
 * with respect to x [B][T][D], W [D][4H], U [H][4H], b [4H], h0, c0 [B][H].
 *
 * A step that a row does not take passes its state through unchanged, so
 * the gradient of such a step is the identity; each row is therefore
 * differentiated through its own L[b] steps, backwards from the last:
 *   dh += dseq[t]
 *   o-gate:  do  = dh * tanh(c_t)
 *   cell:    dct = dc + dh * o * (1 - tanh(c_t)^2)
 *   di = dct * g, df = dct * c_{t-1}, dg = dct * i, dc <- dct * f
 *   dz = (di i (1 - i), df f (1 - f), dg (1 - g^2), do o (1 - o))
 *   db += dz, dW += x_t^T dz, dU += h_{t-1}^T dz, dx_t = dz W^T, dh <- dz U^T
 * with (i, f, g, o) and c_t recomputed by the forward in double precision.
 * Rows are differentiated one after another in order 0 .. B-1 and the
 * weight gradients summed in that order, step by step from each row's last.
 *
 * Threads (nthreads, <= 0: all) change only the schedule, never the order of
 * any sum: the forward recompute runs rows of a block side by side (each
 * row's recompute is serial), and each reverse step splits its products by
 * k, so every entry of dW, dU and dx (and of dh through dz U^T) is summed by
 * one thread in the order above.  The result is the same bits for every
 * thread count.
 */

/* Rows of one block whose forward recompute is held at once: at most nt,
 * and at most about 1 GB of saved states. */
static int bwd_block_rows(int nt, int T, int per_step_doubles) {
    const double bytes = (double)(T > 0 ? T : 1) * per_step_doubles * sizeof(double);
    int r = (int)(1.0e9 / bytes);
    if (r < 1) r = 1;
    return r < nt ? r : nt;
}

int lstm_oracle_backward(int B, int T, int D, int H, const float* x, const int32_t* L,
                         const float* W, const float* U, const float* bias, const double* h0,
                         const double* c0, const double* dh_out, const double* dc_out,
                         const double* dseq, double* dx, double* dW, double* dU, double* db,
                         double* dh0, double* dc0, int nthreads) {
    if (B <= 0 || T < 0 || D <= 0 || H <= 0 || !x || !L || !W || !U || !bias || !h0 || !c0 ||
        !dh_out || !dc_out || !dx || !dW || !dU || !db || !dh0 || !dc0)
        return ORACLE_BAD_ARGS;
    for (int b = 0; b < B; ++b)
        if (L[b] < 0 || L[b] > T) return ORACLE_BAD_LENGTHS;
    const int G = 4 * H;
    int nt = 1;
#ifdef _OPENMP
    nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#endif
    /* per row of a block: z_t per step, c_{t-1} and h_{t-1} for t = 0..T */
    const size_t zrow = (size_t)(T > 0 ? T : 1) * G, srow = (size_t)(T + 1) * H;
    const int nb = bwd_block_rows(nt, T, 6 * H);
    double* zblk = (double*)malloc((size_t)nb * zrow * sizeof(double));
    double* cblk = (double*)malloc((size_t)nb * srow * sizeof(double));
    double* hblk = (double*)malloc((size_t)nb * srow * sizeof(double));
    double* dz = (double*)malloc((size_t)G * sizeof(double));
    double* dh = (double*)malloc((size_t)H * sizeof(double));
    double* dc = (double*)malloc((size_t)H * sizeof(double));
    double* nh = (double*)malloc((size_t)H * sizeof(double));
    if (!zblk || !cblk || !hblk || !dz || !dh || !dc || !nh) {
        free(zblk); free(cblk); free(hblk); free(dz); free(dh); free(dc); free(nh);
        return ORACLE_NOMEM;
    }
    memset(dx, 0, (size_t)B * T * D * sizeof(double));
    memset(dW, 0, (size_t)D * G * sizeof(double));
    memset(dU, 0, (size_t)H * G * sizeof(double));
    memset(db, 0, (size_t)G * sizeof(double));
    for (int b0 = 0; b0 < B; b0 += nb) {
        const int rows = B - b0 < nb ? B - b0 : nb;
        /* forward through each row's own steps, keeping z_t, c and h */
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(dynamic, 1)
#endif
        for (int r = 0; r < rows; ++r) {
            const int b = b0 + r, n = L[b];
            double* zs = zblk + (size_t)r * zrow;
            double* cs = cblk + (size_t)r * srow;
            double* hs = hblk + (size_t)r * srow;
            memcpy(hs, h0 + (size_t)b * H, (size_t)H * sizeof(double));
            memcpy(cs, c0 + (size_t)b * H, (size_t)H * sizeof(double));
            for (int t = 0; t < n; ++t) {
                const float* xin = &x[((size_t)b * T + t) * D];
                lstm_cell_row(D, H, xin, W, U, bias, hs + (size_t)t * H, cs + (size_t)t * H,
                              zs + (size_t)t * G, hs + (size_t)(t + 1) * H, cs + (size_t)(t + 1) * H);
            }
        }
        for (int r = 0; r < rows; ++r) {
            const int b = b0 + r, n = L[b];
            const double* zs = zblk + (size_t)r * zrow;
            const double* cs = cblk + (size_t)r * srow;
            const double* hs = hblk + (size_t)r * srow;
            memcpy(dh, dh_out + (size_t)b * H, (size_t)H * sizeof(double));
            memcpy(dc, dc_out + (size_t)b * H, (size_t)H * sizeof(double));
            for (int t = n - 1; t >= 0; --t) {
                if (dseq)
                    for (int u = 0; u < H; ++u) dh[u] += dseq[((size_t)b * T + t) * H + u];
                const double* z = zs + (size_t)t * G;
                const double* cprev = cs + (size_t)t * H;
                const double* cnew = cs + (size_t)(t + 1) * H;
                for (int u = 0; u < H; ++u) {
                    const double ig = sig(z[u]), fg = sig(z[H + u]);
                    const double gg = tanh(z[2 * H + u]), og = sig(z[3 * H + u]);
                    const double tc = tanh(cnew[u]);
                    const double d_o = dh[u] * tc;
                    const double dct = dc[u] + dh[u] * og * (1.0 - tc * tc);
                    dz[u] = dct * gg * ig * (1.0 - ig);
                    dz[H + u] = dct * cprev[u] * fg * (1.0 - fg);
                    dz[2 * H + u] = dct * ig * (1.0 - gg * gg);
                    dz[3 * H + u] = d_o * og * (1.0 - og);
                    dc[u] = dct * fg;
                }
                for (int j = 0; j < G; ++j) db[j] += dz[j];
                const float* xin = &x[((size_t)b * T + t) * D];
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(static)
#endif
                for (int k = 0; k < D; ++k) {      /* dW += x_t^T dz, dx_t = dz W^T */
                    double acc = 0.0;
                    for (int j = 0; j < G; ++j) {
                        dW[(size_t)k * G + j] += (double)xin[k] * dz[j];
                        acc += dz[j] * (double)W[(size_t)k * G + j];
                    }
                    dx[((size_t)b * T + t) * D + k] = acc;
                }
                const double* hprev = hs + (size_t)t * H;
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(static)
#endif
                for (int k = 0; k < H; ++k) {      /* dU += h_{t-1}^T dz, dh = dz U^T */
                    double acc = 0.0;
                    for (int j = 0; j < G; ++j) {
                        dU[(size_t)k * G + j] += hprev[k] * dz[j];
                        acc += dz[j] * (double)U[(size_t)k * G + j];
                    }
                    nh[k] = acc;
                }
                memcpy(dh, nh, (size_t)H * sizeof(double));
            }
            memcpy(dh0 + (size_t)b * H, dh, (size_t)H * sizeof(double));
            memcpy(dc0 + (size_t)b * H, dc, (size_t)H * sizeof(double));
        }
    }
    free(zblk); free(cblk); free(hblk); free(dz); free(dh); free(dc); free(nh);
    return ORACLE_OK;
}

/*
 * lstm_oracle_backward_cell: the backward pass for the GRU (cell = CELL_GRU;
 * W [D][3H], U [H][3H], bias = b_ih [3H], bhh = b_hh [3H]) and the tanh RNN
 * (cell = CELL_RNN; W [D][H], U [H][H], bias [H]).  Same loss and masking as
 * lstm_oracle_backward, no cell state: returns dx, dW, dU, the bias gradients
 * (db = d b_ih, dbhh = d b_hh for the GRU; dbhh unused for the RNN) and dh0.
 *   GRU, with a = x W + b_ih and e = h U + b_hh of the step:
 *     dn = dh (1 - u), du = dh (h - n), dh_prev = dh u + (de) U^T
 *     dzn = dn (1 - n^2); da_n = dzn; de_n = dzn r; dr = dzn e_n
 *     da_r = de_r = dr r (1 - r); da_u = de_u = du u (1 - u)
 *     dW += x^T da, dU += h^T de, db_ih += da, db_hh += de, dx = da W^T
 *   RNN, with h' = tanh(z):  dz = dh (1 - h'^2), dh_prev = dz U^T, and the
 *     same weight, bias and input gradients with da = de = dz.
 * Order of the sums and threads (nthreads) as for lstm_oracle_backward.
 */
int lstm_oracle_backward_cell(int B, int T, int D, int H, int cell, const float* x,
                              const int32_t* L, const float* W, const float* U,
                              const float* bias, const float* bhh, const double* h0,
                              const double* dh_out, const double* dseq, double* dx, double* dW,
                              double* dU, double* db, double* dbhh, double* dh0, int nthreads) {
    if (B <= 0 || T < 0 || D <= 0 || H <= 0 || !x || !L || !W || !U || !bias || !h0 ||
        !dh_out || !dx || !dW || !dU || !db || !dh0)
        return ORACLE_BAD_ARGS;
    if (cell != CELL_GRU && cell != CELL_RNN) return ORACLE_BAD_ARGS;
    if (cell == CELL_GRU && (!bhh || !dbhh)) return ORACLE_BAD_ARGS;
    for (int b = 0; b < B; ++b)
        if (L[b] < 0 || L[b] > T) return ORACLE_BAD_LENGTHS;
    const int G = cell == CELL_GRU ? 3 * H : H;
    int nt = 1;
#ifdef _OPENMP
    nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#endif
    /* per row of a block: h_{t-1} for t = 0..T, and a, e (GRU) or z (RNN) per step */
    const size_t hrow = (size_t)(T + 1) * H, zrow = (size_t)(T > 0 ? T : 1) * 2 * G;
    const int nb = bwd_block_rows(nt, T, H + 2 * G);
    double* hblk = (double*)malloc((size_t)nb * hrow * sizeof(double));
    double* zblk = (double*)malloc((size_t)nb * zrow * sizeof(double));
    double* da = (double*)malloc((size_t)G * sizeof(double));              /* input-side grads */
    double* de = (double*)malloc((size_t)G * sizeof(double));              /* recurrent-side */
    double* dh = (double*)malloc((size_t)H * sizeof(double));
    double* nh = (double*)malloc((size_t)H * sizeof(double));
    if (!hblk || !zblk || !da || !de || !dh || !nh) {
        free(hblk); free(zblk); free(da); free(de); free(dh); free(nh);
        return ORACLE_NOMEM;
    }
    memset(dx, 0, (size_t)B * T * D * sizeof(double));
    memset(dW, 0, (size_t)D * G * sizeof(double));
    memset(dU, 0, (size_t)H * G * sizeof(double));
    memset(db, 0, (size_t)G * sizeof(double));
    if (cell == CELL_GRU) memset(dbhh, 0, (size_t)G * sizeof(double));
    for (int b0 = 0; b0 < B; b0 += nb) {
        const int rows = B - b0 < nb ? B - b0 : nb;
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(dynamic, 1)
#endif
        for (int r = 0; r < rows; ++r) {        /* forward, keeping a and e (GRU) or z (RNN) */
            const int b = b0 + r, n = L[b];
            double* hs = hblk + (size_t)r * hrow;
            double* zs = zblk + (size_t)r * zrow;
            memcpy(hs, h0 + (size_t)b * H, (size_t)H * sizeof(double));
            for (int t = 0; t < n; ++t) {
                const float* xr = x + ((size_t)b * T + t) * D;
                double* za = zs + (size_t)t * 2 * G;
                if (cell == CELL_GRU)
                    gru_cell_row(D, H, xr, W, U, bias, bhh, hs + (size_t)t * H, za, za + G,
                                 hs + (size_t)(t + 1) * H);
                else
                    rnn_cell_row(D, H, xr, W, U, bias, hs + (size_t)t * H, za, hs + (size_t)(t + 1) * H);
            }
        }
        for (int r = 0; r < rows; ++r) {
            const int b = b0 + r, n = L[b];
            const double* hs = hblk + (size_t)r * hrow;
            const double* zs = zblk + (size_t)r * zrow;
            memcpy(dh, dh_out + (size_t)b * H, (size_t)H * sizeof(double));
            for (int t = n; t-- > 0;) {          /* last step first */
                if (dseq)
                    for (int v = 0; v < H; ++v) dh[v] += dseq[((size_t)b * T + t) * H + v];
                const double* hp = hs + (size_t)t * H;
                const double* za = zs + (size_t)t * 2 * G;
                if (cell == CELL_GRU) {
                    const double* ze = za + G;
                    for (int v = 0; v < H; ++v) {
                        const double rg = sig(za[v] + ze[v]);
                        const double ug = sig(za[H + v] + ze[H + v]);
                        const double ng = tanh(za[2 * H + v] + rg * ze[2 * H + v]);
                        const double dn = dh[v] * (1.0 - ug);
                        const double du = dh[v] * (hp[v] - ng);
                        const double dzn = dn * (1.0 - ng * ng);
                        const double dr = dzn * ze[2 * H + v];
                        const double dzr = dr * rg * (1.0 - rg), dzu = du * ug * (1.0 - ug);
                        da[v] = dzr;              de[v] = dzr;
                        da[H + v] = dzu;          de[H + v] = dzu;
                        da[2 * H + v] = dzn;      de[2 * H + v] = dzn * rg;
                        nh[v] = dh[v] * ug;       /* h reaches h' directly through u */
                    }
                } else {
                    const double* hnew = hs + (size_t)(t + 1) * H;
                    for (int v = 0; v < H; ++v) {
                        const double hn = hnew[v];       /* tanh(z) of the step */
                        da[v] = dh[v] * (1.0 - hn * hn);
                        de[v] = da[v];
                        nh[v] = 0.0;
                    }
                }
                for (int j = 0; j < G; ++j) {
                    db[j] += da[j];
                    if (cell == CELL_GRU) dbhh[j] += de[j];
                }
                const float* xr = x + ((size_t)b * T + t) * D;
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(static)
#endif
                for (int k = 0; k < D; ++k) {      /* dW += x^T da, dx = da W^T */
                    double acc = 0.0;
                    for (int j = 0; j < G; ++j) {
                        dW[(size_t)k * G + j] += (double)xr[k] * da[j];
                        acc += da[j] * (double)W[(size_t)k * G + j];
                    }
                    dx[((size_t)b * T + t) * D + k] = acc;
                }
#ifdef _OPENMP
#pragma omp parallel for num_threads(nt) schedule(static)
#endif
                for (int k = 0; k < H; ++k) {      /* dU += h^T de, dh_prev = direct + de U^T */
                    double acc = nh[k];
                    for (int j = 0; j < G; ++j) {
                        dU[(size_t)k * G + j] += hp[k] * de[j];
                        acc += de[j] * (double)U[(size_t)k * G + j];
                    }
                    dh[k] = acc;
                }
            }
            memcpy(dh0 + (size_t)b * H, dh, (size_t)H * sizeof(double));
        }
    }
    free(hblk); free(zblk); free(da); free(de); free(dh); free(nh);
    return ORACLE_OK;
}

/* Number of OpenMP threads a call with nthreads <= 0 would use. */
int lstm_oracle_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
