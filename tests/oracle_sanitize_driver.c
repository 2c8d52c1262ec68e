/*
 * A CPU driver that runs every entry point of the C oracle on small and
 * degenerate inputs (lengths 0 and T, one row, widths of 1, ragged sizes, one
 * and several threads).  It is compiled together with the oracle source under
 * -fsanitize=address,undefined by tests/test_oracle_sanitize.py; any invalid
 * access, leak or undefined behaviour ends the run with an error.  Inputs come
 * from a fixed linear congruential generator; nothing here checks values (the
 * pins do that), only that every call returns its documented status.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int lstm_oracle_forward(int, int, int, int, const float*, const int32_t*, const float*,
                        const float*, const float*, const double*, const double*, double*,
                        double*, int, int, int64_t*);
int lstm_oracle_forward_seq(int, int, int, int, const float*, const int32_t*, const float*,
                            const float*, const float*, const double*, const double*, double*,
                            double*, int, int, int64_t*, double*);
int lstm_oracle_forward_gru(int, int, int, int, const float*, const int32_t*, const float*,
                            const float*, const float*, const float*, const double*,
                            const double*, double*, double*, int, int, int64_t*, double*);
int lstm_oracle_forward_rnn(int, int, int, int, const float*, const int32_t*, const float*,
                            const float*, const float*, const double*, const double*, double*,
                            double*, int, int, int64_t*, double*);
int lstm_oracle_forward_stop(int, int, int, int, const float*, const int32_t*, const float*,
                             const float*, const float*, const float*, int, const float*, double,
                             const double*, const double*, double*, double*, int32_t*, int64_t*,
                             double*, int);
int lstm_oracle_backward(int, int, int, int, const float*, const int32_t*, const float*,
                         const float*, const float*, const double*, const double*, const double*,
                         const double*, const double*, double*, double*, double*, double*,
                         double*, double*, int);
int lstm_oracle_backward_cell(int, int, int, int, int, const float*, const int32_t*,
                              const float*, const float*, const float*, const float*,
                              const double*, const double*, const double*, double*, double*,
                              double*, double*, double*, double*, int);

static uint64_t g_state = 0x9e3779b97f4a7c15ull;
static double uni(void) {               /* in [-1, 1) */
    g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
    return (double)(g_state >> 11) * (2.0 / 9007199254740992.0) - 1.0;
}
static float* fvec(size_t n, double s) {
    float* p = (float*)malloc((n ? n : 1) * sizeof(float));
    for (size_t i = 0; i < n; ++i) p[i] = (float)(s * uni());
    return p;
}
static double* dvec(size_t n, double s) {
    double* p = (double*)malloc((n ? n : 1) * sizeof(double));
    for (size_t i = 0; i < n; ++i) p[i] = s * uni();
    return p;
}

static int failures = 0;
static void expect(int rc, int want, const char* what, int B, int T, int D, int H) {
    if (rc != want) {
        fprintf(stderr, "%s B=%d T=%d D=%d H=%d: status %d, expected %d\n", what, B, T, D, H, rc, want);
        ++failures;
    }
}

static void run_case(int B, int T, int D, int H, int zero_lengths, int threads) {
    const size_t G4 = 4 * (size_t)H, G3 = 3 * (size_t)H;
    float* x = fvec((size_t)B * T * D, 1.0);
    int32_t* L = (int32_t*)malloc((size_t)B * sizeof(int32_t));
    for (int b = 0; b < B; ++b)
        L[b] = zero_lengths ? 0 : (b == 0 ? T : (int)((uni() * 0.5 + 0.5) * (T + 1)) % (T + 1));
    float* W = fvec((size_t)D * G4, 0.5);
    float* U = fvec((size_t)H * G4, 0.5);
    float* bias = fvec(G4, 0.5);
    float* bhh = fvec(G3, 0.5);
    float* v = fvec((size_t)H, 1.0);
    double* h0 = dvec((size_t)B * H, 0.3);
    double* c0 = dvec((size_t)B * H, 0.3);
    double* h = dvec((size_t)B * H, 0.0);
    double* c = dvec((size_t)B * H, 0.0);
    double* seq = dvec((size_t)B * T * H, 0.0);
    double* dh = dvec((size_t)B * H, 1.0);
    double* dc = dvec((size_t)B * H, 1.0);
    double* dseq = dvec((size_t)B * T * H, 1.0);
    double* dx = dvec((size_t)B * T * D, 0.0);
    double* dW = dvec((size_t)D * G4, 0.0);
    double* dU = dvec((size_t)H * G4, 0.0);
    double* db = dvec(G4, 0.0);
    double* dbhh = dvec(G3, 0.0);
    double* dh0 = dvec((size_t)B * H, 0.0);
    double* dc0 = dvec((size_t)B * H, 0.0);
    int32_t* steps = (int32_t*)malloc((size_t)B * sizeof(int32_t));
    int64_t n = 0;
    for (int literal = 0; literal < 2; ++literal) {
        expect(lstm_oracle_forward(B, T, D, H, x, L, W, U, bias, h0, c0, h, c, literal, threads, &n),
               0, "forward", B, T, D, H);
        expect(lstm_oracle_forward_seq(B, T, D, H, x, L, W, U, bias, h0, c0, h, c, literal, threads,
                                       &n, seq), 0, "forward_seq", B, T, D, H);
        expect(lstm_oracle_forward_gru(B, T, D, H, x, L, W, U, bias, bhh, h0, c0, h, c, literal,
                                       threads, &n, seq), 0, "forward_gru", B, T, D, H);
        expect(lstm_oracle_forward_rnn(B, T, D, H, x, L, W, U, bias, h0, c0, h, c, literal, threads,
                                       &n, seq), 0, "forward_rnn", B, T, D, H);
    }
    for (int cell = 0; cell < 3; ++cell)
        expect(lstm_oracle_forward_stop(B, T, D, H, x, L, W, U, bias, bhh, cell, v, -0.1, h0, c0, h,
                                        c, steps, &n, seq, threads), 0, "forward_stop", B, T, D, H);
    expect(lstm_oracle_backward(B, T, D, H, x, L, W, U, bias, h0, c0, dh, dc, dseq, dx, dW, dU, db,
                                dh0, dc0, threads), 0, "backward", B, T, D, H);
    expect(lstm_oracle_backward(B, T, D, H, x, L, W, U, bias, h0, c0, dh, dc, NULL, dx, dW, dU, db,
                                dh0, dc0, threads), 0, "backward (no dseq)", B, T, D, H);
    expect(lstm_oracle_backward_cell(B, T, D, H, 1, x, L, W, U, bias, bhh, h0, dh, dseq, dx, dW,
                                     dU, db, dbhh, dh0, threads), 0, "backward_gru", B, T, D, H);
    expect(lstm_oracle_backward_cell(B, T, D, H, 2, x, L, W, U, bias, NULL, h0, dh, NULL, dx, dW,
                                     dU, db, NULL, dh0, threads), 0, "backward_rnn", B, T, D, H);
    /* rejected inputs leave the outputs untouched and return their codes */
    if (B > 1 && T > 0) {
        const int32_t keep = L[1];
        L[1] = T + 1;
        expect(lstm_oracle_forward(B, T, D, H, x, L, W, U, bias, h0, c0, h, c, 0, threads, &n), 2,
               "forward, length past T", B, T, D, H);
        expect(lstm_oracle_backward(B, T, D, H, x, L, W, U, bias, h0, c0, dh, dc, dseq, dx, dW, dU,
                                    db, dh0, dc0, threads), 2, "backward, length past T", B, T, D, H);
        L[1] = -1;
        expect(lstm_oracle_forward_stop(B, T, D, H, x, L, W, U, bias, bhh, 0, v, -0.1, h0, c0, h, c,
                                        steps, &n, seq, threads), 2, "forward_stop, negative length",
               B, T, D, H);
        L[1] = keep;
    }
    expect(lstm_oracle_forward(B, T, D, H, NULL, L, W, U, bias, h0, c0, h, c, 0, threads, &n), 1,
           "forward, null x", B, T, D, H);
    expect(lstm_oracle_backward_cell(B, T, D, H, 1, x, L, W, U, bias, NULL, h0, dh, dseq, dx, dW,
                                     dU, db, dbhh, dh0, threads), 1, "backward_gru, null b_hh",
           B, T, D, H);
    free(x); free(L); free(W); free(U); free(bias); free(bhh); free(v); free(h0); free(c0);
    free(h); free(c); free(seq); free(dh); free(dc); free(dseq); free(dx); free(dW); free(dU);
    free(db); free(dbhh); free(dh0); free(dc0); free(steps);
}

int main(void) {
    static const int shapes[][4] = {
        {1, 1, 1, 1}, {1, 3, 1, 1}, {3, 5, 2, 3}, {4, 6, 7, 5}, {7, 4, 3, 9}, {2, 9, 1, 16},
    };
    for (size_t i = 0; i < sizeof(shapes) / sizeof(shapes[0]); ++i)
        for (int threads = 1; threads <= 3; threads += 2) {
            run_case(shapes[i][0], shapes[i][1], shapes[i][2], shapes[i][3], 0, threads);
            run_case(shapes[i][0], shapes[i][1], shapes[i][2], shapes[i][3], 1, threads);
        }
    run_case(3, 0, 2, 2, 1, 1);   /* T = 0: no steps at all */
    if (failures) {
        fprintf(stderr, "%d unexpected statuses\n", failures);
        return 1;
    }
    printf("oracle sanitizer run: ok\n");
    return 0;
}
