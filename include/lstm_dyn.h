/*
 * lstm_dyn.h -- C ABI of the MI355X (gfx950) variable-length LSTM time loop.
 *
 * The operation (AutoGraph paper, Section 9 "RNN cells", and its hand-written
 * graph form in Appendix A): starting from (h0, c0), run an LSTM cell over the
 * batch for t = 0, 1, ... while any sequence still has steps left; a sequence
 * whose length L[b] has been reached keeps its state unchanged (a per-row
 * select); the loop stops after max_b L[b] steps.  The result is the final
 * state (h, c) of every sequence.  The paper leaves the cell abstract; here it
 * is the standard LSTM with one bias vector and gate blocks (i, f, g, o):
 *
 *     z  = x[b, t] W + h U + b
 *     c' = sigmoid(z_f) * c + sigmoid(z_i) * tanh(z_g)
 *     h' = sigmoid(z_o) * tanh(c')
 *
 * Layouts (all row-major, contiguous, caller-owned DEVICE memory):
 *     x        [B][T_max][D]   element type = dtype (fp32 or bf16)
 *     lengths  [B]             int32, each expected in [0, T_max]
 *     W        [D][4H]         element type = dtype
 *     U        [H][4H]         element type = dtype
 *     b        [4H]            fp32
 *     h0, c0   [B][H]          fp32
 *     out_h, out_c [B][H]      fp32 (written)
 * Gate blocks along 4H are i = [0, H), f = [H, 2H), g = [2H, 3H), o = [3H, 4H).
 * With bf16 data, x W is formed from bf16 operands; the recurrent product h U
 * from fp16 operands (U widened from bf16, exact for 2^-14 <= |U| <= 65504;
 * h rounded to fp16, so h0 entries must lie within +-65504); every product
 * is accumulated in fp32 and the state (h, c) is kept in fp32.
 *
 * Threading: a handle may be used from one host thread at a time, and one
 * forward may be in flight per handle.  Forward calls only enqueue work on the
 * given stream (a hipStream_t; NULL = the default stream); inputs and outputs
 * must stay valid until that work completes.
 *
 * Error classes mirror the paper's split of failures (Appendix B): argument
 * problems found on the host are reported synchronously (LSTM_DYN_ERR_INVALID,
 * LSTM_DYN_ERR_UNSUPPORTED); problems in device data (lengths outside
 * [0, T_max]) are clamped for memory safety and reported by
 * lstm_dyn_query(LSTM_DYN_Q_LAST_STATUS) after the forward has run.
 */
#ifndef LSTM_DYN_H
#define LSTM_DYN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lstm_dyn lstm_dyn_t; /* opaque handle */

/* Element type of x, W and U. */
enum { LSTM_DYN_F32 = 0, LSTM_DYN_BF16 = 1 };

/* Execution mode.
 * PERSISTENT: the time loop runs on the device inside one persistent kernel
 *   (one grid barrier at its start, then each step waits only for the hidden
 *   state it reads; loop bound and early exit read on the device).  Launches
 *   per forward: length preparation, input projection (two launches with
 *   bf16 data: a transpose of W, then the GEMM), the loop; one more for the
 *   GRU and RNN cells (their weights are repacked); a single launch when the
 *   hidden width is at most 32 and the whole forward fits one workgroup.
 *   None of them waits for the host.
 * PER_STEP: the comparison path of the paper's eager-vs-graph experiment
 *   (Section 9, Table 1): the loop bound is copied to the host (one
 *   synchronisation), then the host issues two kernel launches per step. */
enum { LSTM_DYN_PERSISTENT = 0, LSTM_DYN_PER_STEP = 1 };

/* Recurrent cell run by the loop (lstm_dyn_create_cell).
 * LSTM: the cell above (the default of lstm_dyn_create).
 * GRU:  the gated recurrent unit, the other common cell the paper's RNN loop
 *   (Section 9 "RNN cells") can run; gate blocks (r, u, n) along 3H and two
 *   bias vectors, b = [b_ih (3H) ++ b_hh (3H)]:
 *       a = x[b, t] W + b_ih,   e = h U + b_hh
 *       r = sigmoid(a_r + e_r),  u = sigmoid(a_u + e_u)
 *       n = tanh(a_n + r * e_n)
 *       h' = (1 - u) * n + u * h
 *   Layouts: W [D][3H], U [H][3H] (element type = dtype), b [6H] fp32.
 * RNN:  the plain tanh recurrent cell with one bias vector,
 *       h' = tanh(x[b, t] W + h U + b)
 *   Layouts: W [D][H], U [H][H] (element type = dtype), b [H] fp32.
 * GRU and RNN have no cell state: c0 is ignored (may be NULL) and out_c is
 * written with zeros. */
enum { LSTM_DYN_CELL_LSTM = 0, LSTM_DYN_CELL_GRU = 1, LSTM_DYN_CELL_RNN = 2 };

/* Status codes. */
enum {
    LSTM_DYN_OK = 0,
    LSTM_DYN_ERR_INVALID = 1,     /* NULL handle/pointer, bad sizes, misaligned or overlapping buffers */
    LSTM_DYN_ERR_HIP = 2,         /* a HIP runtime call failed */
    LSTM_DYN_ERR_NOMEM = 3,       /* device workspace allocation failed */
    LSTM_DYN_ERR_UNSUPPORTED = 4, /* sizes outside what the compiled kernel variants cover */
    LSTM_DYN_ERR_BAD_LENGTHS = 5, /* (device status) a length was outside [0, T_max] and was clamped */
    LSTM_DYN_ERR_TIMEOUT = 6,     /* (device status) a wait of a cooperative kernel exceeded its bound */
    LSTM_DYN_ERR_TOO_LARGE = 7    /* lstm_dyn_forward_noalloc: the workspace exceeds its scratch */
};

/* lstm_dyn_query selectors. */
enum {
    LSTM_DYN_Q_LAST_STATUS = 0,        /* status of the last forward (synchronises its stream) */
    LSTM_DYN_Q_STEPS_EXECUTED = 1,     /* loop iterations of the last forward = max_b L[b] (synchronises) */
    LSTM_DYN_Q_LAUNCHES_PER_FORWARD = 2, /* kernel launches issued by the last forward */
    LSTM_DYN_Q_GROUPS = 3,             /* workgroups of the persistent kernel */
    LSTM_DYN_Q_WORKSPACE_BYTES = 4,    /* device workspace owned by the handle */
    LSTM_DYN_Q_TOTAL_ROWS = 5,         /* sum of the (clamped) lengths of the last forward (synchronises) */
    LSTM_DYN_Q_TIME_PREP_NS = 6,       /* with LSTM_DYN_OPT_TIMING: device time of the length
                                          preparation kernel (and, for a GRU or RNN handle, the weight
                                          repacking) in the last forward (synchronises) */
    LSTM_DYN_Q_TIME_INPROJ_NS = 7,     /* ... of the input projection GEMM */
    LSTM_DYN_Q_TIME_LOOP_NS = 8        /* ... of the time loop (the persistent kernel, or the
                                          per-step path's host loop of launches) */
};

/* lstm_dyn_set_option selectors. */
enum {
    LSTM_DYN_OPT_TIMING = 0,    /* 1: record HIP events on the forward's stream around each phase */
    LSTM_DYN_OPT_STEP_TRACE = 1, /* 1: the persistent kernel records device wall-clock
                                    timestamps within each step (diagnostics) */
    LSTM_DYN_OPT_TIMEOUT_US = 2  /* bound, in microseconds, of every wait of the
                                    cooperative kernels (grid barriers, polls for
                                    other workgroups' data); 0 restores the default of
                                    5 s, at most 60 s.  Past it a kernel stops, sets
                                    LSTM_DYN_ERR_TIMEOUT (LSTM_DYN_Q_LAST_STATUS) and
                                    exits normally */
};

/* Launch plan of a handle: pure host arithmetic, no device access. */
typedef struct {
    int mt;             /* 16-column gate tiles per workgroup (4 hidden units each) */
    int groups;         /* workgroups of the persistent kernel (at most one per CU) */
    int ksw;            /* MFMA K-steps per wave over the hidden width */
    int kw;             /* waves per workgroup (they split the hidden width) */
    int hpad;           /* hidden width padded to the recurrent MFMA's K granularity */
    int bpad;           /* batch padded to 16 rows */
    int lds_bytes;      /* dynamic LDS of the persistent kernel */
    int nstate;         /* (row tile, gate tile) pairs held per wave */
    long long workspace_bytes; /* device workspace a handle allocates */
    int single;         /* 1: persistent mode runs the whole forward as one launch of a
                           single workgroup (hidden width <= 32); groups is then 1 */
    int single_kd;      /* K-step capacity over D of that kernel */
    int single_nt;      /* 16-row tiles of that kernel */
} lstm_dyn_plan_t;

/*
 * lstm_dyn_create: validate sizes, choose a plan for the current HIP device
 * and allocate the handle's device workspace (hipMalloc; freed by destroy).
 *   B >= 1, D >= 1, H >= 1, T_max >= 1; dtype LSTM_DYN_F32/BF16; mode
 *   LSTM_DYN_PERSISTENT/PER_STEP.  *out receives the handle (NULL on error).
 * Sizes covered: B <= 8192 and B * T_max < 2^31; one workgroup per compute
 * unit owns 4 hidden units (fp32 data, and bf16 data with H <= 1024) or 8
 * (bf16 data, H > 1024), so H <= 4 x CUs with fp32 data and H <= 8 x CUs
 * with bf16 data (1024 and 2048 on a 256-CU device), in either mode; the
 * persistent mode also holds at most 512 rows.  lstm_dyn_plan gives the
 * answer for a device without a handle.
 * Returns LSTM_DYN_OK, ERR_INVALID (bad arguments; no HIP call is made),
 * ERR_UNSUPPORTED (sizes the compiled kernel variants do not cover), ERR_HIP, ERR_NOMEM.
 */
int lstm_dyn_create(lstm_dyn_t** out, int B, int D, int H, int T_max, int dtype, int mode);

/*
 * lstm_dyn_create_cell: lstm_dyn_create for the cell `cell` (LSTM_DYN_CELL_*).
 * A GRU or RNN handle takes that cell's layouts above in lstm_dyn_forward
 * and lstm_dyn_forward_seq; its forward first repacks W, U and b into the
 * handle's workspace (one more kernel launch), so the loop kernels see the
 * LSTM's four gate blocks (the RNN's three unused blocks hold zeros).  Returns as lstm_dyn_create; an unknown cell is
 * ERR_INVALID.
 */
int lstm_dyn_create_cell(lstm_dyn_t** out, int B, int D, int H, int T_max, int dtype, int mode,
                         int cell);

/*
 * lstm_dyn_forward: enqueue one forward of the loop on `stream`.
 * Pointer arguments are caller-owned device buffers with the layouts above;
 * x, W and U must be 16-byte aligned, the others 4-byte aligned.  Outputs may
 * alias their own initial state exactly (out_h == h0, out_c == c0); any other
 * overlap between an output and an input or the other output is ERR_INVALID.
 * Persistent mode never synchronises with the host; per-step mode performs
 * exactly one device-to-host copy of the loop bound.
 */
int lstm_dyn_forward(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                     const void* U, const float* b, const float* h0, const float* c0,
                     float* out_h, float* out_c, void* stream);

/*
 * lstm_dyn_forward_seq: lstm_dyn_forward, and also the output sequence.  The
 * paper's loop (Section 9 "RNN cells"; Appendix A) appends the cell's output
 * at every step; here
 *     out_seq [B][T_max][H] fp32 (caller-owned device memory, 4-byte aligned,
 *     written in full): out_seq[b][t] = the hidden state of sequence b after
 *     step t for t < L[b] (so out_seq[b][L[b]-1] = out_h[b]), and zero for
 *     t >= L[b] (no output is defined past a sequence's length; zero is the
 *     padding chosen).  Lengths outside [0, T_max] are clamped as in
 *     lstm_dyn_forward.
 * out_seq may not overlap any other argument.  One more kernel launch than
 * lstm_dyn_forward (it writes the zeros past each length; the loop writes
 * the valid steps).  Returns as lstm_dyn_forward.
 */
int lstm_dyn_forward_seq(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                         const void* U, const float* b, const float* h0, const float* c0,
                         float* out_h, float* out_c, float* out_seq, void* stream);

/*
 * lstm_dyn_forward_stop: the loop with its termination computed on the device
 * from the state.  The paper's decoders (beam search, seq2seq; Appendix D)
 * leave their loop once every candidate sequence has terminated; here a
 * sequence terminates when a linear read-out of its hidden state, the halting
 * score
 *     s = v . h + stop_c        (v = stop_v [H] fp32, device memory),
 * is positive after one of its steps.  lengths[b] is now a cap: row b runs
 * step t while t < L[b] and it has not terminated; a terminated row keeps its
 * state.  The loop ends on the device at the first step in which no row runs
 * (lstm_dyn_query(LSTM_DYN_Q_STEPS_EXECUTED) gives the steps in which some
 * row ran).
 *     out_steps [B] int32 (written): the steps row b ran (<= its clamped cap).
 *     out_seq: NULL, or the output sequence as in lstm_dyn_forward_seq, zero
 *     from step out_steps[b] on.
 * The score is formed from h in the precision of the recurrent operand (fp16
 * with bf16 data, fp32 with fp32 data) and accumulated in fp32, so a score
 * within rounding of zero may be decided either way.  In per-step mode the
 * host reads the number of running rows after every step (the eager form of
 * the loop condition).  stop_v is 4-byte aligned and may not overlap an
 * output; out_steps is 4-byte aligned and may not overlap any argument; NaN
 * stop_c is ERR_INVALID.  Returns as lstm_dyn_forward, or ERR_UNSUPPORTED if
 * the persistent variant with the halting score does not fit the device for
 * this handle's sizes.
 */
int lstm_dyn_forward_stop(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                          const void* U, const float* b, const float* h0, const float* c0,
                          const float* stop_v, float stop_c, float* out_h, float* out_c,
                          int32_t* out_steps, float* out_seq, void* stream);

/*
 * lstm_dyn_forward_train: lstm_dyn_forward, also keeping in the handle what
 * lstm_dyn_backward needs: for every valid (b, t), the cell's pre-activations
 * and the state the step started from (fp32).  The first call
 * allocates that training workspace (hipMalloc; about 8 B*T_max*H + 4 B*T_max*D
 * + 32 (D+H) H bytes, freed by destroy).  out_seq may be NULL, or receives the
 * output sequence as in lstm_dyn_forward_seq.  out_h/out_c may not alias
 * h0/c0 (the backward reads h0, c0).  Any other forward on the handle
 * discards what was kept.  Returns as lstm_dyn_forward.
 */
int lstm_dyn_forward_train(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                           const void* U, const float* b, const float* h0, const float* c0,
                           float* out_h, float* out_c, float* out_seq, void* stream);

/*
 * lstm_dyn_backward: gradients of a loss through the masked loop
 * (backpropagation through time; the paper trains its staged models
 * in-graph, Section 9), after lstm_dyn_forward_train on the same handle with
 * the same inputs (x, lengths, W, U, b, h0, c0 -- the caller keeps them).
 * Upstream gradients: d_out_h, d_out_c [B][H] fp32 (of out_h, out_c) and
 * d_seq [B][T_max][H] fp32 of the output sequence, or NULL (entries at
 * t >= L[b] have no effect).  Written, all fp32, caller-owned device memory,
 * 4-byte aligned: dx [B][T_max][D] (zero at t >= L[b]), dW, dU and db
 * in the layouts of the handle's cell (LSTM [D][4H], [H][4H], [4H]; GRU
 * [D][3H], [H][3H], [6H] = d b_ih ++ d b_hh; RNN [D][H], [H][H], [H]), dh0
 * and dc0 [B][H]; no output may overlap another argument.  GRU and RNN
 * handles have no cell state: c0 and d_out_c are ignored and dc0 may be
 * NULL (else zeros).  A step a row does not take passes its state through
 * unchanged, so its gradient is the identity.  Step t's dz comes from the
 * kept pre-activations; dh <- dz U^T and the weight gradients (sums over all
 * valid steps) are products with fp32 accumulation, of fp32 operands with
 * fp32 data and of fp16 operands with bf16 data (each scaled by a power of
 * two: U and the weight-gradient operands as a whole, dz per row or per row
 * and 32-column block).  Synchronises once with the host (the step offsets),
 * then issues two launches per step; a persistent handle with bf16 data (H
 * even, 16 <= H <= 2048, B <= 512) takes the steps with at most 16 rows in
 * one cooperative launch with a bounded grid barrier per step (a timeout
 * shows in LSTM_DYN_Q_LAST_STATUS).  Consumes what the forward kept (a
 * second backward needs another forward for training).  Returns LSTM_DYN_OK,
 * ERR_INVALID (bad arguments, or no forward for training kept), ERR_HIP.
 */
int lstm_dyn_backward(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                      const void* U, const float* b, const float* h0, const float* c0,
                      const float* d_out_h, const float* d_out_c, const float* d_seq, float* dx,
                      float* dW, float* dU, float* db, float* dh0, float* dc0, void* stream);

/* Free the handle and its workspace.  Waits for the stream of the handle's
 * last forward or backward (the only work that may use the workspace), not
 * for the whole device; the runtime's free may still wait for the device.
 * NULL is a no-op. */
int lstm_dyn_destroy(lstm_dyn_t* h);

/* Read a property of the handle or of its last forward (see LSTM_DYN_Q_*). */
int lstm_dyn_query(lstm_dyn_t* h, int what, long long* value);

/* Set a handle option (see LSTM_DYN_OPT_*).  Returns LSTM_DYN_OK, ERR_INVALID or ERR_HIP. */
int lstm_dyn_set_option(lstm_dyn_t* h, int option, long long value);

/*
 * lstm_dyn_step_trace: with LSTM_DYN_OPT_STEP_TRACE set, copy the last
 * forward's step timestamps of workgroup 0 (device wall-clock ticks; four per
 * step -- step start, partial products of the first row-tile chunk done,
 * state update and h stores done, first row tile of h_t complete (the end of
 * the wait for the other workgroups) -- then the loop end) into
 * ticks[0 .. capacity), synchronising the forward's stream; *count receives
 * the number of entries and *khz the clock rate.  A backward pass run as
 * one launch of the whole reverse loop (bf16 data, persistent handle, H a
 * multiple of 256) records there instead, at 4 t for step t: its start, its
 * share of dh published, its cells done (the other shares awaited), the
 * marks for later steps issued; at 4 max_len the product for dh0.
 * Returns LSTM_DYN_OK, ERR_INVALID (option not set, NULL arguments) or ERR_HIP.
 */
int lstm_dyn_step_trace(lstm_dyn_t* h, long long* ticks, int capacity, int* count, int* khz);

/* Static description of a status code (never NULL). */
const char* lstm_dyn_strerror(int status);

/*
 * lstm_dyn_plan: the plan lstm_dyn_create would choose for a device with
 * `num_cus` compute units.  Host arithmetic only.  Returns LSTM_DYN_OK,
 * ERR_INVALID or ERR_UNSUPPORTED.
 */
int lstm_dyn_plan(int B, int D, int H, int T_max, int dtype, int mode, int num_cus,
                  lstm_dyn_plan_t* out);

/*
 * lstm_dyn_check_args: the host-side argument checks of lstm_dyn_forward
 * (NULL pointers, alignment, overlap) for the given sizes, without touching
 * the pointed-to memory.  Returns LSTM_DYN_OK or ERR_INVALID.
 */
int lstm_dyn_check_args(int B, int D, int H, int T_max, int dtype, const void* x,
                        const int32_t* lengths, const void* W, const void* U, const float* b,
                        const float* h0, const float* c0, const float* out_h, const float* out_c);

/* lstm_dyn_check_args, and the checks of out_seq for lstm_dyn_forward_seq
 * (NULL, 4-byte alignment, overlap with any other argument). */
int lstm_dyn_check_seq_args(int B, int D, int H, int T_max, int dtype, const void* x,
                            const int32_t* lengths, const void* W, const void* U, const float* b,
                            const float* h0, const float* c0, const float* out_h,
                            const float* out_c, const float* out_seq);

/* The checks of lstm_dyn_forward (out_seq NULL) or lstm_dyn_forward_seq
 * (out_seq not NULL) for a handle of cell `cell`, with that cell's sizes of
 * W, U and b.  Returns LSTM_DYN_OK or ERR_INVALID. */
int lstm_dyn_check_cell_args(int B, int D, int H, int T_max, int dtype, int cell, const void* x,
                             const int32_t* lengths, const void* W, const void* U, const float* b,
                             const float* h0, const float* c0, const float* out_h,
                             const float* out_c, const float* out_seq);

/* The checks of lstm_dyn_forward_stop for a handle of cell `cell` (out_seq
 * may be NULL).  Returns LSTM_DYN_OK or ERR_INVALID. */
int lstm_dyn_check_stop_args(int B, int D, int H, int T_max, int dtype, int cell, const void* x,
                             const int32_t* lengths, const void* W, const void* U, const float* b,
                             const float* h0, const float* c0, const float* stop_v,
                             const float* out_h, const float* out_c, const int32_t* out_steps,
                             const float* out_seq);

/* The argument checks of lstm_dyn_backward for the given sizes and cell
 * (LSTM_DYN_CELL_*: NULL, alignment, overlap), without touching the memory.
 * Returns LSTM_DYN_OK or ERR_INVALID. */
int lstm_dyn_check_backward_args(int B, int D, int H, int T_max, int dtype, int cell, const void* x,
                                 const int32_t* lengths, const void* W, const void* U,
                                 const float* b, const float* h0, const float* c0,
                                 const float* d_out_h, const float* d_out_c, const float* d_seq,
                                 const float* dx, const float* dW, const float* dU,
                                 const float* db, const float* dh0, const float* dc0);

/*
 * lstm_dyn_forward_noalloc: lstm_dyn_forward (LSTM cell, PERSISTENT mode)
 * without a handle, for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  It calls no hipMalloc, hipFree or other allocating routine;
 * the workspace lies in a fixed scratch array inside the library of
 * LSTM_DYN_NOALLOC_SCRATCH_BYTES on every device it runs on (held until the
 * process ends).  Sizes whose workspace (the input projection of all B *
 * T_max steps, 16 H bytes each, plus the tables and the hidden-state
 * buffers) does not fit return LSTM_DYN_ERR_TOO_LARGE before any work is
 * enqueued; with bf16 data, B = 64 and H = 512 fit up to T_max = 200.
 *   Arguments, layouts and results as for lstm_dyn_forward on a handle
 *   created with lstm_dyn_create(B, D, H, T_max, dtype, LSTM_DYN_PERSISTENT)
 *   (the same kernels: the results are the same bits).  status: NULL, or a
 *   caller-owned device int32 that receives the forward's device status
 *   (LSTM_DYN_OK, ERR_BAD_LENGTHS or ERR_TIMEOUT) when the work on the
 *   stream completes; it must not overlap any other argument.
 *   Returns LSTM_DYN_OK, ERR_INVALID (as lstm_dyn_forward's checks),
 *   ERR_UNSUPPORTED, ERR_TOO_LARGE or ERR_HIP.
 * Every call on one device uses that device's one scratch array: calls whose
 * work overlaps on one device (two streams, two host threads) race and give
 * undefined results; calls in order on one stream are safe.
 */
#define LSTM_DYN_NOALLOC_SCRATCH_BYTES (128LL << 20)
int lstm_dyn_forward_noalloc(int B, int D, int H, int T_max, int dtype, const void* x,
                             const int32_t* lengths, const void* W, const void* U, const float* b,
                             const float* h0, const float* c0, float* out_h, float* out_c,
                             int32_t* status, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LSTM_DYN_H */
