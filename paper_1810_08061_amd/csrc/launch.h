// launch.h -- host-side launchers of the kernels (one translation unit per
// kernel family) and the device workspace they share.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace ldyn {

// Device workspace of one handle (all pointers into one hipMalloc block).
struct Workspace {
    Meta* meta;         // loop bound, row count, status
    int32_t* perm;      // [B] slot -> batch index; slots sorted by length, descending (stable)
    int32_t* offsets;   // [T_max + 1] first compact row of step t; offsets[t+1]-offsets[t] = active rows
    int32_t* rowsrc;    // [B * T_max] compact row -> b * T_max + t
    float* gx;          // [B * T_max][4H] x W + b for valid (b, t), gate-interleaved columns
    void* hx;           // [4][bpad][hpad] recurrent operand (dtype), slot order; row-major in two
                        // buffers for the per-step path, MFMA fragment order in four for the persistent loop
    unsigned* bar;      // grid-barrier counters: [0] global, [64 * (1 + x)] group x (zeroed by prep)
    float* z;           // [bpad][4H] per-step pre-activations (per-step mode only)
    void* wt;           // bf16: W transposed to [np][dp] (gate-interleaved rows, zero padded)
    int32_t* stopped;   // [B] per-step path, termination from the state: 1 once row b ended
    int32_t* running;   // [T_max] per-step path: rows still running after step t
};

struct Dims {
    int B, D, H, T;     // batch, input width, hidden width, padded time extent
    int bf16;           // 1: x, W, U are bf16; 0: fp32
    int hpad, bpad;     // padded hidden width / batch rows of the operand buffer
    int cell;           // CellKind; GRU and RNN weights are packed into the LSTM's four gate blocks
};

// GRU and RNN: the caller's weights packed into the four gate blocks of the
// LSTM path (d.cell selects the packing).  GRU: W [D][3H], U [H][3H] (gate
// blocks r, u, n), b [6H] = b_ih ++ b_hh -> W4 [D][4H] = (W_r, W_u, 0, W_n),
// U4 [H][4H] = (U_r, U_u, U_n, 0), b4 [4H] = (b_ir + b_hr, b_iu + b_hu, b_hn,
// b_in).  RNN: W [D][H], U [H][H], b [H] -> (W, 0, 0, 0), (U, 0, 0, 0),
// (b, 0, 0, 0).
hipError_t launch_cell_pack(const Dims& d, const void* W, const void* U, const float* b, void* W4,
                            void* U4, float* b4, hipStream_t s);

// Preparation: clamp and validate lengths, stable descending length sort,
// per-step active counts and compact row offsets, compact row sources.
hipError_t launch_prep(const Dims& d, const int32_t* lengths, const Workspace& ws, hipStream_t s);

// The workspace of a persistent-mode LSTM forward carved from caller memory
// (api.hip): returns its bytes; fills ws when base is not null.
long long carve_forward_workspace(const Dims& d, char* base, Workspace* ws, long long* hx_off,
                                  long long* hx_bytes);

// Input projection over all valid (b, t): gx[r][c'] = x[rowsrc[r]] . W[:, col(c')] + b[col(c')].
hipError_t launch_inproj(const Dims& d, const void* x, const void* W, const float* b,
                         const Workspace& ws, int grid, hipStream_t s);

// bf16 input projection: W -> Wt, then the tiled GEMM (inproj.hip).
void inproj_bf16_wt_shape(const Dims& d, int* np, int* dp);
int inproj_bf16_tiles_max(const Dims& d);
hipError_t inproj_bf16_setup();
hipError_t launch_transpose_w(const Dims& d, const void* W, const Workspace& ws, hipStream_t s);
hipError_t launch_inproj_bf16(const Dims& d, const void* x, const float* b, const Workspace& ws,
                              int grid, hipStream_t s);

// Persistent on-device time loop.
// Termination computed from the state: a row ends after a step that leaves
// its halting score v . h + c positive.
struct StopArgs {
    const float* v;          // [H]
    float c;
    int32_t* steps;          // [B] (batch order), written: the steps each row ran
    const int32_t* lengths;  // [B] caps
};

struct PersistentConfig {
    int mt, groups, ksw, kw, nst, lds_bytes;
    unsigned long long timeout_ticks;  // barrier wait bound in wall-clock ticks
    unsigned long long* trace;         // per-step timestamps (diagnostics) or null
    float* seq;                        // output sequence [B][T][H]: each step's h of the rows that
                                       // ran it (zeros past them written afterwards), or null
    const StopArgs* stop;              // termination from the state, or null
    float* save_h;                     // forward for training: the state each step starts from,
    float* save_c;                     // [compact rows][H] (z is kept in place of Gx); else null
};
constexpr int BAR_WORDS = 64 * 9;  // global + 8 group counters, 256 bytes apart
hipError_t launch_persistent(const Dims& d, const PersistentConfig& pc, const void* U,
                             const float* h0, const float* c0, float* out_h, float* out_c,
                             const Workspace& ws, hipStream_t s);
// Occupancy check for the co-resident grid; returns blocks per CU (0 if none).
// mode: 0 plain, 1 termination from the state, 2 forward for training
int persistent_blocks_per_cu(int bf16, int mt, int ksw, int kw, int nst, int lds_bytes, int cell,
                             int mode);
// Compiled variant with exactly (mt, kw, ksw) and the smallest state capacity >= nstate.
bool persistent_pick_variant(int bf16, int mt, int kw, int ksw, int nstate, int* nst);
int persistent_lds_bytes(int bf16, int mt, int kw, int nst, int hpad);

// Whole forward in one single-workgroup launch (H <= 32).
bool small_pick(int bf16, int B, int D, int H, int* kd, int* nt);
hipError_t launch_small(const Dims& d, int kd, int nt, const void* x, const int32_t* lengths,
                        const void* W, const void* U, const float* b, const float* h0,
                        const float* c0, float* out_h, float* out_c, float* seq,
                        const StopArgs* stop, const Workspace& ws, hipStream_t s);

// Per-step comparison path.
hipError_t launch_step_init(const Dims& d, const float* h0, const float* c0, float* out_h,
                            float* out_c, const Workspace& ws, hipStream_t s);
hipError_t launch_step_gemm(const Dims& d, int t, const void* U, const Workspace& ws, hipStream_t s);
hipError_t launch_step_gates(const Dims& d, int t, float* out_h, float* out_c, float* seq,
                             bool stop, const Workspace& ws, hipStream_t s,
                             float* save_h = nullptr, float* save_c = nullptr);
// Termination from the state on the per-step path: init (steps = caps, no row
// ended, counters zero), then after the gates of each step the halting scores
// of the rows that ran; running[t] counts the rows that run at step t + 1.
hipError_t launch_step_stop_init(const Dims& d, const StopArgs& stop, const Workspace& ws,
                                 hipStream_t s);
hipError_t launch_step_stop(const Dims& d, int t, const StopArgs& stop, const Workspace& ws,
                            hipStream_t s);

// Backward pass (bwd.hip).
hipError_t launch_bwd_weights(const Dims& d, const void* W, int rows, float* Wil, hipStream_t s);
hipError_t launch_bwd_init(const Dims& d, const float* dh_out, const float* dc_out, float* dH,
                           float* dC, const Workspace& ws, hipStream_t s);
// off, act: the step's first compact row and its number of rows (known to the
// host from the forward's step offsets).
hipError_t launch_bwd_cell(const Dims& d, int t, int off, int act, const float* save_h,
                           const float* save_c,
                           const float* dseq, float* dH, float* dC, const Workspace& ws,
                           hipStream_t s);
// GRU/RNN gradients, packed four-block (interleaved) layout -> the cell's own;
// part 0: input side (W, b_ih / b), 1: recurrent side (U, b_hh).
hipError_t launch_bwd_unpack(const Dims& d, const float* il, float* out, int rows, int part,
                             hipStream_t s);
hipError_t launch_bwd_state_out(const Dims& d, const float* dH, const float* dC, const float* srow,
                                float* dh0, float* dc0, const Workspace& ws, hipStream_t s);
// bf16 data: the cell's backward with one workgroup per row, also writing the
// row's dz in fp16 scaled by a power of two (srow) for dz U^T.
hipError_t launch_bwd_cell16(const Dims& d, int t, int off, int act, const float* save_h,
                             const float* save_c, const float* dseq, float* dH, float* dC,
                             float* srow, _Float16* dz16, const Workspace& ws, hipStream_t s);
hipError_t launch_bwd_ones(float* a, int n, hipStream_t s);
// bf16 data: the reverse loop over steps max_len - 1 .. t_end in one
// cooperative launch (one workgroup of 8 units per CU, those units' rows of U
// in LDS, each step's dz published in fp16 with a power-of-two scale per row
// and 32-column block, one grid barrier per step), leaving in dH the
// gradient entering step t_end - 1.  bwd_loop_fits: its workgroup count, or
// 0 where it does not apply (H odd, below 16 or above 2048, more than 512
// rows, not all resident).
// dzx [2][bpad][kp] fp16, dzs [2][bpad][nblk] and bar [9 * 64] must be zero
// at the launch; dH, dC hold the upstream gradients (slot order) and receive
// dh0, dc0.
int bwd_loop_fits(const Dims& d, int num_cus);
void bwd_loop_shape(int H, int* kp, int* nblk);
hipError_t launch_bwd_loop(const Dims& d, const _Float16* u16, float alpha_u, const float* save_h,
                           const float* save_c, const float* dseq, float* dH, float* dC,
                           _Float16* dzx, float* dzs, unsigned* bar, unsigned long long timeout_ticks,
                           int t_end, const Workspace& ws, hipStream_t s);
// bf16 data, H a multiple of 256 (at most 2048): the whole reverse loop in one
// cooperative launch (H / 8 workgroups, each with a 32-unit x H-column block
// of U in registers; per step the blocks' shares of dh = dz U^T, then the
// cell's backward of 8 units, each exchange polled for, no grid barrier),
// leaving dh0 and dc0 in dH and dC.  bwd_block_fits: its workgroup count, or
// 0 where it does not apply.  dzx [4][bpad][4H] fp16, dzs [4][bpad][H / 8]
// and pdh [4][4][bpad][H] must be all ones (the marker) at the launch; trace
// [T + 1][4] or null.  amax_dz receives the largest |dz| over all compact
// rows (float bits, atomic maximum: it must hold 0 or a lower bound).
int bwd_block_fits(const Dims& d, int num_cus);
hipError_t launch_bwd_block(const Dims& d, const _Float16* u16, float alpha_u, const float* save_h,
                            const float* save_c, const float* dseq, float* dH, float* dC, _Float16* dzx,
                            float* dzs, float* pdh, unsigned* amax_dz, unsigned long long timeout_ticks,
                            unsigned long long* trace, const Workspace& ws, hipStream_t s);
// xc = the compact rows of x in fp32; amax (or null) receives the largest
// |x| of them, as float bits, by atomic maximum.
hipError_t launch_bwd_gather_x(const Dims& d, const void* x, long rows, float* xc, unsigned* amax,
                               const Workspace& ws, hipStream_t s);
// fp16 operands of the backward's GEMMs: the largest magnitude (as float bits,
// atomic and order free) and a scaled conversion.
hipError_t launch_bwd_absmax(const float* a, long n, unsigned* out, hipStream_t s);
hipError_t launch_bwd_to_f16(const float* src, _Float16* dst, long n, float scale, hipStream_t s);
// db = column sums of dz [rows][ncols] (ncols a multiple of 4) through
// part [BWD_CS_CHUNKS][ncols]; with dz16, also dz16 = fp16(dz * scale).
constexpr int BWD_CS_CHUNKS = 64;
hipError_t launch_bwd_colsum(const float* dz, long rows, int ncols, float* part, float* out,
                             _Float16* dz16, float scale, hipStream_t s);
hipError_t launch_bwd_permute(const Dims& d, const float* il, float* out, int rows, hipStream_t s);
hipError_t launch_bwd_dx(const Dims& d, const float* dxc, long rows, const int32_t* lengths,
                         float* dx, const Workspace& ws, hipStream_t s);
// Forward for training from the saved state: out_seq[b][t] for t < L[b]
// (the state after step t is the one step t + 1 started from, or out_h).
hipError_t launch_seq_from_saved(const Dims& d, float* seq, const float* save_h, const float* out_h,
                                 const int32_t* lengths, const Workspace& ws, int num_cus,
                                 hipStream_t s);

// Output sequence: zeros past each row's last step (lengths: that step + 1;
// the loops write the valid steps themselves).
hipError_t launch_seq_finish(const Dims& d, float* seq, const int32_t* lengths, int num_cus,
                             hipStream_t s);

}  // namespace ldyn
