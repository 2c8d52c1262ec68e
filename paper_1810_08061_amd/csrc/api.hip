// api.hip -- the C ABI declared in include/lstm_dyn.h: argument checks,
// launch plan, workspace ownership and the two execution modes.
#include <math.h>
#include <new>
#include <stdint.h>
#include <string.h>
#include <type_traits>

#include <dlfcn.h>
#include <rocblas/rocblas.h>

#include "../../include/lstm_dyn.h"
#include "launch.h"

// rocBLAS serves the backward pass's plain GEMMs only.  It is loaded at the
// first forward for training, so processes that only run forwards never map
// it; it is never unloaded.
namespace {
struct RocblasApi {
    decltype(&rocblas_create_handle) create_handle;
    decltype(&rocblas_destroy_handle) destroy_handle;
    decltype(&rocblas_set_atomics_mode) set_atomics_mode;
    decltype(&rocblas_set_stream) set_stream;
    decltype(&rocblas_sgemm) sgemm;
    decltype(&rocblas_gemm_ex) gemm_ex;
};
RocblasApi g_rb;
bool g_rb_loaded = false;

bool load_rocblas() {
    if (g_rb_loaded) return true;
    void* lib = dlopen("librocblas.so.5", RTLD_NOW | RTLD_LOCAL);
    if (!lib) lib = dlopen("/opt/rocm/lib/librocblas.so.5", RTLD_NOW | RTLD_LOCAL);
    if (!lib) lib = dlopen("librocblas.so", RTLD_NOW | RTLD_LOCAL);
    if (!lib) return false;
    RocblasApi a;
    bool ok = true;
    auto sym = [&](auto& f, const char* name) {
        f = reinterpret_cast<std::remove_reference_t<decltype(f)>>(dlsym(lib, name));
        ok = ok && f != nullptr;
    };
    sym(a.create_handle, "rocblas_create_handle");
    sym(a.destroy_handle, "rocblas_destroy_handle");
    sym(a.set_atomics_mode, "rocblas_set_atomics_mode");
    sym(a.set_stream, "rocblas_set_stream");
    sym(a.sgemm, "rocblas_sgemm");
    sym(a.gemm_ex, "rocblas_gemm_ex");
    if (!ok) return false;
    g_rb = a;
    g_rb_loaded = true;
    return true;
}
}  // namespace

// Workspace of the forward for training and the backward pass, allocated at
// the first lstm_dyn_forward_train of a handle.
struct TrainWs {
    void* block;
    float* save_h;  // [B*T][H] the state each step started from, compact rows
    float* save_c;  // [B*T][H]
    float* xc;      // [B*T][D] x in compact rows (fp32), then the rows of dx
    float* w_il;    // [D][4H] W in fp32, gate-interleaved columns
    float* u_il;    // [H][4H]
    float* dw_il;   // [D][4H] weight gradients, gate-interleaved columns
    float* du_il;   // [H][4H]
    float* db_il;   // [4H]
    float* cs_part; // [BWD_CS_CHUNKS][4H] partial column sums of dz
    float* dH;      // [B][H] gradient of h in slot order
    float* dC;      // [B][H]
    float* z;       // [bpad][4H] per-step pre-activations (handles not in per-step mode)
    // bf16 data: fp16 operands of the weight-gradient GEMMs (scaled by powers of two)
    _Float16* dz16; // [B*T][4H]
    _Float16* x16;  // [B*T][D]
    _Float16* h16;  // [B*T][H]
    _Float16* w16;  // [D][4H]
    _Float16* u16;  // [H][4H] U (gate-interleaved), scaled
    _Float16* dzs16;// [B][4H] one step's dz, each row scaled by srow
    float* srow;    // [B] scale of each row's dH
    unsigned* amax; // [5] largest magnitudes (float bits) of dz, x, h_prev, W, U
    int32_t* host_offsets;  // pinned [T + 8]: step offsets, the sum of lengths, then amax
    rocblas_handle rb;
    // the reverse loop in one launch (bf16 data, persistent handles that fit):
    // all steps with column blocks of U (bwdblk.hip), else the steps with few
    // rows (bwd.hip) and two launches for each other step
    int block_groups;       // workgroups of the whole-loop launch, or 0
    int loop_groups;        // workgroups of the few-row launch, or 0
    _Float16* dzx;          // [2][bpad][kp] each step's published dz
    float* dzs;             // [2][bpad][nblk] their scales
    float* pdh;             // [4][4][bpad][H] the column blocks' shares of dh
    unsigned* bar;          // [9 * 64] barrier counters (the few-row launch)
    long long dzx_bytes, dzs_bytes, pdh_bytes;
};

using namespace ldyn;

struct lstm_dyn {
    int B, D, H, T, dtype, mode, cell;
    void* w4;                  // GRU, RNN: the packed W4, U4, b4 (pack.hip); else null
    void* u4;
    float* b4;
    long long workspace;       // bytes of the device workspace
    int device, num_cus;
    lstm_dyn_plan_t plan;
    Dims dims;
    Workspace ws;
    void* block;               // the one device allocation behind ws
    int32_t* host_maxlen;      // pinned host words for the per-step path: [0] loop bound,
                               // [1] rows still running, [2] iterations run
    int stop_ok;               // the persistent variant with termination from the state fits
    int save_ok;               // the persistent variant of the forward for training fits
    TrainWs* train;            // null until the first forward for training
    int saved;                 // 1: the workspace holds a forward for training not yet used
    unsigned long long timeout_ticks;
    int inproj_grid;
    long long launches_last;
    hipStream_t last_stream;   // the stream of the last forward or backward
    int has_work;              // 1 once work has been enqueued on last_stream
    int timing;                // record phase events on the forward's stream
    unsigned long long* trace; // per-step timestamps (diagnostics), [T + 1], or null
    int wclk_khz;
    hipEvent_t ev[4];          // before prep, after prep, after input projection, after loop
};

namespace {

constexpr int PREP_MAX_B = 8192;
// Backward with bf16 data: steps with at most this many rows go to the
// one-launch reverse loop, the others to two launches per step.
constexpr int BWD_LOOP_ROWS = 16;
constexpr double BARRIER_TIMEOUT_S = 5.0;

long long align_up(long long v, long long a) { return (v + a - 1) / a * a; }


struct Layout {
    long long meta, perm, offsets, rowsrc, gx, hx, bar, z, wt, w4, u4, b4, stopped, running, total;
};

Layout layout_of(int B, int D, int H, int T, int bf16, int mode, int bpad, int hpad, int packed = 0) {
    Layout L{};
    long long o = 0;
    auto take = [&](long long bytes) {
        const long long at = o;
        o = align_up(o + bytes, 256);
        return at;
    };
    L.meta = take(sizeof(Meta));
    L.perm = take(4LL * B);
    L.offsets = take(4LL * (T + 1));
    L.rowsrc = take(4LL * B * T);
    L.gx = take(16LL * H * B * T);
    L.hx = take(4LL * bpad * hpad * (bf16 ? 2 : 4));
    L.bar = take(4LL * BAR_WORDS);
    L.z = take(mode == LSTM_DYN_PER_STEP ? 16LL * H * bpad : 0);
    if (bf16) {
        Dims d{B, D, H, T, 1, hpad, bpad};
        int np, dp;
        inproj_bf16_wt_shape(d, &np, &dp);
        L.wt = take(2LL * np * dp);
    } else {
        L.wt = take(0);
    }
    const long long e = bf16 ? 2 : 4;
    L.w4 = take(packed ? e * D * 4 * H : 0);
    L.u4 = take(packed ? e * H * 4 * H : 0);
    L.b4 = take(packed ? 16LL * H : 0);
    L.stopped = take(4LL * B);
    L.running = take(4LL * T);
    L.total = o;
    return L;
}

static_assert(LSTM_DYN_CELL_LSTM == CELL_LSTM && LSTM_DYN_CELL_GRU == CELL_GRU &&
                  LSTM_DYN_CELL_RNN == CELL_RNN,
              "the C ABI's cell numbers are the kernels' CellKind");

bool valid_cell(int cell) {
    return cell == LSTM_DYN_CELL_LSTM || cell == LSTM_DYN_CELL_GRU || cell == LSTM_DYN_CELL_RNN;
}
// Columns of W and U, and bias floats, per hidden unit of each cell.
int cell_cols(int cell) { return cell == LSTM_DYN_CELL_GRU ? 3 : cell == LSTM_DYN_CELL_RNN ? 1 : 4; }
int cell_bias(int cell) { return cell == LSTM_DYN_CELL_GRU ? 6 : cell == LSTM_DYN_CELL_RNN ? 1 : 4; }

bool overlaps(const void* a, long long na, const void* b, long long nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

}  // namespace

namespace ldyn {
// The workspace of a persistent-mode LSTM forward inside caller memory at
// base (256-byte aligned): fills ws and returns the bytes used, and the
// operand buffer's offset and size (the only part that must start at zero
// on every forward: its padding columns are multiplied by zero weights).
long long carve_forward_workspace(const Dims& d, char* base, Workspace* ws, long long* hx_off,
                                  long long* hx_bytes) {
    const Layout L = layout_of(d.B, d.D, d.H, d.T, d.bf16, LSTM_DYN_PERSISTENT, d.bpad, d.hpad, 0);
    *hx_off = L.hx;
    *hx_bytes = L.bar - L.hx;
    if (base) {
        *ws = Workspace{};
        ws->meta = reinterpret_cast<Meta*>(base + L.meta);
        ws->perm = reinterpret_cast<int32_t*>(base + L.perm);
        ws->offsets = reinterpret_cast<int32_t*>(base + L.offsets);
        ws->rowsrc = reinterpret_cast<int32_t*>(base + L.rowsrc);
        ws->gx = reinterpret_cast<float*>(base + L.gx);
        ws->hx = base + L.hx;
        ws->bar = reinterpret_cast<unsigned*>(base + L.bar);
        ws->wt = d.bf16 ? base + L.wt : nullptr;
        ws->stopped = reinterpret_cast<int32_t*>(base + L.stopped);
        ws->running = reinterpret_cast<int32_t*>(base + L.running);
    }
    return L.total;
}
}  // namespace ldyn

extern "C" const char* lstm_dyn_strerror(int status) {
    switch (status) {
        case LSTM_DYN_OK: return "ok";
        case LSTM_DYN_ERR_INVALID: return "invalid argument";
        case LSTM_DYN_ERR_HIP: return "HIP runtime error";
        case LSTM_DYN_ERR_NOMEM: return "device workspace allocation failed";
        case LSTM_DYN_ERR_UNSUPPORTED: return "sizes not covered by the compiled kernel variants";
        case LSTM_DYN_ERR_BAD_LENGTHS: return "a sequence length was outside [0, T_max] and was clamped";
        case LSTM_DYN_ERR_TIMEOUT: return "a wait of a cooperative kernel exceeded its bound";
        case LSTM_DYN_ERR_TOO_LARGE:
            return "the workspace exceeds the allocation-free entry point's fixed scratch";
        default: return "unknown status";
    }
}

extern "C" int lstm_dyn_plan(int B, int D, int H, int T, int dtype, int mode, int num_cus,
                             lstm_dyn_plan_t* out) {
    if (!out) return LSTM_DYN_ERR_INVALID;
    memset(out, 0, sizeof(*out));
    if (B < 1 || D < 1 || H < 1 || T < 1 || num_cus < 1) return LSTM_DYN_ERR_INVALID;
    if (dtype != LSTM_DYN_F32 && dtype != LSTM_DYN_BF16) return LSTM_DYN_ERR_INVALID;
    if (mode != LSTM_DYN_PERSISTENT && mode != LSTM_DYN_PER_STEP) return LSTM_DYN_ERR_INVALID;
    if (B > PREP_MAX_B || (long long)B * T > 0x7fffffffLL || 4LL * H > 0x7fffffffLL / 4)
        return LSTM_DYN_ERR_UNSUPPORTED;
    const int bf16 = dtype == LSTM_DYN_BF16;
    const int kstep = bf16 ? 32 : 4;
    const int ntmax = (B + 15) / 16;
    // Workgroup shape: 4*mt hidden units per workgroup (one workgroup per CU),
    // kw waves splitting K = H into ksw MFMA K-steps each (a power of two; the
    // operand buffer's padding columns are zero).
    int mt = 1, kw = 4;
    if (bf16 && H > 1024) {
        mt = 2;
        kw = 8;
    }
    const int groups = (H + 4 * mt - 1) / (4 * mt);
    if (groups > num_cus) return LSTM_DYN_ERR_UNSUPPORTED;
    const int kneed = (H + kstep * kw - 1) / (kstep * kw);
    int ksw = bf16 ? 1 : 4;  // fp32 lanes load K-steps in groups of four
    while (ksw < kneed) ksw *= 2;
    const int nstate = (ntmax * mt + kw - 1) / kw;
    int nst = nstate;
    if (mode == LSTM_DYN_PERSISTENT && !persistent_pick_variant(bf16, mt, kw, ksw, nstate, &nst))
        return LSTM_DYN_ERR_UNSUPPORTED;
    out->mt = mt;
    out->groups = groups;
    out->ksw = ksw;
    out->kw = kw;
    out->hpad = ksw * kstep * kw;
    out->bpad = ntmax * 16;
    out->lds_bytes = persistent_lds_bytes(bf16, mt, kw, nst, out->hpad);
    out->nstate = nst;
    out->workspace_bytes =
        layout_of(B, D, H, T, bf16, mode, out->bpad, out->hpad).total;
    if (mode == LSTM_DYN_PERSISTENT && H <= 32 &&
        small_pick(bf16, B, D, H, &out->single_kd, &out->single_nt)) {
        out->single = 1;
        out->groups = 1;
    }
    return LSTM_DYN_OK;
}

// Argument checks for a cell: W [D][G], U [H][G], b [NB] with G = NB = 4H
// (LSTM), G = 3H and NB = 6H (GRU), G = NB = H (RNN); only the LSTM reads c0.
static int check_args_cell(int B, int D, int H, int T, int dtype, int cell, const void* x,
                           const int32_t* lengths, const void* W, const void* U, const float* b,
                           const float* h0, const float* c0, const float* out_h,
                           const float* out_c) {
    if (B < 1 || D < 1 || H < 1 || T < 1) return LSTM_DYN_ERR_INVALID;
    if (dtype != LSTM_DYN_F32 && dtype != LSTM_DYN_BF16) return LSTM_DYN_ERR_INVALID;
    if (!valid_cell(cell)) return LSTM_DYN_ERR_INVALID;
    const bool has_c = cell == LSTM_DYN_CELL_LSTM;
    if (!has_c) c0 = nullptr;  // no cell state: c0 is ignored and may be NULL
    if (!x || !lengths || !W || !U || !b || !h0 || (!c0 && has_c) || !out_h || !out_c)
        return LSTM_DYN_ERR_INVALID;
    auto al = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; };
    if (!al(x, 16) || !al(W, 16) || !al(U, 16)) return LSTM_DYN_ERR_INVALID;
    if (!al(lengths, 4) || !al(b, 4) || !al(h0, 4) || !al(c0, 4) || !al(out_h, 4) || !al(out_c, 4))
        return LSTM_DYN_ERR_INVALID;
    const long long e = dtype == LSTM_DYN_BF16 ? 2 : 4;
    const long long G = (long long)cell_cols(cell) * H;
    const long long nx = (long long)B * T * D * e, nL = 4LL * B, nW = (long long)D * G * e,
                    nU = (long long)H * G * e, nb = 4LL * cell_bias(cell) * H, ns = 4LL * B * H;
    if (overlaps(out_h, ns, out_c, ns)) return LSTM_DYN_ERR_INVALID;
    const void* ins[] = {x, lengths, W, U, b, h0, c0};
    const long long nin[] = {nx, nL, nW, nU, nb, ns, has_c ? ns : 0};
    for (int i = 0; i < 7; ++i) {
        if (overlaps(out_h, ns, ins[i], nin[i]) && !(i == 5 && out_h == h0)) return LSTM_DYN_ERR_INVALID;
        if (overlaps(out_c, ns, ins[i], nin[i]) && !(i == 6 && out_c == c0)) return LSTM_DYN_ERR_INVALID;
    }
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_check_args(int B, int D, int H, int T, int dtype, const void* x,
                                   const int32_t* lengths, const void* W, const void* U,
                                   const float* b, const float* h0, const float* c0,
                                   const float* out_h, const float* out_c) {
    return check_args_cell(B, D, H, T, dtype, 0, x, lengths, W, U, b, h0, c0, out_h, out_c);
}

static int check_seq_args_cell(int B, int D, int H, int T, int dtype, int cell, const void* x,
                               const int32_t* lengths, const void* W, const void* U,
                               const float* b, const float* h0, const float* c0,
                               const float* out_h, const float* out_c, const float* out_seq);

extern "C" int lstm_dyn_check_seq_args(int B, int D, int H, int T, int dtype, const void* x,
                                       const int32_t* lengths, const void* W, const void* U,
                                       const float* b, const float* h0, const float* c0,
                                       const float* out_h, const float* out_c, const float* out_seq) {
    return check_seq_args_cell(B, D, H, T, dtype, 0, x, lengths, W, U, b, h0, c0, out_h, out_c,
                               out_seq);
}

static int check_seq_args_cell(int B, int D, int H, int T, int dtype, int cell, const void* x,
                               const int32_t* lengths, const void* W, const void* U,
                               const float* b, const float* h0, const float* c0,
                               const float* out_h, const float* out_c, const float* out_seq) {
    const int rc = check_args_cell(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0, c0, out_h, out_c);
    if (rc != LSTM_DYN_OK) return rc;
    if (!out_seq || (reinterpret_cast<uintptr_t>(out_seq) & 3) != 0) return LSTM_DYN_ERR_INVALID;
    const long long e = dtype == LSTM_DYN_BF16 ? 2 : 4;
    const long long G = (long long)cell_cols(cell) * H;
    const long long nseq = 4LL * B * T * H;
    const void* others[] = {x, lengths, W, U, b, h0, c0, out_h, out_c};
    const long long sizes[] = {(long long)B * T * D * e, 4LL * B, (long long)D * G * e,
                               (long long)H * G * e, 4LL * cell_bias(cell) * H, 4LL * B * H,
                               cell == LSTM_DYN_CELL_LSTM ? 4LL * B * H : 0, 4LL * B * H,
                               4LL * B * H};
    for (int i = 0; i < 9; ++i)
        if (overlaps(out_seq, nseq, others[i], sizes[i])) return LSTM_DYN_ERR_INVALID;
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_check_cell_args(int B, int D, int H, int T, int dtype, int cell,
                                        const void* x, const int32_t* lengths, const void* W,
                                        const void* U, const float* b, const float* h0,
                                        const float* c0, const float* out_h, const float* out_c,
                                        const float* out_seq) {
    if (!out_seq)
        return check_args_cell(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0, c0, out_h, out_c);
    return check_seq_args_cell(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0, c0, out_h, out_c,
                               out_seq);
}

extern "C" int lstm_dyn_create(lstm_dyn_t** out, int B, int D, int H, int T, int dtype, int mode) {
    return lstm_dyn_create_cell(out, B, D, H, T, dtype, mode, LSTM_DYN_CELL_LSTM);
}

extern "C" int lstm_dyn_create_cell(lstm_dyn_t** out, int B, int D, int H, int T, int dtype,
                                    int mode, int cell) {
    if (!out) return LSTM_DYN_ERR_INVALID;
    *out = nullptr;
    if (!valid_cell(cell)) return LSTM_DYN_ERR_INVALID;
    const int packed = cell != LSTM_DYN_CELL_LSTM;
    lstm_dyn_plan_t plan;
    int rc = lstm_dyn_plan(B, D, H, T, dtype, mode, 1 << 20, &plan);  // size checks only
    if (rc != LSTM_DYN_OK) return rc;
    int dev = 0, cus = 0, wclk_khz = 0;
    if (hipGetDevice(&dev) != hipSuccess) return LSTM_DYN_ERR_HIP;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return LSTM_DYN_ERR_HIP;
    if (hipDeviceGetAttribute(&wclk_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
        return LSTM_DYN_ERR_HIP;
    rc = lstm_dyn_plan(B, D, H, T, dtype, mode, cus, &plan);
    if (rc != LSTM_DYN_OK) return rc;
    const int bf16 = dtype == LSTM_DYN_BF16;
    int stop_ok = 1, save_ok = 1;
    if (mode == LSTM_DYN_PERSISTENT && !plan.single) {
        const int per_cu = persistent_blocks_per_cu(bf16, plan.mt, plan.ksw, plan.kw, plan.nstate,
                                                    plan.lds_bytes, cell, 0);
        if (per_cu < 1 || plan.groups > per_cu * cus) return LSTM_DYN_ERR_UNSUPPORTED;
        const int per_cu_stop = persistent_blocks_per_cu(bf16, plan.mt, plan.ksw, plan.kw,
                                                         plan.nstate, plan.lds_bytes, cell, 1);
        stop_ok = per_cu_stop >= 1 && plan.groups <= per_cu_stop * cus;
        const int per_cu_save = persistent_blocks_per_cu(bf16, plan.mt, plan.ksw, plan.kw,
                                                         plan.nstate, plan.lds_bytes, cell, 2);
        save_ok = per_cu_save >= 1 && plan.groups <= per_cu_save * cus;
    }
    lstm_dyn* h = new (std::nothrow) lstm_dyn();
    if (!h) return LSTM_DYN_ERR_NOMEM;
    h->B = B; h->D = D; h->H = H; h->T = T; h->dtype = dtype; h->mode = mode; h->cell = cell;
    h->stop_ok = stop_ok;
    h->save_ok = save_ok;
    h->device = dev;
    h->num_cus = cus;
    h->plan = plan;
    h->dims = Dims{B, D, H, T, bf16, plan.hpad, plan.bpad, cell};
    const Layout L = layout_of(B, D, H, T, bf16, mode, plan.bpad, plan.hpad, packed);
    h->workspace = L.total;
    if (hipMalloc(&h->block, (size_t)L.total) != hipSuccess) {
        (void)hipGetLastError();
        delete h;
        return LSTM_DYN_ERR_NOMEM;
    }
    char* base = static_cast<char*>(h->block);
    h->ws.meta = reinterpret_cast<Meta*>(base + L.meta);
    h->ws.perm = reinterpret_cast<int32_t*>(base + L.perm);
    h->ws.offsets = reinterpret_cast<int32_t*>(base + L.offsets);
    h->ws.rowsrc = reinterpret_cast<int32_t*>(base + L.rowsrc);
    h->ws.gx = reinterpret_cast<float*>(base + L.gx);
    h->ws.hx = base + L.hx;
    h->ws.bar = reinterpret_cast<unsigned*>(base + L.bar);
    h->ws.z = mode == LSTM_DYN_PER_STEP ? reinterpret_cast<float*>(base + L.z) : nullptr;
    h->ws.wt = bf16 ? base + L.wt : nullptr;
    h->w4 = packed ? base + L.w4 : nullptr;
    h->u4 = packed ? base + L.u4 : nullptr;
    h->b4 = packed ? reinterpret_cast<float*>(base + L.b4) : nullptr;
    h->ws.stopped = reinterpret_cast<int32_t*>(base + L.stopped);
    h->ws.running = reinterpret_cast<int32_t*>(base + L.running);
    // Zero the small tables and the operand buffer (its padding must stay zero).
    if (hipMemset(base, 0, (size_t)L.gx) != hipSuccess ||
        hipMemset(base + L.hx, 0, (size_t)(L.total - L.hx)) != hipSuccess) {
        (void)hipFree(h->block);
        delete h;
        return LSTM_DYN_ERR_HIP;
    }
    if (hipHostMalloc(reinterpret_cast<void**>(&h->host_maxlen), 4 * sizeof(int32_t), hipHostMallocDefault) != hipSuccess) {
        (void)hipFree(h->block);
        delete h;
        return LSTM_DYN_ERR_HIP;
    }
    h->timeout_ticks = (unsigned long long)(BARRIER_TIMEOUT_S * 1e3 * (double)wclk_khz);
    if (bf16) {
        if (inproj_bf16_setup() != hipSuccess) {
            (void)hipFree(h->block);
            (void)hipHostFree(h->host_maxlen);
            delete h;
            return LSTM_DYN_ERR_HIP;
        }
        const long long tiles = inproj_bf16_tiles_max(h->dims);
        h->inproj_grid = (int)(tiles < cus ? tiles : cus);
    } else {
        const long long tiles = ((long long)B * T + 127) / 128 * ((4LL * H + 127) / 128);
        h->inproj_grid = (int)(tiles < 4LL * cus ? tiles : 4LL * cus);
    }
    h->launches_last = 0;
    h->last_stream = nullptr;
    h->has_work = 0;
    h->timing = 0;
    h->trace = nullptr;
    h->wclk_khz = wclk_khz;
    for (auto& e : h->ev) e = nullptr;
    *out = h;
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_set_option(lstm_dyn_t* h, int option, long long value) {
    if (!h) return LSTM_DYN_ERR_INVALID;
    if (option == LSTM_DYN_OPT_TIMING) {
        if (value && !h->ev[0]) {
            for (auto& e : h->ev)
                if (hipEventCreate(&e) != hipSuccess) return LSTM_DYN_ERR_HIP;
        }
        h->timing = value ? 1 : 0;
        return LSTM_DYN_OK;
    }
    if (option == LSTM_DYN_OPT_TIMEOUT_US) {
        if (value < 0 || value > 60000000LL) return LSTM_DYN_ERR_INVALID;
        const double us = value ? (double)value : BARRIER_TIMEOUT_S * 1e6;
        h->timeout_ticks = (unsigned long long)(us * 1e-3 * (double)h->wclk_khz);
        return LSTM_DYN_OK;
    }
    if (option == LSTM_DYN_OPT_STEP_TRACE) {
        if (value && !h->trace) {
            if (hipMalloc(&h->trace, sizeof(unsigned long long) * 4 * (h->T + 1)) != hipSuccess) {
                h->trace = nullptr;
                return LSTM_DYN_ERR_NOMEM;
            }
        } else if (!value && h->trace) {
            // the last forward may still write the trace
            if ((h->has_work && hipStreamSynchronize(h->last_stream) != hipSuccess) ||
                hipFree(h->trace) != hipSuccess)
                return LSTM_DYN_ERR_HIP;
            h->trace = nullptr;
        }
        return LSTM_DYN_OK;
    }
    return LSTM_DYN_ERR_INVALID;
}

extern "C" int lstm_dyn_step_trace(lstm_dyn_t* h, long long* ticks, int capacity, int* count, int* khz) {
    if (!h || !ticks || !count || !khz || !h->trace || capacity < 0) return LSTM_DYN_ERR_INVALID;
    if (hipStreamSynchronize(h->last_stream) != hipSuccess) return LSTM_DYN_ERR_HIP;
    Meta m;
    if (hipMemcpy(&m, h->ws.meta, sizeof(Meta), hipMemcpyDeviceToHost) != hipSuccess) return LSTM_DYN_ERR_HIP;
    const int n = m.max_len > 0 ? 4 * m.max_len + 1 : 0;
    const int c = n < capacity ? n : capacity;
    if (c > 0 && hipMemcpy(ticks, h->trace, sizeof(long long) * c, hipMemcpyDeviceToHost) != hipSuccess)
        return LSTM_DYN_ERR_HIP;
    *count = c;
    *khz = h->wclk_khz;
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_destroy(lstm_dyn_t* h) {
    if (!h) return LSTM_DYN_OK;
    int rc = LSTM_DYN_OK;
    // One forward or backward may be in flight per handle, on the stream it
    // was issued on: wait for that stream only, not for the whole device.
    if (h->has_work && hipStreamSynchronize(h->last_stream) != hipSuccess) rc = LSTM_DYN_ERR_HIP;
    if (h->block && hipFree(h->block) != hipSuccess) rc = LSTM_DYN_ERR_HIP;
    for (auto& e : h->ev)
        if (e && hipEventDestroy(e) != hipSuccess) rc = LSTM_DYN_ERR_HIP;
    if (h->host_maxlen && hipHostFree(h->host_maxlen) != hipSuccess) rc = LSTM_DYN_ERR_HIP;
    if (h->trace && hipFree(h->trace) != hipSuccess) rc = LSTM_DYN_ERR_HIP;
    if (h->train) {
        if (h->train->rb && g_rb.destroy_handle(h->train->rb) != rocblas_status_success)
            rc = LSTM_DYN_ERR_HIP;
        if (h->train->block && hipFree(h->train->block) != hipSuccess) rc = LSTM_DYN_ERR_HIP;
        if (h->train->host_offsets && hipHostFree(h->train->host_offsets) != hipSuccess)
            rc = LSTM_DYN_ERR_HIP;
        delete h->train;
    }
    delete h;
    return rc;
}

// Input projection over all valid steps: bf16 goes through the transposed-W
// tiled GEMM (two launches), fp32 through the generic MFMA GEMM (one launch).
static hipError_t input_projection(lstm_dyn* h, const void* x, const void* W, const float* b,
                                   hipStream_t s) {
    hipError_t e;
    if (h->dims.bf16) {
        if ((e = launch_transpose_w(h->dims, W, h->ws, s)) != hipSuccess) return e;
        h->launches_last++;
        e = launch_inproj_bf16(h->dims, x, b, h->ws, h->inproj_grid, s);
    } else {
        e = launch_inproj(h->dims, x, W, b, h->ws, h->inproj_grid, s);
    }
    h->launches_last++;
    return e;
}

// The forward of both entry points; out_seq is null for lstm_dyn_forward.
static int forward_impl(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                        const void* U, const float* b, const float* h0, const float* c0,
                        float* out_h, float* out_c, float* out_seq, const StopArgs* stop,
                        void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    h->last_stream = s;
    h->has_work = 1;
    h->launches_last = 0;
    h->saved = 0;  // this forward overwrites what a forward for training kept
    const Dims& d = h->dims;
#define LD_CHECK(call)                                   \
    do {                                                 \
        if ((call) != hipSuccess) {                      \
            (void)hipGetLastError();                     \
            return LSTM_DYN_ERR_HIP;                     \
        }                                                \
    } while (0)

    auto mark = [&](int i) { return h->timing ? hipEventRecord(h->ev[i], s) : hipSuccess; };
    LD_CHECK(mark(0));
    const bool packed = h->cell != LSTM_DYN_CELL_LSTM;
    if (packed) {
        // the cell's weights in the four-block layout the kernels use (timed with prep)
        LD_CHECK(launch_cell_pack(d, W, U, b, h->w4, h->u4, h->b4, s));
        W = h->w4;
        U = h->u4;
        b = h->b4;
    }
    const long long pack_launches = packed ? 1 : 0;
    // the output sequence is zero past each row's last step: its cap, or the
    // step it ended at
    const int32_t* seq_ends = stop ? stop->steps : lengths;
    if (h->mode == LSTM_DYN_PERSISTENT && h->plan.single) {
        LD_CHECK(mark(1));
        LD_CHECK(mark(2));
        LD_CHECK(launch_small(d, h->plan.single_kd, h->plan.single_nt, x, lengths, W, U, b, h0, c0,
                              out_h, out_c, out_seq, stop, h->ws, s));
        h->launches_last = 1 + pack_launches;
        LD_CHECK(mark(3));
        if (out_seq) {
            LD_CHECK(launch_seq_finish(d, out_seq, seq_ends, h->num_cus, s));
            h->launches_last++;
        }
        return LSTM_DYN_OK;
    }
    LD_CHECK(launch_prep(d, lengths, h->ws, s));
    h->launches_last += 1 + pack_launches;
    LD_CHECK(mark(1));
    if (h->mode == LSTM_DYN_PERSISTENT) {
        LD_CHECK(input_projection(h, x, W, b, s));
        LD_CHECK(mark(2));
        PersistentConfig pc{h->plan.mt,     h->plan.groups,    h->plan.ksw, h->plan.kw,
                            h->plan.nstate, h->plan.lds_bytes, h->timeout_ticks, h->trace,
                            out_seq,        stop};
        LD_CHECK(launch_persistent(d, pc, U, h0, c0, out_h, out_c, h->ws, s));
        h->launches_last++;
        LD_CHECK(mark(3));
        if (out_seq) {  // the loop wrote the valid steps; zeros past each row's last
            LD_CHECK(launch_seq_finish(d, out_seq, seq_ends, h->num_cus, s));
            h->launches_last++;
        }
        return LSTM_DYN_OK;
    }
    // Per-step comparison path.
    LD_CHECK(launch_step_init(d, h0, c0, out_h, out_c, h->ws, s));
    h->launches_last++;
    if (stop) {
        LD_CHECK(launch_step_stop_init(d, *stop, h->ws, s));
        h->launches_last++;
    }
    LD_CHECK(input_projection(h, x, W, b, s));
    LD_CHECK(mark(2));
    LD_CHECK(hipMemcpyAsync(h->host_maxlen, &h->ws.meta->max_len, sizeof(int32_t),
                            hipMemcpyDeviceToHost, s));
    LD_CHECK(hipStreamSynchronize(s));
    const int max_len = *h->host_maxlen;
    int iters = max_len;
    for (int t = 0; t < max_len; ++t) {
        LD_CHECK(launch_step_gemm(d, t, U, h->ws, s));
        LD_CHECK(launch_step_gates(d, t, out_h, out_c, out_seq, stop != nullptr, h->ws, s));
        h->launches_last += 2;
        if (stop) {
            // the eager loop condition: read on the host after every step
            LD_CHECK(launch_step_stop(d, t, *stop, h->ws, s));
            h->launches_last++;
            LD_CHECK(hipMemcpyAsync(h->host_maxlen + 1, h->ws.running + t, sizeof(int32_t),
                                    hipMemcpyDeviceToHost, s));
            LD_CHECK(hipStreamSynchronize(s));
            if (h->host_maxlen[1] == 0) {
                iters = t + 1;
                break;
            }
        }
    }
    if (stop) {
        h->host_maxlen[2] = iters;
        LD_CHECK(hipMemcpyAsync(&h->ws.meta->iters, h->host_maxlen + 2, sizeof(int32_t),
                                hipMemcpyHostToDevice, s));
    }
    LD_CHECK(mark(3));
    if (out_seq) {
        LD_CHECK(launch_seq_finish(d, out_seq, seq_ends, h->num_cus, s));
        h->launches_last++;
    }
#undef LD_CHECK
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_forward(lstm_dyn_t* h, const void* x, const int32_t* lengths, const void* W,
                                const void* U, const float* b, const float* h0, const float* c0,
                                float* out_h, float* out_c, void* stream) {
    if (!h) return LSTM_DYN_ERR_INVALID;
    const int rc = check_args_cell(h->B, h->D, h->H, h->T, h->dtype, h->cell,
                                   x, lengths, W, U, b, h0, c0, out_h, out_c);
    if (rc != LSTM_DYN_OK) return rc;
    return forward_impl(h, x, lengths, W, U, b, h0, c0, out_h, out_c, nullptr, nullptr, stream);
}

extern "C" int lstm_dyn_forward_seq(lstm_dyn_t* h, const void* x, const int32_t* lengths,
                                    const void* W, const void* U, const float* b, const float* h0,
                                    const float* c0, float* out_h, float* out_c, float* out_seq,
                                    void* stream) {
    if (!h) return LSTM_DYN_ERR_INVALID;
    const int rc = check_seq_args_cell(h->B, h->D, h->H, h->T, h->dtype,
                                       h->cell, x, lengths, W, U, b, h0, c0,
                                       out_h, out_c, out_seq);
    if (rc != LSTM_DYN_OK) return rc;
    return forward_impl(h, x, lengths, W, U, b, h0, c0, out_h, out_c, out_seq, nullptr, stream);
}

static int check_stop_args_cell(int B, int D, int H, int T, int dtype, int cell, const void* x,
                                const int32_t* lengths, const void* W, const void* U,
                                const float* b, const float* h0, const float* c0,
                                const float* stop_v, const float* out_h, const float* out_c,
                                const int32_t* out_steps, const float* out_seq) {
    const int rc = out_seq ? check_seq_args_cell(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0,
                                                 c0, out_h, out_c, out_seq)
                           : check_args_cell(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0, c0,
                                             out_h, out_c);
    if (rc != LSTM_DYN_OK) return rc;
    if (!stop_v || !out_steps) return LSTM_DYN_ERR_INVALID;
    if ((reinterpret_cast<uintptr_t>(stop_v) & 3) || (reinterpret_cast<uintptr_t>(out_steps) & 3))
        return LSTM_DYN_ERR_INVALID;
    const long long e = dtype == LSTM_DYN_BF16 ? 2 : 4;
    const long long G = (long long)cell_cols(cell) * H;
    const bool has_c = cell == LSTM_DYN_CELL_LSTM;
    const long long nv = 4LL * H, nst = 4LL * B, ns = 4LL * B * H;
    const long long nseq = out_seq ? 4LL * B * T * H : 0;
    // out_steps overlaps nothing; v overlaps no output
    const void* all[] = {x, lengths, W, U, b, h0, has_c ? c0 : nullptr, stop_v, out_h, out_c, out_seq};
    const long long sz[] = {(long long)B * T * D * e, 4LL * B, (long long)D * G * e,
                            (long long)H * G * e, 4LL * cell_bias(cell) * H, ns, has_c ? ns : 0, nv,
                            ns, ns, nseq};
    for (int i = 0; i < 11; ++i)
        if (all[i] && overlaps(out_steps, nst, all[i], sz[i])) return LSTM_DYN_ERR_INVALID;
    const void* outs[] = {out_h, out_c, out_seq};
    const long long osz[] = {ns, ns, nseq};
    for (int i = 0; i < 3; ++i)
        if (outs[i] && overlaps(stop_v, nv, outs[i], osz[i])) return LSTM_DYN_ERR_INVALID;
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_check_stop_args(int B, int D, int H, int T, int dtype, int cell,
                                        const void* x, const int32_t* lengths, const void* W,
                                        const void* U, const float* b, const float* h0,
                                        const float* c0, const float* stop_v, const float* out_h,
                                        const float* out_c, const int32_t* out_steps,
                                        const float* out_seq) {
    if (!valid_cell(cell)) return LSTM_DYN_ERR_INVALID;
    return check_stop_args_cell(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0, c0, stop_v,
                                out_h, out_c, out_steps, out_seq);
}

extern "C" int lstm_dyn_forward_stop(lstm_dyn_t* h, const void* x, const int32_t* lengths,
                                     const void* W, const void* U, const float* b, const float* h0,
                                     const float* c0, const float* stop_v, float stop_c,
                                     float* out_h, float* out_c, int32_t* out_steps,
                                     float* out_seq, void* stream) {
    if (!h) return LSTM_DYN_ERR_INVALID;
    const int rc = check_stop_args_cell(h->B, h->D, h->H, h->T, h->dtype, h->cell, x, lengths, W,
                                        U, b, h0, c0, stop_v, out_h, out_c, out_steps, out_seq);
    if (rc != LSTM_DYN_OK) return rc;
    if (!h->stop_ok) return LSTM_DYN_ERR_UNSUPPORTED;
    if (stop_c != stop_c) return LSTM_DYN_ERR_INVALID;  // NaN
    const StopArgs stop{stop_v, stop_c, out_steps, lengths};
    return forward_impl(h, x, lengths, W, U, b, h0, c0, out_h, out_c, out_seq, &stop, stream);
}

// ---------------------------------------------------------------------------
// Forward for training and the backward pass (LSTM handles).

// The power of two that brings a largest magnitude (float bits) into
// [2^13, 2^14): fp16 keeps its 11 bits there, far from overflow.
static float f16_scale(unsigned bits) {
    float m;
    memcpy(&m, &bits, sizeof(m));
    if (!(m > 0.0f) || !(m < 3.0e38f)) return 1.0f;
    int e;
    (void)frexpf(m, &e);
    const int k = 14 - e;
    return ldexpf(1.0f, k < 126 ? k : 126);
}

static int ensure_train(lstm_dyn* h) {
    if (h->train) return LSTM_DYN_OK;
    TrainWs* tw = new (std::nothrow) TrainWs();
    if (!tw) return LSTM_DYN_ERR_NOMEM;
    const long long B = h->B, D = h->D, H = h->H, T = h->T, bpad = h->dims.bpad;
    long long o = 0;
    auto take = [&](long long bytes) {
        const long long at = o;
        o = align_up(o + bytes, 256);
        return at;
    };
    const long long oh = take(4 * B * T * H), oc = take(4 * B * T * H), ox = take(4 * B * T * D),
                    ow = take(4 * D * 4 * H), ou = take(4 * H * 4 * H), odw = take(4 * D * 4 * H),
                    odu = take(4 * H * 4 * H), odb = take(16 * H), odh = take(4 * B * H),
                    odc = take(4 * B * H), oz = take(16 * H * bpad);
    const bool h16 = h->dtype == LSTM_DYN_BF16;
    const long long odz16 = take(h16 ? 2 * B * T * 4 * H : 0), ox16 = take(h16 ? 2 * B * T * D : 0),
                    oh16 = take(h16 ? 2 * B * T * H : 0), ow16 = take(h16 ? 2 * D * 4 * H : 0),
                    ou16 = take(h16 ? 2 * H * 4 * H : 0), odzs = take(h16 ? 2 * B * 4 * H : 0),
                    osr = take(4 * B), osm = take(256), ocs = take(4LL * BWD_CS_CHUNKS * 4 * H);
    const bool pers16 = h16 && h->mode == LSTM_DYN_PERSISTENT;
    tw->block_groups = pers16 ? bwd_block_fits(h->dims, h->num_cus) : 0;
    tw->loop_groups = pers16 && !tw->block_groups ? bwd_loop_fits(h->dims, h->num_cus) : 0;
    int kp = 0, nblk = 0;
    if (tw->loop_groups) bwd_loop_shape((int)H, &kp, &nblk);
    int slots = 2;  // the few-row launch: by step parity
    if (tw->block_groups) {
        kp = (int)(4 * H);
        nblk = (int)(H / 8);
        slots = 4;
    }
    const bool one_launch = tw->block_groups || tw->loop_groups;
    tw->dzx_bytes = 2LL * slots * bpad * kp;
    tw->dzs_bytes = 4LL * slots * bpad * nblk;
    tw->pdh_bytes = tw->block_groups ? 4LL * 4 * 4 * bpad * H : 0;
    const long long odzx = take(tw->dzx_bytes), odzsc = take(tw->dzs_bytes), opdh = take(tw->pdh_bytes),
                    obar = take(tw->loop_groups ? 9 * 64 * 4 : 0);
    if (hipMalloc(&tw->block, (size_t)o) != hipSuccess) {
        (void)hipGetLastError();
        delete tw;
        return LSTM_DYN_ERR_NOMEM;
    }
    char* base = static_cast<char*>(tw->block);
    tw->save_h = reinterpret_cast<float*>(base + oh);
    tw->save_c = reinterpret_cast<float*>(base + oc);
    tw->xc = reinterpret_cast<float*>(base + ox);
    tw->w_il = reinterpret_cast<float*>(base + ow);
    tw->u_il = reinterpret_cast<float*>(base + ou);
    tw->dw_il = reinterpret_cast<float*>(base + odw);
    tw->du_il = reinterpret_cast<float*>(base + odu);
    tw->db_il = reinterpret_cast<float*>(base + odb);
    tw->cs_part = reinterpret_cast<float*>(base + ocs);
    tw->dH = reinterpret_cast<float*>(base + odh);
    tw->dC = reinterpret_cast<float*>(base + odc);
    tw->z = reinterpret_cast<float*>(base + oz);
    tw->dz16 = h16 ? reinterpret_cast<_Float16*>(base + odz16) : nullptr;
    tw->x16 = h16 ? reinterpret_cast<_Float16*>(base + ox16) : nullptr;
    tw->h16 = h16 ? reinterpret_cast<_Float16*>(base + oh16) : nullptr;
    tw->w16 = h16 ? reinterpret_cast<_Float16*>(base + ow16) : nullptr;
    tw->u16 = h16 ? reinterpret_cast<_Float16*>(base + ou16) : nullptr;
    tw->dzs16 = h16 ? reinterpret_cast<_Float16*>(base + odzs) : nullptr;
    tw->srow = reinterpret_cast<float*>(base + osr);
    tw->amax = reinterpret_cast<unsigned*>(base + osm);
    tw->dzx = one_launch ? reinterpret_cast<_Float16*>(base + odzx) : nullptr;
    tw->dzs = one_launch ? reinterpret_cast<float*>(base + odzsc) : nullptr;
    tw->pdh = tw->block_groups ? reinterpret_cast<float*>(base + opdh) : nullptr;
    tw->bar = tw->loop_groups ? reinterpret_cast<unsigned*>(base + obar) : nullptr;
    if (hipHostMalloc(reinterpret_cast<void**>(&tw->host_offsets), (size_t)(T + 8) * sizeof(int32_t),
                      hipHostMallocDefault) != hipSuccess) {
        (void)hipFree(tw->block);
        delete tw;
        return LSTM_DYN_ERR_HIP;
    }
    // no atomics in rocBLAS's kernels: the same inputs give the same
    // gradients bit for bit
    if (!load_rocblas() || g_rb.create_handle(&tw->rb) != rocblas_status_success ||
        g_rb.set_atomics_mode(tw->rb, rocblas_atomics_not_allowed) != rocblas_status_success) {
        (void)hipFree(tw->block);
        (void)hipHostFree(tw->host_offsets);
        delete tw;
        return LSTM_DYN_ERR_HIP;
    }
    h->train = tw;
    h->workspace += o;
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_forward_train(lstm_dyn_t* h, const void* x, const int32_t* lengths,
                                      const void* W, const void* U, const float* b,
                                      const float* h0, const float* c0, float* out_h,
                                      float* out_c, float* out_seq, void* stream) {
    if (!h) return LSTM_DYN_ERR_INVALID;
    const int rc = out_seq ? check_seq_args_cell(h->B, h->D, h->H, h->T, h->dtype, h->cell, x,
                                                 lengths, W, U, b, h0, c0, out_h, out_c, out_seq)
                           : check_args_cell(h->B, h->D, h->H, h->T, h->dtype, h->cell, x, lengths,
                                             W, U, b, h0, c0, out_h, out_c);
    if (rc != LSTM_DYN_OK) return rc;
    if (out_h == h0 || (h->cell == LSTM_DYN_CELL_LSTM && out_c == c0))
        return LSTM_DYN_ERR_INVALID;  // the backward reads h0, c0
    const int trc = ensure_train(h);
    if (trc != LSTM_DYN_OK) return trc;
    TrainWs* tw = h->train;
    hipStream_t s = static_cast<hipStream_t>(stream);
    h->last_stream = s;
    h->has_work = 1;
    h->launches_last = 0;
    h->saved = 0;
    const Dims& d = h->dims;
#define LD_CHECK(call)              \
    do {                            \
        if ((call) != hipSuccess) { \
            (void)hipGetLastError(); \
            return LSTM_DYN_ERR_HIP; \
        }                           \
    } while (0)
    auto mark = [&](int i) { return h->timing ? hipEventRecord(h->ev[i], s) : hipSuccess; };
    LD_CHECK(mark(0));
    if (h->cell != LSTM_DYN_CELL_LSTM) {
        // the cell's weights in the four-block layout (the backward uses them too)
        LD_CHECK(launch_cell_pack(d, W, U, b, h->w4, h->u4, h->b4, s));
        W = h->w4;
        U = h->u4;
        b = h->b4;
        h->launches_last++;
    }
    LD_CHECK(launch_prep(d, lengths, h->ws, s));
    LD_CHECK(mark(1));
    h->launches_last++;
    if (h->mode == LSTM_DYN_PERSISTENT && !h->plan.single && h->save_ok) {
        LD_CHECK(input_projection(h, x, W, b, s));
        LD_CHECK(mark(2));
        PersistentConfig pc{h->plan.mt,     h->plan.groups,    h->plan.ksw, h->plan.kw,
                            h->plan.nstate, h->plan.lds_bytes, h->timeout_ticks, h->trace,
                            nullptr,        nullptr,           tw->save_h,  tw->save_c};
        LD_CHECK(launch_persistent(d, pc, U, h0, c0, out_h, out_c, h->ws, s));
        h->launches_last++;
    } else {
        // the per-step kernels (single-workgroup sizes, per-step handles)
        Workspace ws = h->ws;
        if (!ws.z) ws.z = tw->z;
        LD_CHECK(launch_step_init(d, h0, c0, out_h, out_c, ws, s));
        h->launches_last++;
        LD_CHECK(input_projection(h, x, W, b, s));
        LD_CHECK(mark(2));
        LD_CHECK(hipMemcpyAsync(h->host_maxlen, &ws.meta->max_len, sizeof(int32_t),
                                hipMemcpyDeviceToHost, s));
        LD_CHECK(hipStreamSynchronize(s));
        const int max_len = *h->host_maxlen;
        for (int t = 0; t < max_len; ++t) {
            LD_CHECK(launch_step_gemm(d, t, U, ws, s));
            LD_CHECK(launch_step_gates(d, t, out_h, out_c, nullptr, false, ws, s, tw->save_h, tw->save_c));
            h->launches_last += 2;
        }
    }
    LD_CHECK(mark(3));
    if (out_seq) {
        LD_CHECK(launch_seq_from_saved(d, out_seq, tw->save_h, out_h, lengths, h->ws, h->num_cus, s));
        h->launches_last++;
    }
#undef LD_CHECK
    h->saved = 1;
    return LSTM_DYN_OK;
}

static int check_backward_args(int B, int D, int H, int T, int dtype, int cell, const void* x,
                               const int32_t* lengths, const void* W, const void* U,
                               const float* b, const float* h0, const float* c0,
                               const float* d_out_h, const float* d_out_c, const float* d_seq,
                               const float* dx, const float* dW, const float* dU,
                               const float* db, const float* dh0, const float* dc0) {
    if (B < 1 || D < 1 || H < 1 || T < 1) return LSTM_DYN_ERR_INVALID;
    if (dtype != LSTM_DYN_F32 && dtype != LSTM_DYN_BF16) return LSTM_DYN_ERR_INVALID;
    if (!valid_cell(cell)) return LSTM_DYN_ERR_INVALID;
    const bool has_c = cell == LSTM_DYN_CELL_LSTM;  // GRU, RNN: c0, d_out_c, dc0 may be NULL
    if (!has_c) {
        c0 = nullptr;
        d_out_c = nullptr;
    }
    const void* ins[] = {x, lengths, W, U, b, h0, c0, d_out_h, d_out_c, d_seq};
    const void* outs[] = {dx, dW, dU, db, dh0, dc0};
    const long long e = dtype == LSTM_DYN_BF16 ? 2 : 4;
    const long long G = (long long)cell_cols(cell) * H, nb = 4LL * cell_bias(cell) * H;
    const long long nin[] = {(long long)B * T * D * e, 4LL * B, (long long)D * G * e,
                             (long long)H * G * e, nb, 4LL * B * H, 4LL * B * H,
                             4LL * B * H, 4LL * B * H, d_seq ? 4LL * B * T * H : 0};
    const long long nout[] = {4LL * B * T * D, 4LL * D * G, 4LL * H * G, nb, 4LL * B * H,
                              4LL * B * H};
    for (int i = 0; i < 10; ++i) {
        const bool optional = i == 9 || (!has_c && (i == 6 || i == 8));
        if (!ins[i] && !optional) return LSTM_DYN_ERR_INVALID;
        if (ins[i] && (reinterpret_cast<uintptr_t>(ins[i]) & 3)) return LSTM_DYN_ERR_INVALID;
    }
    for (int i = 0; i < 6; ++i) {
        if (!outs[i]) {
            if (i == 5 && !has_c) continue;
            return LSTM_DYN_ERR_INVALID;
        }
        if (reinterpret_cast<uintptr_t>(outs[i]) & 3) return LSTM_DYN_ERR_INVALID;
        for (int j = 0; j < 10; ++j)
            if (ins[j] && overlaps(outs[i], nout[i], ins[j], nin[j])) return LSTM_DYN_ERR_INVALID;
        for (int j = 0; j < i; ++j)
            if (outs[j] && overlaps(outs[i], nout[i], outs[j], nout[j])) return LSTM_DYN_ERR_INVALID;
    }
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_check_backward_args(int B, int D, int H, int T, int dtype, int cell,
                                            const void* x, const int32_t* lengths, const void* W,
                                            const void* U, const float* b, const float* h0,
                                            const float* c0, const float* d_out_h,
                                            const float* d_out_c, const float* d_seq,
                                            const float* dx, const float* dW, const float* dU,
                                            const float* db, const float* dh0, const float* dc0) {
    return check_backward_args(B, D, H, T, dtype, cell, x, lengths, W, U, b, h0, c0, d_out_h,
                               d_out_c, d_seq, dx, dW, dU, db, dh0, dc0);
}

extern "C" int lstm_dyn_backward(lstm_dyn_t* h, const void* x, const int32_t* lengths,
                                 const void* W, const void* U, const float* b, const float* h0,
                                 const float* c0, const float* d_out_h, const float* d_out_c,
                                 const float* d_seq, float* dx, float* dW, float* dU, float* db,
                                 float* dh0, float* dc0, void* stream) {
    if (!h) return LSTM_DYN_ERR_INVALID;
    const int rc = check_backward_args(h->B, h->D, h->H, h->T, h->dtype, h->cell, x, lengths, W,
                                       U, b, h0, c0, d_out_h, d_out_c, d_seq, dx, dW, dU, db, dh0,
                                       dc0);
    if (rc != LSTM_DYN_OK) return rc;
    if (!h->saved || !h->train) return LSTM_DYN_ERR_INVALID;  // needs a forward for training
    const bool packed = h->cell != LSTM_DYN_CELL_LSTM;
    if (packed) {  // the four-block weights the forward for training packed
        W = h->w4;
        U = h->u4;
        d_out_c = nullptr;
    }
    // GRU: the cell kernel leaves h's direct path to h' in dH, the product adds to it
    const float beta = h->cell == LSTM_DYN_CELL_GRU ? 1.0f : 0.0f;
    TrainWs* tw = h->train;
    hipStream_t s = static_cast<hipStream_t>(stream);
    h->last_stream = s;
    h->has_work = 1;
    h->launches_last = 0;
    h->saved = 0;  // the backward overwrites the kept pre-activations
    const Dims& d = h->dims;
    const int H4 = 4 * d.H;
#define LD_CHECK(call)              \
    do {                            \
        if ((call) != hipSuccess) { \
            (void)hipGetLastError(); \
            return LSTM_DYN_ERR_HIP; \
        }                           \
    } while (0)
#define RB_CHECK(call)                                 \
    do {                                               \
        if ((call) != rocblas_status_success) return LSTM_DYN_ERR_HIP; \
    } while (0)
    RB_CHECK(g_rb.set_stream(tw->rb, s));
    LD_CHECK(launch_bwd_weights(d, W, d.D, tw->w_il, s));
    LD_CHECK(launch_bwd_weights(d, U, d.H, tw->u_il, s));
    h->launches_last += 2;
    if (d.bf16) {  // the largest |U|, for U's fp16 scale
        LD_CHECK(hipMemsetAsync(tw->amax, 0, 5 * sizeof(unsigned), s));
        LD_CHECK(launch_bwd_absmax(tw->u_il, (long)d.H * H4, tw->amax + 4, s));
        LD_CHECK(hipMemcpyAsync(tw->host_offsets + d.T + 2, tw->amax + 4, sizeof(unsigned),
                                hipMemcpyDeviceToHost, s));
        h->launches_last++;
    }
    // step offsets and the sum of lengths of the forward, on the host
    LD_CHECK(hipMemcpyAsync(tw->host_offsets, h->ws.offsets, (size_t)(d.T + 1) * sizeof(int32_t),
                            hipMemcpyDeviceToHost, s));
    LD_CHECK(hipMemcpyAsync(tw->host_offsets + d.T + 1, &h->ws.meta->total_rows, sizeof(int32_t),
                            hipMemcpyDeviceToHost, s));
    LD_CHECK(hipMemcpyAsync(h->host_maxlen, &h->ws.meta->max_len, sizeof(int32_t),
                            hipMemcpyDeviceToHost, s));
    LD_CHECK(hipStreamSynchronize(s));
    const int32_t* off = tw->host_offsets;
    const int rows = off[d.T + 1], max_len = *h->host_maxlen;
    const float one = 1.0f, zero = 0.0f;
    LD_CHECK(launch_bwd_init(d, d_out_h, d_out_c, tw->dH, tw->dC, h->ws, s));
    h->launches_last++;
    if (!d.bf16) {
        for (int t = max_len - 1; t >= 0; --t) {
            const int act = off[t + 1] - off[t];
            LD_CHECK(launch_bwd_cell(d, t, off[t], act, tw->save_h, tw->save_c, d_seq, tw->dH,
                                     tw->dC, h->ws, s));
            // dH[0:act] (+)= dz_t U^T (column-major: dH^T = U_il^T-as-stored^T dz_t^T)
            RB_CHECK(g_rb.sgemm(tw->rb, rocblas_operation_transpose, rocblas_operation_none, d.H,
                                   act, H4, &one, tw->u_il, H4, h->ws.gx + (size_t)off[t] * H4, H4,
                                   &beta, tw->dH, d.H));
            h->launches_last += 2;
        }
        LD_CHECK(launch_bwd_state_out(d, tw->dH, tw->dC, nullptr, dh0, dc0, h->ws, s));
    } else {
        // bf16 data: dh = dz U^T on fp16 operands, U scaled once, each row's dz
        // by its own power of two (kept in srow and divided out when dH is read)
        const float su = f16_scale(static_cast<unsigned>(off[d.T + 2])), alpha_u = 1.0f / su;
        LD_CHECK(launch_bwd_to_f16(tw->u_il, tw->u16, (long)d.H * H4, su, s));
        h->launches_last++;
        // The whole reverse loop in one cooperative launch where U splits into
        // column blocks; else the steps with at most BWD_LOOP_ROWS rows (the
        // last ones, taken first) in one, which leaves dH complete and
        // unscaled for the step before them, and the others two launches each.
        int t_end = max_len;
        if (tw->block_groups) {
            // the published dz, its scales and the shares of dh start as the
            // marker (all ones)
            LD_CHECK(hipMemsetAsync(tw->dzx, 0xff, (size_t)tw->dzx_bytes, s));
            LD_CHECK(hipMemsetAsync(tw->dzs, 0xff, (size_t)tw->dzs_bytes, s));
            LD_CHECK(hipMemsetAsync(tw->pdh, 0xff, (size_t)tw->pdh_bytes, s));
            LD_CHECK(launch_bwd_block(d, tw->u16, alpha_u, tw->save_h, tw->save_c, d_seq, tw->dH, tw->dC,
                                      tw->dzx, tw->dzs, tw->pdh, tw->amax + 0, h->timeout_ticks, h->trace,
                                      h->ws, s));
            h->launches_last++;
            t_end = 0;
        } else if (tw->loop_groups) {
            while (t_end > 0 && off[t_end] - off[t_end - 1] <= BWD_LOOP_ROWS) --t_end;
        }
        if (!tw->block_groups && t_end < max_len) {
            LD_CHECK(hipMemsetAsync(tw->dzx, 0, (size_t)tw->dzx_bytes, s));
            LD_CHECK(hipMemsetAsync(tw->dzs, 0, (size_t)tw->dzs_bytes, s));
            LD_CHECK(hipMemsetAsync(tw->bar, 0, 9 * 64 * sizeof(unsigned), s));
            LD_CHECK(launch_bwd_loop(d, tw->u16, alpha_u, tw->save_h, tw->save_c, d_seq, tw->dH,
                                     tw->dC, tw->dzx, tw->dzs, tw->bar, h->timeout_ticks, t_end,
                                     h->ws, s));
            h->launches_last++;
        }
        LD_CHECK(launch_bwd_ones(tw->srow, d.B, s));
        h->launches_last++;
        for (int t = t_end - 1; t >= 0; --t) {
            const int act = off[t + 1] - off[t];
            LD_CHECK(launch_bwd_cell16(d, t, off[t], act, tw->save_h, tw->save_c, d_seq, tw->dH,
                                       tw->dC, tw->srow, tw->dzs16, h->ws, s));
            RB_CHECK(g_rb.gemm_ex(tw->rb, rocblas_operation_transpose, rocblas_operation_none,
                                     d.H, act, H4, &alpha_u, tw->u16, rocblas_datatype_f16_r, H4,
                                     tw->dzs16, rocblas_datatype_f16_r, H4, &beta, tw->dH,
                                     rocblas_datatype_f32_r, d.H, tw->dH, rocblas_datatype_f32_r,
                                     d.H, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0));
            h->launches_last += 2;
        }
        LD_CHECK(launch_bwd_state_out(d, tw->dH, tw->dC, tw->srow, dh0, dc0, h->ws, s));
    }
    h->launches_last++;
    if (rows > 0) {
        // (bf16: the largest |x| of the rows for x's fp16 scale, in the same pass)
        LD_CHECK(launch_bwd_gather_x(d, x, rows, tw->xc, d.bf16 ? tw->amax + 1 : nullptr, h->ws, s));
        h->launches_last++;
        if (!d.bf16) {
            // db = dz^T 1 (K = the sum of lengths)
            LD_CHECK(launch_bwd_colsum(h->ws.gx, rows, H4, tw->cs_part, tw->db_il, nullptr, 1.0f, s));
            h->launches_last += 2;
            // dW = X^T dz, dU = H_prev^T dz, then dx rows = dz W^T over the gathered x
            RB_CHECK(g_rb.sgemm(tw->rb, rocblas_operation_none, rocblas_operation_transpose, H4,
                                   d.D, rows, &one, h->ws.gx, H4, tw->xc, d.D, &zero, tw->dw_il, H4));
            RB_CHECK(g_rb.sgemm(tw->rb, rocblas_operation_none, rocblas_operation_transpose, H4,
                                   d.H, rows, &one, h->ws.gx, H4, tw->save_h, d.H, &zero, tw->du_il,
                                   H4));
            RB_CHECK(g_rb.sgemm(tw->rb, rocblas_operation_transpose, rocblas_operation_none, d.D,
                                   rows, H4, &one, tw->w_il, H4, h->ws.gx, H4, &zero, tw->xc, d.D));
            h->launches_last += 3;
        } else {
            // bf16 data: the same GEMMs on fp16 operands, each scaled by a power
            // of two (its largest magnitude into [2^13, 2^14)), fp32 accumulation,
            // alpha undoing the scales
            const long n_dz = (long)rows * H4, n_x = (long)rows * d.D, n_h = (long)rows * d.H,
                       n_w = (long)d.D * H4;
            // (the whole-loop launch took the largest |dz| as it went, and the
            // gather of x its largest |x|)
            if (!tw->block_groups) LD_CHECK(launch_bwd_absmax(h->ws.gx, n_dz, tw->amax + 0, s));
            LD_CHECK(launch_bwd_absmax(tw->save_h, n_h, tw->amax + 2, s));
            LD_CHECK(launch_bwd_absmax(tw->w_il, n_w, tw->amax + 3, s));
            unsigned* am = reinterpret_cast<unsigned*>(tw->host_offsets + d.T + 3);
            LD_CHECK(hipMemcpyAsync(am, tw->amax, 4 * sizeof(unsigned), hipMemcpyDeviceToHost, s));
            LD_CHECK(hipStreamSynchronize(s));
            const float sz = f16_scale(am[0]), sx = f16_scale(am[1]), sh = f16_scale(am[2]),
                        sw = f16_scale(am[3]);
            // db and the fp16 dz in one pass over dz
            LD_CHECK(launch_bwd_colsum(h->ws.gx, rows, H4, tw->cs_part, tw->db_il, tw->dz16, sz, s));
            LD_CHECK(launch_bwd_to_f16(tw->xc, tw->x16, n_x, sx, s));
            LD_CHECK(launch_bwd_to_f16(tw->save_h, tw->h16, n_h, sh, s));
            LD_CHECK(launch_bwd_to_f16(tw->w_il, tw->w16, n_w, sw, s));
            const rocblas_datatype f16 = rocblas_datatype_f16_r, f32 = rocblas_datatype_f32_r;
            const float a_w = 1.0f / (sz * sx), a_u = 1.0f / (sz * sh), a_x = 1.0f / (sz * sw);
            RB_CHECK(g_rb.gemm_ex(tw->rb, rocblas_operation_none, rocblas_operation_transpose, H4,
                                     d.D, rows, &a_w, tw->dz16, f16, H4, tw->x16, f16, d.D, &zero,
                                     tw->dw_il, f32, H4, tw->dw_il, f32, H4, f32,
                                     rocblas_gemm_algo_standard, 0, 0));
            RB_CHECK(g_rb.gemm_ex(tw->rb, rocblas_operation_none, rocblas_operation_transpose, H4,
                                     d.H, rows, &a_u, tw->dz16, f16, H4, tw->h16, f16, d.H, &zero,
                                     tw->du_il, f32, H4, tw->du_il, f32, H4, f32,
                                     rocblas_gemm_algo_standard, 0, 0));
            RB_CHECK(g_rb.gemm_ex(tw->rb, rocblas_operation_transpose, rocblas_operation_none, d.D,
                                     rows, H4, &a_x, tw->w16, f16, H4, tw->dz16, f16, H4, &zero,
                                     tw->xc, f32, d.D, tw->xc, f32, d.D, f32,
                                     rocblas_gemm_algo_standard, 0, 0));
            h->launches_last += tw->block_groups ? 10 : 11;
        }
    } else {
        LD_CHECK(hipMemsetAsync(tw->dw_il, 0, (size_t)d.D * H4 * sizeof(float), s));
        LD_CHECK(hipMemsetAsync(tw->du_il, 0, (size_t)d.H * H4 * sizeof(float), s));
        LD_CHECK(hipMemsetAsync(tw->db_il, 0, (size_t)H4 * sizeof(float), s));
    }
    if (!packed) {
        LD_CHECK(launch_bwd_permute(d, tw->dw_il, dW, d.D, s));
        LD_CHECK(launch_bwd_permute(d, tw->du_il, dU, d.H, s));
        LD_CHECK(launch_bwd_permute(d, tw->db_il, db, 1, s));
    } else {
        // from the four blocks to the cell's layout; the GRU's two bias vectors
        // take the input and the recurrent side of the packed bias gradient
        LD_CHECK(launch_bwd_unpack(d, tw->dw_il, dW, d.D, 0, s));
        LD_CHECK(launch_bwd_unpack(d, tw->du_il, dU, d.H, 1, s));
        LD_CHECK(launch_bwd_unpack(d, tw->db_il, db, 1, 0, s));
        if (h->cell == LSTM_DYN_CELL_GRU) LD_CHECK(launch_bwd_unpack(d, tw->db_il, db + 3 * d.H, 1, 1, s));
    }
    LD_CHECK(launch_bwd_dx(d, tw->xc, rows, lengths, dx, h->ws, s));
    h->launches_last += 4;
#undef RB_CHECK
#undef LD_CHECK
    return LSTM_DYN_OK;
}

extern "C" int lstm_dyn_query(lstm_dyn_t* h, int what, long long* value) {
    if (!h || !value) return LSTM_DYN_ERR_INVALID;
    switch (what) {
        case LSTM_DYN_Q_LAUNCHES_PER_FORWARD: *value = h->launches_last; return LSTM_DYN_OK;
        case LSTM_DYN_Q_GROUPS: *value = h->plan.groups; return LSTM_DYN_OK;
        case LSTM_DYN_Q_WORKSPACE_BYTES: *value = h->workspace; return LSTM_DYN_OK;
        case LSTM_DYN_Q_LAST_STATUS:
        case LSTM_DYN_Q_STEPS_EXECUTED:
        case LSTM_DYN_Q_TOTAL_ROWS: {
            if (hipStreamSynchronize(h->last_stream) != hipSuccess) return LSTM_DYN_ERR_HIP;
            Meta m;
            if (hipMemcpy(&m, h->ws.meta, sizeof(Meta), hipMemcpyDeviceToHost) != hipSuccess)
                return LSTM_DYN_ERR_HIP;
            if (what == LSTM_DYN_Q_STEPS_EXECUTED) *value = m.iters;
            else if (what == LSTM_DYN_Q_TOTAL_ROWS) *value = m.total_rows;
            else if (m.status & STATUS_TIMEOUT) *value = LSTM_DYN_ERR_TIMEOUT;
            else if (m.status & STATUS_BAD_LENGTHS) *value = LSTM_DYN_ERR_BAD_LENGTHS;
            else *value = LSTM_DYN_OK;
            return LSTM_DYN_OK;
        }
        case LSTM_DYN_Q_TIME_PREP_NS:
        case LSTM_DYN_Q_TIME_INPROJ_NS:
        case LSTM_DYN_Q_TIME_LOOP_NS: {
            if (!h->timing) return LSTM_DYN_ERR_INVALID;
            const int i = what - LSTM_DYN_Q_TIME_PREP_NS;
            if (hipEventSynchronize(h->ev[i + 1]) != hipSuccess) return LSTM_DYN_ERR_HIP;
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, h->ev[i], h->ev[i + 1]) != hipSuccess) return LSTM_DYN_ERR_HIP;
            *value = (long long)(ms * 1e6);
            return LSTM_DYN_OK;
        }
        default: return LSTM_DYN_ERR_INVALID;
    }
}
