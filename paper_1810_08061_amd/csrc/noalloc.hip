// noalloc.hip -- lstm_dyn_forward_noalloc: the persistent LSTM forward with
// its workspace in a fixed device array, for callers that cannot allocate.
//
// The kernels are those of lstm_dyn_forward (length preparation, input
// projection, the persistent loop, or the single-workgroup kernel for H <= 32);
// only the workspace differs: it is carved from `scratch`, a file-scope device
// array that every GPU the library runs on holds until the process ends.  In
// host code the array's name is only a stand-in for the symbol: its device
// address comes from hipGetSymbolAddress, taken once per device with that
// device current, and only that address is handed to kernels.
#include <mutex>

#include "../../include/lstm_dyn.h"
#include "launch.h"

namespace ldyn {

static_assert(LSTM_DYN_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
static __device__ __align__(256) unsigned char scratch[LSTM_DYN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int NOALLOC_MAX_DEVICES = 64;

struct DeviceScratch {
    char* ptr;       // device address of `scratch` on this device
    int num_cus;
    int wclk_khz;
    bool ready;
};
DeviceScratch g_dev[NOALLOC_MAX_DEVICES];
std::mutex g_mu;

// The scratch address and device facts of the current device (looked up at
// the first call on it).
int device_scratch(DeviceScratch* out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return LSTM_DYN_ERR_HIP;
    if (dev < 0 || dev >= NOALLOC_MAX_DEVICES) return LSTM_DYN_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_mu);
    DeviceScratch& d = g_dev[dev];
    if (!d.ready) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return LSTM_DYN_ERR_HIP;
        }
        int cus = 0, khz = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
            return LSTM_DYN_ERR_HIP;
        d.ptr = static_cast<char*>(p);
        d.num_cus = cus;
        d.wclk_khz = khz;
        d.ready = true;
    }
    *out = d;
    return LSTM_DYN_OK;
}

// Zero fill of the operand buffer (a kernel, not a memset, so the call can be
// captured in a graph).
__global__ void __launch_bounds__(256) zero_kernel(uint4* p, long n16) {
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n16; i += (long)gridDim.x * 256)
        p[i] = uint4{0u, 0u, 0u, 0u};
}

// The forward's device status as a C ABI status code.
__global__ void status_kernel(const Meta* meta, int32_t* out) {
    const int32_t s = meta->status;
    *out = (s & STATUS_TIMEOUT) ? LSTM_DYN_ERR_TIMEOUT
           : (s & STATUS_BAD_LENGTHS) ? LSTM_DYN_ERR_BAD_LENGTHS
                                      : LSTM_DYN_OK;
}

bool overlaps(const void* a, long long na, const void* b, long long nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

}  // namespace
}  // namespace ldyn

using namespace ldyn;

extern "C" int lstm_dyn_forward_noalloc(int B, int D, int H, int T, int dtype, const void* x,
                                        const int32_t* lengths, const void* W, const void* U,
                                        const float* b, const float* h0, const float* c0,
                                        float* out_h, float* out_c, int32_t* status,
                                        void* stream) {
    int rc = lstm_dyn_check_args(B, D, H, T, dtype, x, lengths, W, U, b, h0, c0, out_h, out_c);
    if (rc != LSTM_DYN_OK) return rc;
    const long long e = dtype == LSTM_DYN_BF16 ? 2 : 4;
    if (status) {
        if (reinterpret_cast<uintptr_t>(status) & 3) return LSTM_DYN_ERR_INVALID;
        const void* all[] = {x, lengths, W, U, b, h0, c0, out_h, out_c};
        const long long sz[] = {(long long)B * T * D * e, 4LL * B, (long long)D * 4 * H * e,
                                (long long)H * 4 * H * e, 16LL * H, 4LL * B * H, 4LL * B * H,
                                4LL * B * H, 4LL * B * H};
        for (int i = 0; i < 9; ++i)
            if (overlaps(status, 4, all[i], sz[i])) return LSTM_DYN_ERR_INVALID;
    }
    DeviceScratch ds;
    if ((rc = device_scratch(&ds)) != LSTM_DYN_OK) return rc;
    lstm_dyn_plan_t plan;
    if ((rc = lstm_dyn_plan(B, D, H, T, dtype, LSTM_DYN_PERSISTENT, ds.num_cus, &plan)) != LSTM_DYN_OK)
        return rc;
    const int bf16 = dtype == LSTM_DYN_BF16;
    const Dims d{B, D, H, T, bf16, plan.hpad, plan.bpad, CELL_LSTM};
    Workspace ws;
    long long hx_off = 0, hx_bytes = 0;
    const long long need = carve_forward_workspace(d, nullptr, &ws, &hx_off, &hx_bytes);
    if (need > LSTM_DYN_NOALLOC_SCRATCH_BYTES) return LSTM_DYN_ERR_TOO_LARGE;
    (void)carve_forward_workspace(d, ds.ptr, &ws, &hx_off, &hx_bytes);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const unsigned long long timeout_ticks = (unsigned long long)(5.0 * 1e3 * (double)ds.wclk_khz);
#define NA_CHECK(call)               \
    do {                             \
        if ((call) != hipSuccess) {  \
            (void)hipGetLastError(); \
            return LSTM_DYN_ERR_HIP; \
        }                            \
    } while (0)
    if (plan.single) {
        NA_CHECK(launch_small(d, plan.single_kd, plan.single_nt, x, lengths, W, U, b, h0, c0, out_h,
                              out_c, nullptr, nullptr, ws, s));
    } else {
        const int per_cu = persistent_blocks_per_cu(bf16, plan.mt, plan.ksw, plan.kw, plan.nstate,
                                                    plan.lds_bytes, CELL_LSTM, 0);
        if (per_cu < 1 || plan.groups > per_cu * ds.num_cus) return LSTM_DYN_ERR_UNSUPPORTED;
        // the operand buffer holds the previous call's values in another layout
        const long n16 = (long)(hx_bytes / 16);
        long zgrid = (n16 + 255) / 256;
        if (zgrid > 4L * ds.num_cus) zgrid = 4L * ds.num_cus;
        hipLaunchKernelGGL(zero_kernel, dim3((unsigned)zgrid), dim3(256), 0, s,
                           reinterpret_cast<uint4*>(ds.ptr + hx_off), n16);
        NA_CHECK(hipGetLastError());
        NA_CHECK(launch_prep(d, lengths, ws, s));
        if (bf16) {
            NA_CHECK(inproj_bf16_setup());
            const long long tiles = inproj_bf16_tiles_max(d);
            NA_CHECK(launch_transpose_w(d, W, ws, s));
            NA_CHECK(launch_inproj_bf16(d, x, b, ws, (int)(tiles < ds.num_cus ? tiles : ds.num_cus), s));
        } else {
            const long long tiles = ((long long)B * T + 127) / 128 * ((4LL * H + 127) / 128);
            NA_CHECK(launch_inproj(d, x, W, b, ws, (int)(tiles < 4LL * ds.num_cus ? tiles : 4LL * ds.num_cus), s));
        }
        PersistentConfig pc{plan.mt, plan.groups, plan.ksw, plan.kw, plan.nstate, plan.lds_bytes,
                            timeout_ticks, nullptr, nullptr, nullptr};
        NA_CHECK(launch_persistent(d, pc, U, h0, c0, out_h, out_c, ws, s));
    }
    if (status) {
        hipLaunchKernelGGL(status_kernel, dim3(1), dim3(1), 0, s, ws.meta, status);
        NA_CHECK(hipGetLastError());
    }
#undef NA_CHECK
    return LSTM_DYN_OK;
}
