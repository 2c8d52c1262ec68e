// step.hip -- kernels of the per-step comparison path.
//
// The paper compares the staged loop against running the same loop body one
// operation at a time from the host (Section 9, Table 1, "Eager").  This path
// keeps the math and the data layout of the persistent path but launches two
// kernels per step from a host loop: the recurrent product h U + Gx[t]
// (gemm.hip, MODE_STEP) and the gate update below.
#include "launch.h"

namespace ldyn {

// out_h/out_c <- h0/c0 (batch order); operand buffer <- h0 in slot order.
template <typename E>
__global__ void __launch_bounds__(256)
step_init_kernel(const float* __restrict__ h0, const float* __restrict__ c0, float* out_h,
                 float* out_c, const int32_t* __restrict__ perm, typename E::store_t* hx,
                 int B, int H, int hpad, int cell) {
    const long n = (long)B * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const int b = perm[s];
        const float hv = h0[(long)b * H + u];
        hx[(long)s * hpad + u] = E::from_f32(hv);
        // Exact aliasing out_h == h0 is allowed: each element is read before it is written.
        const long ib = (long)b * H + u;
        out_h[ib] = hv;
        out_c[ib] = cell == CELL_LSTM ? c0[ib] : 0.0f;  // only the LSTM has a cell state
    }
}

// Gate update of the rows active at step t (slots [0, active(t))).
template <typename E>
__global__ void __launch_bounds__(256)
step_gates_kernel(const float* __restrict__ z, float* out_h, float* out_c,
                  const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
                  typename E::store_t* hx, int t, int H, int hpad, float* seq, int T, int cell) {
    const int act = offsets[t + 1] - offsets[t];
    const long n = (long)act * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const int b = perm[s];
        const f32x4_t zz = *reinterpret_cast<const f32x4_t*>(z + (long)s * 4 * H + 4 * u);
        const long ib = (long)b * H + u;
        float c = out_c[ib], h = out_h[ib];
        apply_cell(cell, zz, c, h);
        out_c[ib] = c;
        out_h[ib] = h;
        hx[(long)s * hpad + u] = E::from_f32(h);
        if (seq) seq[((size_t)b * T + t) * H + u] = h;  // the output sequence at step t
    }
}

static int grid_for(long n) {
    long g = (n + 255) / 256;
    if (g < 1) g = 1;
    if (g > 4096) g = 4096;
    return (int)g;
}

hipError_t launch_step_init(const Dims& d, const float* h0, const float* c0, float* out_h,
                            float* out_c, const Workspace& ws, hipStream_t s) {
    const int grid = grid_for((long)d.B * d.H);
    if (d.bf16)
        hipLaunchKernelGGL(step_init_kernel<EltH16>, dim3(grid), dim3(256), 0, s, h0, c0, out_h,
                           out_c, ws.perm, static_cast<_Float16*>(ws.hx), d.B, d.H, d.hpad, d.cell);
    else
        hipLaunchKernelGGL(step_init_kernel<EltF32>, dim3(grid), dim3(256), 0, s, h0, c0, out_h,
                           out_c, ws.perm, static_cast<float*>(ws.hx), d.B, d.H, d.hpad, d.cell);
    return hipGetLastError();
}

hipError_t launch_step_gates(const Dims& d, int t, float* out_h, float* out_c, float* seq,
                             const Workspace& ws, hipStream_t s) {
    const int grid = grid_for((long)d.B * d.H);
    if (d.bf16)
        hipLaunchKernelGGL(step_gates_kernel<EltH16>, dim3(grid), dim3(256), 0, s, ws.z, out_h,
                           out_c, ws.perm, ws.offsets, static_cast<_Float16*>(ws.hx), t, d.H, d.hpad, seq, d.T, d.cell);
    else
        hipLaunchKernelGGL(step_gates_kernel<EltF32>, dim3(grid), dim3(256), 0, s, ws.z, out_h,
                           out_c, ws.perm, ws.offsets, static_cast<float*>(ws.hx), t, d.H, d.hpad, seq, d.T, d.cell);
    return hipGetLastError();
}

}  // namespace ldyn
