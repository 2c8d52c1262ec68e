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
// Rows that ended (stopped[b], termination from the state; null: none) keep
// their state.
template <typename E>
__global__ void __launch_bounds__(256)
step_gates_kernel(const float* __restrict__ z, float* out_h, float* out_c,
                  const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
                  typename E::store_t* hx, int t, int H, int hpad, float* seq, int T, int cell,
                  const int32_t* __restrict__ stopped, float* gx, float* save_h, float* save_c) {
    const int act = offsets[t + 1] - offsets[t];
    const long n = (long)act * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const int b = perm[s];
        if (stopped && stopped[b]) continue;
        const f32x4_t zz = *reinterpret_cast<const f32x4_t*>(z + (long)s * 4 * H + 4 * u);
        const long ib = (long)b * H + u;
        float c = out_c[ib], h = out_h[ib];
        if (save_h) {  // forward for training: z in place of Gx, the state the step starts from
            const long r = offsets[t] + s;
            *reinterpret_cast<f32x4_t*>(gx + r * 4 * H + 4 * u) = zz;
            save_h[r * H + u] = h;
            save_c[r * H + u] = c;
        }
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
                             bool stop, const Workspace& ws, hipStream_t s, float* save_h,
                             float* save_c) {
    const int grid = grid_for((long)d.B * d.H);
    const int32_t* stopped = stop ? ws.stopped : nullptr;
    if (d.bf16)
        hipLaunchKernelGGL(step_gates_kernel<EltH16>, dim3(grid), dim3(256), 0, s, ws.z, out_h,
                           out_c, ws.perm, ws.offsets, static_cast<_Float16*>(ws.hx), t, d.H, d.hpad, seq, d.T, d.cell,
                           stopped, ws.gx, save_h, save_c);
    else
        hipLaunchKernelGGL(step_gates_kernel<EltF32>, dim3(grid), dim3(256), 0, s, ws.z, out_h,
                           out_c, ws.perm, ws.offsets, static_cast<float*>(ws.hx), t, d.H, d.hpad, seq, d.T, d.cell,
                           stopped, ws.gx, save_h, save_c);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Termination from the state (the decoders of the paper's Appendix D leave
// their loop once every candidate has ended): a row ends after a step that
// leaves its halting score v . h + c positive.

__global__ void __launch_bounds__(256)
step_stop_init_kernel(const int32_t* __restrict__ lengths, int32_t* steps, int32_t* stopped,
                      int32_t* running, int B, int T) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < B) {
        steps[i] = min(max(lengths[i], 0), T);  // a row that never ends runs to its cap
        stopped[i] = 0;
    }
    if (i < T) running[i] = 0;
}

// One workgroup per row slot of step t.  The score is formed from the row's
// h operand as the next step's product reads it, k in a fixed order: each
// thread sums k = tid, tid + 256, ..., then a tree over the threads.
template <typename E>
__global__ void __launch_bounds__(256)
step_stop_kernel(const typename E::store_t* __restrict__ hx, const float* __restrict__ v, float c,
                 const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
                 int32_t* steps, int32_t* stopped, int32_t* running, int t, int H, int hpad,
                 int max_len) {
    __shared__ float red[256];
    const int s = blockIdx.x, tid = threadIdx.x;
    const int act = offsets[t + 1] - offsets[t];
    if (s >= act) return;  // uniform over the workgroup
    const int b = perm[s];
    if (stopped[b]) return;
    float acc = 0.f;
    for (int k = tid; k < H; k += 256) acc += v[k] * E::to_f32(hx[(long)s * hpad + k]);
    red[tid] = acc;
    __syncthreads();
    for (int span = 128; span > 0; span >>= 1) {
        if (tid < span) red[tid] += red[tid + span];
        __syncthreads();
    }
    if (tid == 0) {
        const int act1 = t + 1 < max_len ? offsets[t + 2] - offsets[t + 1] : 0;
        if (red[0] + c > 0.f) {
            stopped[b] = 1;
            steps[b] = t + 1;
        } else if (s < act1) {
            atomicAdd(&running[t], 1);
        }
    }
}

hipError_t launch_step_stop_init(const Dims& d, const StopArgs& stop, const Workspace& ws,
                                 hipStream_t s) {
    const int n = d.B > d.T ? d.B : d.T;
    hipLaunchKernelGGL(step_stop_init_kernel, dim3((n + 255) / 256), dim3(256), 0, s, stop.lengths,
                       stop.steps, ws.stopped, ws.running, d.B, d.T);
    return hipGetLastError();
}

hipError_t launch_step_stop(const Dims& d, int t, const StopArgs& stop, const Workspace& ws,
                            hipStream_t s) {
    if (d.bf16)
        hipLaunchKernelGGL(step_stop_kernel<EltH16>, dim3(d.B), dim3(256), 0, s,
                           static_cast<const _Float16*>(ws.hx), stop.v, stop.c, ws.perm, ws.offsets,
                           stop.steps, ws.stopped, ws.running, t, d.H, d.hpad, d.T);
    else
        hipLaunchKernelGGL(step_stop_kernel<EltF32>, dim3(d.B), dim3(256), 0, s,
                           static_cast<const float*>(ws.hx), stop.v, stop.c, ws.perm, ws.offsets,
                           stop.steps, ws.stopped, ws.running, t, d.H, d.hpad, d.T);
    return hipGetLastError();
}

}  // namespace ldyn
