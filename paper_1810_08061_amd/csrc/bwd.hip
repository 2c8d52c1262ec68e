// bwd.hip -- kernels of the backward pass of the masked LSTM loop.
//
// Backpropagation through time of the loop of the paper's Section 9 "RNN
// cells" experiment (the paper trains its staged models in-graph).  A step a
// row does not take passes its state through unchanged, so its gradient is
// the identity: going back from the last step, the rows of step t are the
// prefix [0, active(t)) of the length-sorted slot order, exactly as going
// forward, and rows outside it keep their gradient.
//
// The forward for training leaves, for every compact row r (one valid
// (b, t)), the pre-activations z in place of the row's Gx (gate-interleaved
// columns c' = 4u + gate) and the state (h, c) the step started from.  Each
// step back is then
//   * bwd_cell_kernel: dz of the step's rows from z, c_{t-1}, dh, dc (and the
//     gradient of the output sequence at t), written over z; dc <- dc_total f;
//   * dh <- dz U^T for those rows, a GEMM (K = 4H) issued by the host;
// and after the last one the weight gradients are GEMMs over all compact
// rows (K = sum of lengths): dW = X^T dz, dU = H_prev^T dz, db = column sums,
// dx = dz W^T, in gate-interleaved columns, permuted back to the caller's
// gate blocks at the end.
#include "launch.h"

namespace ldyn {

// W or U [rows][4H] (element type S, gate blocks) -> fp32 [rows][4H] with
// gate-interleaved columns.
template <typename S>
__global__ void __launch_bounds__(256)
bwd_weights_kernel(const S* __restrict__ W, float* __restrict__ Wil, int rows, int H) {
    const long n = (long)rows * 4 * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const long k = i / (4 * H);
        const int cp = (int)(i - k * 4 * H);
        Wil[i] = (float)W[k * 4 * H + gate_col(cp, H)];
    }
}

// Upstream gradients of the final state, batch order -> slot order.
__global__ void __launch_bounds__(256)
bwd_init_kernel(const float* __restrict__ dh_out, const float* __restrict__ dc_out,
                const int32_t* __restrict__ perm, float* dH, float* dC, int B, int H) {
    const long n = (long)B * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const long ib = (long)perm[s] * H + u;
        dH[i] = dh_out[ib];
        dC[i] = dc_out[ib];
    }
}

// The cell's backward for the rows of step t: one (row, unit) per thread.
__global__ void __launch_bounds__(256)
bwd_cell_kernel(float* gx, const float* __restrict__ save_c, const float* __restrict__ dseq,
                const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets, float* dH,
                float* dC, int t, int H, int T) {
    const int off = offsets[t], act = offsets[t + 1] - off;
    const long n = (long)act * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const long r = off + s;
        f32x4_t* zp = reinterpret_cast<f32x4_t*>(gx + r * 4 * H + 4 * u);
        const f32x4_t z = *zp;
        const float ig = sigmoid_f(z[0]), fg = sigmoid_f(z[1]);
        const float gg = tanh_f(z[2]), og = sigmoid_f(z[3]);
        const float cp = save_c[r * H + u];
        const float c = fg * cp + ig * gg;
        const float tc = tanh_f(c);
        float dh = dH[i];
        if (dseq) dh += dseq[((long)perm[s] * T + t) * H + u];
        const float d_o = dh * tc;
        const float dct = dC[i] + dh * og * (1.0f - tc * tc);
        f32x4_t dz;
        dz[0] = dct * gg * ig * (1.0f - ig);
        dz[1] = dct * cp * fg * (1.0f - fg);
        dz[2] = dct * ig * (1.0f - gg * gg);
        dz[3] = d_o * og * (1.0f - og);
        *zp = dz;
        dC[i] = dct * fg;
    }
}

// dh0, dc0: slot order -> batch order.
__global__ void __launch_bounds__(256)
bwd_state_out_kernel(const float* __restrict__ dH, const float* __restrict__ dC,
                     const int32_t* __restrict__ perm, float* dh0, float* dc0, int B, int H) {
    const long n = (long)B * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const long ib = (long)perm[s] * H + u;
        dh0[ib] = dH[i];
        dc0[ib] = dC[i];
    }
}

// x rows in the compact order, fp32.
template <typename S>
__global__ void __launch_bounds__(256)
bwd_gather_x_kernel(const S* __restrict__ x, const int32_t* __restrict__ rowsrc,
                    const Meta* __restrict__ meta, float* xc, int D) {
    const long n = (long)meta->total_rows * D;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const long r = i / D;
        const int k = (int)(i - r * D);
        xc[i] = (float)x[(long)rowsrc[r] * D + k];
    }
}

// db in interleaved columns: the sum of dz over the compact rows, in row
// order (one thread per column).
__global__ void __launch_bounds__(256)
bwd_colsum_kernel(const float* __restrict__ dz, const Meta* __restrict__ meta, float* db_il, int H4) {
    const int cp = blockIdx.x * 256 + threadIdx.x;
    if (cp >= H4) return;
    const long rows = meta->total_rows;
    float acc = 0.f;
    for (long r = 0; r < rows; ++r) acc += dz[r * H4 + cp];
    db_il[cp] = acc;
}

// Interleaved columns -> the caller's gate blocks: out[k][g H + u] = il[k][4u + g].
__global__ void __launch_bounds__(256)
bwd_permute_kernel(const float* __restrict__ il, float* out, int rows, int H) {
    const long n = (long)rows * 4 * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const long k = i / (4 * H);
        const int cp = (int)(i - k * 4 * H);
        out[k * 4 * H + gate_col(cp, H)] = il[i];
    }
}

// dx [B][T][D]: the compact rows' dz W^T at their (b, t), zero elsewhere.  The
// two loops write disjoint rows.
__global__ void __launch_bounds__(256)
bwd_dx_kernel(const float* __restrict__ dxc, const int32_t* __restrict__ rowsrc,
              const Meta* __restrict__ meta, const int32_t* __restrict__ lengths, float* dx, int B,
              int T, int D) {
    const long rows = meta->total_rows;
    const long n = rows * D;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const long r = i / D;
        const int k = (int)(i - r * D);
        dx[(long)rowsrc[r] * D + k] = dxc[i];
    }
    const long m = (long)B * T * D;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < m; i += (long)gridDim.x * 256) {
        const long bt = i / D;
        const int b = (int)(bt / T), t = (int)(bt - (long)b * T);
        if (t >= min(max(lengths[b], 0), T)) dx[i] = 0.0f;
    }
}

static unsigned grid_of(long n) {
    long g = (n + 255) / 256;
    if (g < 1) g = 1;
    if (g > 8192) g = 8192;
    return (unsigned)g;
}

hipError_t launch_bwd_weights(const Dims& d, const void* W, int rows, float* Wil, hipStream_t s) {
    const unsigned g = grid_of((long)rows * 4 * d.H);
    if (d.bf16)
        hipLaunchKernelGGL(bwd_weights_kernel<__bf16>, dim3(g), dim3(256), 0, s,
                           static_cast<const __bf16*>(W), Wil, rows, d.H);
    else
        hipLaunchKernelGGL(bwd_weights_kernel<float>, dim3(g), dim3(256), 0, s,
                           static_cast<const float*>(W), Wil, rows, d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_init(const Dims& d, const float* dh_out, const float* dc_out, float* dH,
                           float* dC, const Workspace& ws, hipStream_t s) {
    hipLaunchKernelGGL(bwd_init_kernel, dim3(grid_of((long)d.B * d.H)), dim3(256), 0, s, dh_out,
                       dc_out, ws.perm, dH, dC, d.B, d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_cell(const Dims& d, int t, int act, const float* save_c, const float* dseq,
                           float* dH, float* dC, const Workspace& ws, hipStream_t s) {
    hipLaunchKernelGGL(bwd_cell_kernel, dim3(grid_of((long)act * d.H)), dim3(256), 0, s, ws.gx,
                       save_c, dseq, ws.perm, ws.offsets, dH, dC, t, d.H, d.T);
    return hipGetLastError();
}

hipError_t launch_bwd_state_out(const Dims& d, const float* dH, const float* dC, float* dh0,
                                float* dc0, const Workspace& ws, hipStream_t s) {
    hipLaunchKernelGGL(bwd_state_out_kernel, dim3(grid_of((long)d.B * d.H)), dim3(256), 0, s, dH,
                       dC, ws.perm, dh0, dc0, d.B, d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_gather_x(const Dims& d, const void* x, long rows, float* xc,
                               const Workspace& ws, hipStream_t s) {
    const unsigned g = grid_of(rows * d.D);
    if (d.bf16)
        hipLaunchKernelGGL(bwd_gather_x_kernel<__bf16>, dim3(g), dim3(256), 0, s,
                           static_cast<const __bf16*>(x), ws.rowsrc, ws.meta, xc, d.D);
    else
        hipLaunchKernelGGL(bwd_gather_x_kernel<float>, dim3(g), dim3(256), 0, s,
                           static_cast<const float*>(x), ws.rowsrc, ws.meta, xc, d.D);
    return hipGetLastError();
}

hipError_t launch_bwd_colsum(const Dims& d, float* db_il, const Workspace& ws, hipStream_t s) {
    hipLaunchKernelGGL(bwd_colsum_kernel, dim3((4 * d.H + 255) / 256), dim3(256), 0, s, ws.gx,
                       ws.meta, db_il, 4 * d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_permute(const Dims& d, const float* il, float* out, int rows, hipStream_t s) {
    hipLaunchKernelGGL(bwd_permute_kernel, dim3(grid_of((long)rows * 4 * d.H)), dim3(256), 0, s, il,
                       out, rows, d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_dx(const Dims& d, const float* dxc, long rows, const int32_t* lengths,
                         float* dx, const Workspace& ws, hipStream_t s) {
    const long n = rows * d.D > (long)d.B * d.T * d.D ? rows * d.D : (long)d.B * d.T * d.D;
    hipLaunchKernelGGL(bwd_dx_kernel, dim3(grid_of(n)), dim3(256), 0, s, dxc, ws.rowsrc, ws.meta,
                       lengths, dx, d.B, d.T, d.D);
    return hipGetLastError();
}

}  // namespace ldyn
