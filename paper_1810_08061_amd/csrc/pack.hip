// pack.hip -- GRU and tanh-RNN weights in the LSTM's four-gate-block layout.
//
// The paper's loop takes the cell as a parameter (Section 9 "RNN cells").
// Every kernel of this library reads W [D][4H], U [H][4H] and b [4H] as four
// gate blocks of H columns and hands each hidden unit its four
// pre-activations; the gate step then applies the cell's update to them.
//
// GRU: a unit has three gate blocks (r, u, n), and its n block needs the
// input and recurrent parts separately (the reset gate scales only the
// recurrent part), so the four blocks carry r, u, the recurrent part of n and
// the input part of n, with zero weights where a part has no term:
//   W4 = (W_r, W_u, 0, W_n),  U4 = (U_r, U_u, U_n, 0),
//   b4 = (b_ir + b_hr, b_iu + b_hu, b_hn, b_in).
// RNN: one pre-activation per unit in block 0, zeros elsewhere:
//   W4 = (W, 0, 0, 0),  U4 = (U, 0, 0, 0),  b4 = (b, 0, 0, 0).
// One pass per forward; the three zero blocks of the RNN cost MFMA work (the
// loop is bound by the exchange of h, not by the products, at the sizes it is
// built for).
#include "launch.h"

namespace ldyn {

// Source column (in the caller's W or U, G columns per row) of packed column
// (g, u), or -1 for a zero column.
__device__ inline int w_src(int cell, int g, int u, int H) {
    if (cell == CELL_RNN) return g == 0 ? u : -1;
    return g == 2 ? -1 : (g == 3 ? 2 : g) * H + u;  // GRU: (r, u, 0, n)
}
__device__ inline int u_src(int cell, int g, int u, int H) {
    if (cell == CELL_RNN) return g == 0 ? u : -1;
    return g == 3 ? -1 : g * H + u;  // GRU: (r, u, n, 0)
}

template <typename S>
__global__ void __launch_bounds__(256)
cell_pack_kernel(const S* __restrict__ W, const S* __restrict__ U, const float* __restrict__ b,
                 S* __restrict__ W4, S* __restrict__ U4, float* __restrict__ b4, int D, int H,
                 int cell) {
    const int G = cell == CELL_RNN ? H : 3 * H, H4 = 4 * H;
    const long nw = (long)D * H4, nu = (long)H * H4;
    const S zero = (S)0.0f;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < nw + nu + H4; i += (long)gridDim.x * 256) {
        if (i < nw) {
            const long k = i / H4;
            const int c = (int)(i - k * H4), g = c / H, u = c - g * H;
            const int src = w_src(cell, g, u, H);
            W4[i] = src < 0 ? zero : W[k * G + src];
        } else if (i < nw + nu) {
            const long j = i - nw, k = j / H4;
            const int c = (int)(j - k * H4), g = c / H, u = c - g * H;
            const int src = u_src(cell, g, u, H);
            U4[j] = src < 0 ? zero : U[k * G + src];
        } else {
            const int c = (int)(i - nw - nu), g = c / H, u = c - g * H;
            if (cell == CELL_RNN) {
                b4[c] = g == 0 ? b[u] : 0.0f;
            } else {
                const float* bih = b;
                const float* bhh = b + 3 * H;
                b4[c] = g < 2 ? bih[g * H + u] + bhh[g * H + u]
                              : g == 2 ? bhh[2 * H + u] : bih[2 * H + u];
            }
        }
    }
}

hipError_t launch_cell_pack(const Dims& d, const void* W, const void* U, const float* b, void* W4,
                            void* U4, float* b4, hipStream_t s) {
    if (d.cell != CELL_GRU && d.cell != CELL_RNN) return hipErrorInvalidValue;
    const long n = (long)d.D * 4 * d.H + (long)d.H * 4 * d.H + 4L * d.H;
    long grid = (n + 255) / 256;
    if (grid > 8192) grid = 8192;
    if (d.bf16)
        hipLaunchKernelGGL(cell_pack_kernel<__bf16>, dim3((unsigned)grid), dim3(256), 0, s,
                           static_cast<const __bf16*>(W), static_cast<const __bf16*>(U), b,
                           static_cast<__bf16*>(W4), static_cast<__bf16*>(U4), b4, d.D, d.H,
                           d.cell);
    else
        hipLaunchKernelGGL(cell_pack_kernel<float>, dim3((unsigned)grid), dim3(256), 0, s,
                           static_cast<const float*>(W), static_cast<const float*>(U), b,
                           static_cast<float*>(W4), static_cast<float*>(U4), b4, d.D, d.H,
                           d.cell);
    return hipGetLastError();
}

}  // namespace ldyn
