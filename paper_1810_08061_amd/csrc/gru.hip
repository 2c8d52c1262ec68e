// gru.hip -- the GRU cell's weights in the LSTM's four-gate-block layout.
//
// The paper's loop takes the cell as a parameter (Section 9 "RNN cells").
// Every kernel of this library reads W [D][4H], U [H][4H] and b [4H] as four
// gate blocks of H columns and hands each hidden unit its four
// pre-activations.  A GRU unit has three gate blocks (r, u, n), and its n
// block needs the input and recurrent parts separately (the reset gate scales
// only the recurrent part), so the four blocks carry r, u, the recurrent part
// of n and the input part of n, with zero weights where a part has no term:
//   W4 [D][4H] = (W_r, W_u, 0, W_n),  U4 [H][4H] = (U_r, U_u, U_n, 0),
//   b4 [4H]    = (b_ir + b_hr, b_iu + b_hu, b_hn, b_in).
// One pass per forward; the rest of the path then runs unchanged, and the
// gate step of each kernel applies the GRU update to the four values.
#include "launch.h"

namespace ldyn {

template <typename S>
__global__ void __launch_bounds__(256)
gru_pack_kernel(const S* __restrict__ W, const S* __restrict__ U, const float* __restrict__ b,
                S* __restrict__ W4, S* __restrict__ U4, float* __restrict__ b4, int D, int H) {
    const int H3 = 3 * H, H4 = 4 * H;
    const long nw = (long)D * H4, nu = (long)H * H4;
    const S zero = (S)0.0f;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < nw + nu + H4; i += (long)gridDim.x * 256) {
        if (i < nw) {
            const long k = i / H4;
            const int c = (int)(i - k * H4), g = c / H, u = c - g * H;
            W4[i] = g == 2 ? zero : W[k * H3 + (g == 3 ? 2 : g) * H + u];
        } else if (i < nw + nu) {
            const long j = i - nw, k = j / H4;
            const int c = (int)(j - k * H4), g = c / H, u = c - g * H;
            U4[j] = g == 3 ? zero : U[k * H3 + g * H + u];
        } else {
            const int c = (int)(i - nw - nu), g = c / H, u = c - g * H;
            const float* bih = b;
            const float* bhh = b + H3;
            b4[c] = g < 2 ? bih[g * H + u] + bhh[g * H + u] : g == 2 ? bhh[2 * H + u] : bih[2 * H + u];
        }
    }
}

hipError_t launch_gru_pack(const Dims& d, const void* W, const void* U, const float* b, void* W4,
                           void* U4, float* b4, hipStream_t s) {
    const long n = (long)d.D * 4 * d.H + (long)d.H * 4 * d.H + 4L * d.H;
    long grid = (n + 255) / 256;
    if (grid > 8192) grid = 8192;
    if (d.bf16)
        hipLaunchKernelGGL(gru_pack_kernel<__bf16>, dim3((unsigned)grid), dim3(256), 0, s,
                           static_cast<const __bf16*>(W), static_cast<const __bf16*>(U), b,
                           static_cast<__bf16*>(W4), static_cast<__bf16*>(U4), b4, d.D, d.H);
    else
        hipLaunchKernelGGL(gru_pack_kernel<float>, dim3((unsigned)grid), dim3(256), 0, s,
                           static_cast<const float*>(W), static_cast<const float*>(U), b,
                           static_cast<float*>(W4), static_cast<float*>(U4), b4, d.D, d.H);
    return hipGetLastError();
}

}  // namespace ldyn
