// seq.hip -- the output sequence of the loop.
//
// The loop of the paper (Section 9 "RNN cells", Appendix A) appends the
// cell's output at every step.  out_seq[b][t] is the hidden state of row b
// after step t for t < L[b]; past a sequence's length (or past the step at
// which a row ended, with termination from the state) the output is zero (no
// value is defined there; zero is the padding convention chosen).
//
// Every loop writes the valid outputs itself; this kernel writes the zeros
// past each row's last step.
#include "launch.h"

namespace ldyn {

struct SeqParams {
    float* seq;              // [B][T][H]
    const int32_t* lengths;  // [B] last step + 1 of each row: its length as passed, or the
                             // step it ended at (clamped here to [0, T])
    int B, T, H;
};

// One wave per output row; float4 stores when H is a multiple of 4 and
// out_seq is 16-byte aligned.
template <bool VEC>
__global__ void __launch_bounds__(256)
seq_finish_kernel(SeqParams p) {
    const int lane = threadIdx.x & 63;
    const long wave = ((long)blockIdx.x * 256 + threadIdx.x) >> 6;
    const long nwaves = (long)gridDim.x * 4;
    const int H = p.H, T = p.T;
    const long nrows = (long)p.B * T;
    for (long row = wave; row < nrows; row += nwaves) {
        const int b = (int)(row / T), t = (int)(row - (long)b * T);
        const int L = min(max(p.lengths[b], 0), T);
        if (t < L) continue;
        float* dst = p.seq + (size_t)row * H;
        if constexpr (VEC) {
            for (int u = 4 * lane; u < H; u += 256) *reinterpret_cast<f32x4_t*>(dst + u) = f32x4_t{0.f, 0.f, 0.f, 0.f};
        } else {
            for (int u = lane; u < H; u += 64) dst[u] = 0.0f;
        }
    }
}

// Output sequence of the forward for training: the state after step t of a
// row is the state step t + 1 started from (kept per compact row), or its
// final state after its last step.  Zeros past each length.
__global__ void __launch_bounds__(256)
seq_from_saved_kernel(float* seq, const float* __restrict__ save_h, const float* __restrict__ out_h,
                      const int32_t* __restrict__ perm, const int32_t* __restrict__ offsets,
                      const int32_t* __restrict__ lengths, int B, int T, int H) {
    // one slot s per workgroup row; slot order is the length order
    const long n = (long)B * T * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const long bt = i / H;
        const int u = (int)(i - bt * H);
        const int s = (int)(bt / T), t = (int)(bt - (long)s * T);
        const int b = perm[s];
        const int L = min(max(lengths[b], 0), T);
        float v = 0.0f;
        if (t + 1 < L) v = save_h[(long)(offsets[t + 1] + s) * H + u];
        else if (t + 1 == L) v = out_h[(long)b * H + u];
        seq[((long)b * T + t) * H + u] = v;
    }
}

hipError_t launch_seq_from_saved(const Dims& d, float* seq, const float* save_h, const float* out_h,
                                 const int32_t* lengths, const Workspace& ws, int num_cus,
                                 hipStream_t s) {
    const long n = (long)d.B * d.T * d.H;
    long grid = (n + 255) / 256;
    if (grid > 16L * num_cus) grid = 16L * num_cus;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(seq_from_saved_kernel, dim3((unsigned)grid), dim3(256), 0, s, seq, save_h,
                       out_h, ws.perm, ws.offsets, lengths, d.B, d.T, d.H);
    return hipGetLastError();
}

hipError_t launch_seq_finish(const Dims& d, float* seq, const int32_t* lengths, int num_cus,
                             hipStream_t s) {
    SeqParams p{seq, lengths, d.B, d.T, d.H};
    const long rows = (long)d.B * d.T;
    long grid = (rows + 3) / 4;
    if (grid > 8L * num_cus) grid = 8L * num_cus;
    if (grid < 1) grid = 1;
    const bool vec = d.H % 4 == 0 && (reinterpret_cast<uintptr_t>(seq) & 15) == 0;
    if (vec)
        hipLaunchKernelGGL(seq_finish_kernel<true>, dim3((unsigned)grid), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(seq_finish_kernel<false>, dim3((unsigned)grid), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace ldyn
