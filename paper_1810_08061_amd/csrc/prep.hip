// prep.hip -- loop bound, length sort and compact row tables, on the device.
//
// The paper's loop bound is the maximum sequence length (Section 9 "RNN
// cells"; Appendix A); here it is reduced on the device so no host round trip
// is needed.  Sorting the slots by length (descending) makes the rows still
// running at step t a prefix [0, active(t)) of the slot order, so every later
// kernel touches only live rows.
#include "launch.h"

namespace ldyn {

constexpr int PREP_THREADS = 1024;
constexpr int PREP_MAX_B = 8192;  // two int32 tables of B entries in LDS

__global__ void __launch_bounds__(PREP_THREADS)
prep_kernel(const int32_t* __restrict__ lengths, int B, int T, Meta* __restrict__ meta,
            int32_t* __restrict__ perm, int32_t* __restrict__ offsets,
            int32_t* __restrict__ rowsrc, unsigned* __restrict__ bar) {
    extern __shared__ int32_t sh[];
    int32_t* len = sh;       // [B] clamped lengths, batch order
    int32_t* sperm = sh + B; // [B] slot -> batch index
    __shared__ int bad, maxlen;
    const int tid = threadIdx.x;
    if (tid == 0) {
        bad = 0;
        maxlen = 0;
    }
    if (tid < BAR_WORDS / 64) bar[64 * tid] = 0u;  // grid-barrier counters of the loop kernel
    __syncthreads();
    for (int i = tid; i < B; i += PREP_THREADS) {
        int v = lengths[i];
        if (v < 0 || v > T) {
            atomicOr(&bad, 1);
            v = v < 0 ? 0 : T;
        }
        len[i] = v;
        atomicMax(&maxlen, v);
    }
    __syncthreads();
    // Stable descending rank: slot of row i.
    for (int i = tid; i < B; i += PREP_THREADS) {
        const int vi = len[i];
        int r = 0;
        for (int j = 0; j < B; ++j) {
            const int vj = len[j];
            r += (vj > vi) | ((vj == vi) & (j < i));
        }
        sperm[r] = i;
        perm[r] = i;
    }
    // offsets[t] = sum_b min(L_b, t): rows of all steps before t.
    for (int t = tid; t <= T; t += PREP_THREADS) {
        int s = 0;
        for (int j = 0; j < B; ++j) s += min(len[j], t);
        offsets[t] = s;
    }
    __syncthreads();
    const int ml = maxlen;
    // Compact rows of step t are slots [0, active(t)); one wave per step, lanes over slots.
    const int wave = tid >> 6, lane = tid & 63;
    for (int t = wave; t < ml; t += PREP_THREADS / 64) {
        const int off = offsets[t];
        const int act = offsets[t + 1] - off;
        for (int s = lane; s < act; s += 64) rowsrc[off + s] = sperm[s] * T + t;
    }
    if (tid == 0) {
        int total = 0;
        for (int j = 0; j < B; ++j) total += len[j];
        meta->max_len = ml;
        meta->total_rows = total;
        meta->status = bad ? STATUS_BAD_LENGTHS : 0;
        meta->iters = ml;
    }
}

hipError_t launch_prep(const Dims& d, const int32_t* lengths, const Workspace& ws, hipStream_t s) {
    if (d.B > PREP_MAX_B) return hipErrorInvalidValue;
    const size_t lds = (size_t)2 * d.B * sizeof(int32_t);
    hipLaunchKernelGGL(prep_kernel, dim3(1), dim3(PREP_THREADS), lds, s, lengths, d.B, d.T, ws.meta,
                       ws.perm, ws.offsets, ws.rowsrc, ws.bar);
    return hipGetLastError();
}

}  // namespace ldyn
