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
constexpr int PREP_REG_SLOTS = 256;  // slots whose batch rows each wave keeps in registers

__global__ void __launch_bounds__(PREP_THREADS)
prep_kernel(const int32_t* __restrict__ lengths, int B, int T, Meta* __restrict__ meta,
            int32_t* __restrict__ perm, int32_t* __restrict__ offsets,
            int32_t* __restrict__ rowsrc, unsigned* __restrict__ bar) {
    constexpr int NW = PREP_THREADS / 64;
    extern __shared__ int32_t sh[];
    int32_t* len = sh;       // [B] clamped lengths: batch order, then slot order
    int32_t* sperm = sh + B; // [B] slot -> batch index
    __shared__ int bad, maxlen, wsum[NW];
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    if (tid == 0) {
        bad = 0;
        maxlen = 0;
    }
    if (tid < BAR_WORDS / 64) bar[64 * tid] = 0u;  // grid-barrier counters of the loop kernel
    __syncthreads();
    int mx = 0, bd = 0;
    for (int i = tid; i < B; i += PREP_THREADS) {
        int v = lengths[i];
        if (v < 0 || v > T) {
            bd = 1;
            v = v < 0 ? 0 : T;
        }
        len[i] = v;
        mx = max(mx, v);
    }
    for (int m = 1; m < 64; m <<= 1) {
        mx = max(mx, __shfl_xor(mx, m));
        bd |= __shfl_xor(bd, m);
    }
    if (lane == 0) {
        atomicMax(&maxlen, mx);
        if (bd) atomicOr(&bad, 1);
    }
    __syncthreads();

    // Stable descending rank of row i, its slot: the rows with a longer length
    // and the rows before it with the same length.  With B <= 1024 / P, P lanes
    // of one wave share row i, each counting over every P-th row, and their
    // counts are added across those lanes.
    const int P = B <= PREP_THREADS / 4 ? 4 : (B <= PREP_THREADS / 2 ? 2 : 1);
    const int G = 64 / P;  // rows per wave and pass
    for (int i0 = wave * G; i0 < B; i0 += NW * G) {
        const int i = i0 + lane % G, q = lane / G;
        const int vi = len[min(i, B - 1)];
        int r = 0, j = q;
        for (; j + 7 * P < B; j += 8 * P) {  // eight reads in flight
            int vj[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) vj[u] = len[j + u * P];
#pragma unroll
            for (int u = 0; u < 8; ++u) r += (vj[u] > vi) | ((vj[u] == vi) & (j + u * P < i));
        }
        for (; j < B; j += P) {
            const int vj = len[j];
            r += (vj > vi) | ((vj == vi) & (j < i));
        }
        for (int m = G; m < 64; m <<= 1) r += __shfl_xor(r, m);
        if (q == 0 && i < B) {
            sperm[r] = i;
            perm[r] = i;
        }
    }
    __syncthreads();
    // the lengths in slot order (descending)
    constexpr int LPT = PREP_MAX_B / PREP_THREADS;
    int ls[LPT];
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
        const int s = tid + k * PREP_THREADS;
        ls[k] = s < B ? len[sperm[s]] : 0;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
        const int s = tid + k * PREP_THREADS;
        if (s < B) len[s] = ls[k];
    }
    __syncthreads();
    const int ml = maxlen;

    // offsets[t] = sum over t' < t of active(t'), the rows of all steps before
    // t (= sum_b min(L_b, t)); active(t), the slots whose length exceeds t, by
    // binary search in the sorted lengths.  Each thread takes a run of
    // consecutive t, and the runs' sums are scanned across the workgroup.
    // offsets[T] is the number of valid rows.
    auto active = [&](int t) {
        if (t >= ml) return 0;
        int lo = 0, hi = B;
        while (lo < hi) {
            const int mid = (lo + hi) >> 1;
            if (len[mid] > t) lo = mid + 1;
            else hi = mid;
        }
        return lo;
    };
    const long long per = T / PREP_THREADS + 1;  // >= (T + 1) / PREP_THREADS, rounded up
    const int ta = (int)min(tid * per, (long long)T + 1), tb = (int)min(ta + per, (long long)T + 1);
    int local = 0;
    for (int t = ta; t < tb; ++t) local += active(t);
    int x = local;
    for (int m = 1; m < 64; m <<= 1) {
        const int y = __shfl_up(x, m);
        if (lane >= m) x += y;
    }
    if (lane == 63) wsum[wave] = x;
    __syncthreads();
    int run = x - local;
    for (int v = 0; v < wave; ++v) run += wsum[v];
    for (int t = ta; t < tb; ++t) {
        offsets[t] = run;
        if (t == T) meta->total_rows = run;
        run += active(t);
    }
    __syncthreads();

    // Compact rows of step t are slots [0, active(t)); one wave per step, lanes
    // over slots.  A wave takes steps wave, wave + NW, ...; lane k loads the
    // offset and row count of its k-th next step up front, so the loads of 64
    // steps are in flight together, and the loop reads them from that lane.
    // The batch rows of the first PREP_REG_SLOTS slots stay in registers; a
    // step's stores go through a buffer bounded at its rows, so the lanes past
    // them are dropped without a branch.
    constexpr int NR = PREP_REG_SLOTS / 64;
    int sp[NR];
#pragma unroll
    for (int r = 0; r < NR; ++r) sp[r] = sperm[min(lane + 64 * r, B - 1)];
    for (int t0 = wave; t0 < ml; t0 += NW * 64) {
        const int tk = t0 + NW * lane;
        const int ok = tk < ml ? offsets[tk] : 0;
        const int ak = tk < ml ? offsets[tk + 1] - ok : 0;
        const int n = min(64, (ml - t0 + NW - 1) / NW);
        for (int k = 0; k < n; ++k) {
            const int t = t0 + NW * k;
            const int off = __builtin_amdgcn_readlane(ok, k), act = __builtin_amdgcn_readlane(ak, k);
            const __amdgpu_buffer_rsrc_t R =
                __builtin_amdgcn_make_buffer_rsrc(rowsrc + off, (short)0, act * 4, 0x00020000);
#pragma unroll
            for (int r = 0; r < NR; ++r)
                if (64 * r < act)  // uniform: a scalar branch
                    __builtin_amdgcn_raw_buffer_store_b32((unsigned)(sp[r] * T + t), R, 4 * (lane + 64 * r), 0, 0);
            for (int s0 = PREP_REG_SLOTS; s0 < act; s0 += 64)
                __builtin_amdgcn_raw_buffer_store_b32((unsigned)(sperm[min(s0 + lane, B - 1)] * T + t), R,
                                                      4 * (s0 + lane), 0, 0);
        }
    }
    if (tid == 0) {
        meta->max_len = ml;
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
