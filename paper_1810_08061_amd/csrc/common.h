// common.h -- types, workspace layout and device helpers shared by the
// kernels of the variable-length LSTM loop (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ldyn {

// ---------------------------------------------------------------------------
// Workspace written on the device by the preparation kernel.
struct Meta {
    int32_t max_len;     // loop bound: largest (clamped) length
    int32_t total_rows;  // sum of (clamped) lengths = rows of the compact input projection
    int32_t status;      // bit 0: a length was clamped; bit 1: a barrier wait timed out
    int32_t iters;       // loop iterations in which some row ran (= max_len unless rows end early)
};
constexpr int32_t STATUS_BAD_LENGTHS = 1;
constexpr int32_t STATUS_TIMEOUT = 2;

// Gate-interleaved column order used by the input projection Gx and by the
// recurrent tiles: column c' = 4u + g holds gate g in (i, f, g, o) of hidden
// unit u, which is column g*H + u of W, U and b.  A lane that owns c' = 4u..4u+3
// of one row then holds all four gates of (row, u).
__host__ __device__ inline int gate_col(int cprime, int H) { return (cprime & 3) * H + (cprime >> 2); }

// ---------------------------------------------------------------------------
// Element types.  MFMA 16x16xK fragments: lane l holds operand row/column
// (l & 15) and the K slice [(l >> 4) * KPL, (l >> 4) * KPL + KPL); the 16x16
// fp32 result gives lane l rows 4*(l >> 4) + j (j = 0..3) of column (l & 15).
// src_t is the element type of the caller's U (and of x, W); store_t the
// type of the MFMA operands the kernels keep (U fragments, the h operand).
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

struct EltF32 {
    using store_t = float;
    using src_t = float;
    using frag_t = float;
    static constexpr int KSTEP = 4;  // K per MFMA
    static constexpr int KPL = 1;    // K values per lane
    __device__ static inline f32x4_t mfma(frag_t a, frag_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static inline frag_t zero() { return 0.0f; }
    __device__ static inline store_t from_f32(float v) { return v; }
    __device__ static inline float to_f32(store_t v) { return v; }
    __device__ static inline store_t from_src(src_t v) { return v; }
    // Load KPL consecutive elements at p (aligned to KPL elements).
    __device__ static inline frag_t load(const store_t* p) { return *p; }
};

struct EltBF16 {
    using store_t = __bf16;
    using src_t = __bf16;
    using frag_t = bf16x8_t;
    static constexpr int KSTEP = 32;
    static constexpr int KPL = 8;
    __device__ static inline f32x4_t mfma(frag_t a, frag_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static inline frag_t zero() {
        frag_t z;
#pragma unroll
        for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
        return z;
    }
    __device__ static inline store_t from_f32(float v) { return (__bf16)v; }
    __device__ static inline float to_f32(store_t v) { return (float)v; }
    __device__ static inline store_t from_src(src_t v) { return v; }
    __device__ static inline frag_t load(const store_t* p) {
        return *reinterpret_cast<const frag_t*>(p);
    }
};

// bf16 data with fp16 recurrent operands: U is widened from bf16 to fp16
// (exact for 2^-14 <= |U| <= 65504, the fp16 normal range; smaller entries
// land on the fp16 subnormal grid, an absolute error <= 2^-25) and h is
// rounded to fp16 for the product h U.  h lies in (-1, 1) after the first
// step of every cell here, where fp16 keeps 11 significant bits against
// bf16's 8 at the same MFMA rate.
struct EltH16 {
    using store_t = _Float16;
    using src_t = __bf16;
    using frag_t = f16x8_t;
    static constexpr int KSTEP = 32;
    static constexpr int KPL = 8;
    __device__ static inline f32x4_t mfma(frag_t a, frag_t b, f32x4_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    __device__ static inline frag_t zero() {
        frag_t z;
#pragma unroll
        for (int i = 0; i < 8; ++i) z[i] = (_Float16)0.0f;
        return z;
    }
    __device__ static inline store_t from_f32(float v) { return (_Float16)v; }
    __device__ static inline float to_f32(store_t v) { return (float)v; }
    __device__ static inline store_t from_src(src_t v) { return (_Float16)(float)v; }
    __device__ static inline frag_t load(const store_t* p) {
        return *reinterpret_cast<const frag_t*>(p);
    }
};

// ---------------------------------------------------------------------------
// Gate non-linearities in fp32 from the hardware exp2 and reciprocal.
// sigmoid(0) and tanh(0) come out exactly 1/2 and 0.
__device__ inline float rcp_f(float x) { return __builtin_amdgcn_rcpf(x); }
__device__ inline float sigmoid_f(float z) { return rcp_f(1.0f + __expf(-z)); }
__device__ inline float tanh_f(float z) {
    // tanh|z| = (1 - e) / (1 + e) with e = exp(-2|z|) in (0, 1]: no overflow.
    const float e = __expf(-2.0f * fabsf(z));
    return copysignf((1.0f - e) * rcp_f(1.0f + e), z);
}

// The GRU cell (gate blocks r, u, n) in the four columns of a unit: the loop's
// weights are packed so that the pre-activations hold
//   z[0] = r, z[1] = u (input and recurrent parts and both biases),
//   z[2] = h U_n + b_hn (the recurrent part of n), z[3] = x W_n + b_in;
// then n = tanh(z[3] + r z[2]) and h' = (1 - u) n + u h.  No cell state.
__device__ inline void gru_cell(f32x4_t z, float& h) {
    const float rg = sigmoid_f(z[0]);
    const float ug = sigmoid_f(z[1]);
    const float ng = tanh_f(z[3] + rg * z[2]);
    h = (1.0f - ug) * ng + ug * h;
}

// The tanh RNN cell in the four columns of a unit: the weights are packed so
// that z[0] = x W + h U + b and the other three columns are zero.
__device__ inline void rnn_cell(f32x4_t z, float& h) { h = tanh_f(z[0]); }

// One LSTM cell update from the four pre-activations of a (row, unit).
__device__ inline void lstm_cell(f32x4_t z, float& c, float& h) {
    const float ig = sigmoid_f(z[0]);
    const float fg = sigmoid_f(z[1]);
    const float gg = tanh_f(z[2]);
    const float og = sigmoid_f(z[3]);
    c = fg * c + ig * gg;
    h = og * tanh_f(c);
}

// Cells of the loop (the kinds the C ABI's cell argument names).
enum CellKind { CELL_LSTM = 0, CELL_GRU = 1, CELL_RNN = 2 };

// The update of `cell` from the four pre-activations of a (row, unit); c is
// the LSTM's cell state and left unchanged by the other cells.
__device__ inline void apply_cell(int cell, f32x4_t z, float& c, float& h) {
    if (cell == CELL_GRU) gru_cell(z, h);
    else if (cell == CELL_RNN) rnn_cell(z, h);
    else lstm_cell(z, c, h);
}


// The backward of one cell step for one (row, unit), from its pre-activations
// z (the four gate blocks of the packed layout), the state the step started
// from (hp, cp) and the gradients of the state after it (dh, dc).  Returns dz
// and sets the gradient reaching the previous state other than through
// dz U^T: dc_prev (LSTM) and dh_direct (GRU: h' depends on h through u).
template <int CELL>
__device__ inline f32x4_t cell_backward(f32x4_t z, float hp, float cp, float dh, float dc,
                                        float& dc_prev, float& dh_direct) {
    f32x4_t dz;
    dc_prev = 0.0f;
    dh_direct = 0.0f;
    if constexpr (CELL == CELL_LSTM) {
        const float ig = sigmoid_f(z[0]), fg = sigmoid_f(z[1]);
        const float gg = tanh_f(z[2]), og = sigmoid_f(z[3]);
        const float c = fg * cp + ig * gg;
        const float tc = tanh_f(c);
        const float d_o = dh * tc;
        const float dct = dc + dh * og * (1.0f - tc * tc);
        dz[0] = dct * gg * ig * (1.0f - ig);
        dz[1] = dct * cp * fg * (1.0f - fg);
        dz[2] = dct * ig * (1.0f - gg * gg);
        dz[3] = d_o * og * (1.0f - og);
        dc_prev = dct * fg;
    } else if constexpr (CELL == CELL_GRU) {
        // z = (r, u, recurrent part of n, input part of n)
        const float rg = sigmoid_f(z[0]), ug = sigmoid_f(z[1]);
        const float ng = tanh_f(z[3] + rg * z[2]);
        const float dzn = dh * (1.0f - ug) * (1.0f - ng * ng);
        dz[0] = dzn * z[2] * rg * (1.0f - rg);
        dz[1] = dh * (hp - ng) * ug * (1.0f - ug);
        dz[2] = dzn * rg;
        dz[3] = dzn;
        dh_direct = dh * ug;
    } else {
        const float hn = tanh_f(z[0]);
        dz[0] = dh * (1.0f - hn * hn);
        dz[1] = 0.0f;
        dz[2] = 0.0f;
        dz[3] = 0.0f;
    }
    return dz;
}

// ---------------------------------------------------------------------------
// Grid barrier k (k = 0, 1, ... in order) of a cooperative launch of `groups`
// workgroups: each workgroup drains its stores, then counts itself in the
// counter of its group (blockIdx mod 8, at bar[64 (1 + x)]); the last of a
// group counts the group in bar[0], which every workgroup polls.  The
// counters must be zero at the launch.  Bounded: past the deadline the
// timeout status is set and false is returned.
__device__ inline bool grid_barrier_bounded(unsigned* bar, int groups, int k,
                                            unsigned long long timeout_ticks, Meta* meta,
                                            int* lds_ok) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (threadIdx.x == 0) {
        int ok = 1;
        if (groups > 1) {
            const int x = blockIdx.x & 7;
            const unsigned members = (unsigned)((groups - x + 7) >> 3);
            const unsigned old = __hip_atomic_fetch_add(bar + 64 * (1 + x), 1u, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
            if (old + 1u == (unsigned)(k + 1) * members)
                __hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            const unsigned want = (unsigned)(k + 1) * (unsigned)(groups < 8 ? groups : 8);
            const unsigned long long t0 = wall_clock64();
            while (__hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < want) {
                if (wall_clock64() - t0 > timeout_ticks) {
                    ok = 0;
                    __hip_atomic_fetch_or(&meta->status, STATUS_TIMEOUT, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        *lds_ok = ok;
    }
    __syncthreads();
    return *lds_ok != 0;
}

// Timing stress (a diagnostic build, LDYN_STRESS defined): a wave sleeps for a
// pseudo-random time (0 to about 1 us, from a hash of the workgroup, wave,
// step and site) before it publishes data for other workgroups, marks a
// buffer or starts polling, so the exchanges between workgroups (h in the
// forward loop, dz in the reverse loop) are exercised under orders of
// arrival that the plain build rarely produces.  The plain build compiles it
// away.
__device__ inline void stress_delay(int t, int site) {
#ifdef LDYN_STRESS
    unsigned x = (unsigned)blockIdx.x * 0x9e3779b1u ^ (unsigned)(threadIdx.x >> 6) * 0x85ebca77u ^
                 (unsigned)t * 0xc2b2ae3du ^ (unsigned)site * 0x27d4eb2fu;
    x ^= x >> 15;
    x *= 0x2c1b3c6du;
    x ^= x >> 12;
    const int n = __builtin_amdgcn_readfirstlane((int)(x & 31));
    for (int i = 0; i < n; ++i) __builtin_amdgcn_s_sleep(1);
#else
    (void)t;
    (void)site;
#endif
}

}  // namespace ldyn
