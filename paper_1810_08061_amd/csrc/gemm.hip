// gemm.hip -- MFMA GEMM with gathered rows and gate-interleaved columns.
//
// Two uses:
//   * the input projection hoisted out of the time loop: x does not depend on
//     the state, so x[b, t] W + b for every valid (b, t) is one GEMM over all
//     time steps, M = sum of lengths (compact rows), N = 4H, K = D;
//   * the per-step comparison path's recurrent product h U + Gx[t] for the
//     rows active at step t, M = active(t), N = 4H, K = H (with bf16 data in
//     fp16 operands, as in the persistent loop: U is widened from bf16 on its
//     way into LDS, h is kept in fp16).
//
// C^T is formed as (W^T)(A^T): MFMA rows are gate-interleaved columns c', MFMA
// columns are data rows, so each lane's four fp32 results are the four gates
// (i, f, g, o) of one (row, unit) and leave as one 16-byte store.
#include "launch.h"

namespace ldyn {

constexpr int G_THREADS = 256;
constexpr int G_CM = 128;  // c' per tile (MFMA M)
constexpr int G_RN = 128;  // rows per tile (MFMA N)

enum GemmMode { MODE_INPROJ = 0, MODE_STEP = 1 };

struct GemmParams {
    const void* A;         // INPROJ: x [B*T][D]; STEP: operand buffer [bpad][hpad]
    const void* Bw;        // W [D][4H] or U [H][4H]
    const float* bias;     // INPROJ: b [4H]
    const float* gx;       // STEP: addend rows gx[offsets[t] + r]
    float* out;            // INPROJ: gx; STEP: z  (row stride 4H)
    const Meta* meta;
    const int32_t* rowsrc;
    const int32_t* offsets;
    int K, lda, H, t;
    int a_vec, b_vec;      // 16-byte vector loads allowed for the A rows / B rows
};

template <typename E>
struct GemmTile {
    using S = typename E::store_t;
    static constexpr int VE = 16 / sizeof(S);      // elements per 16-byte vector
    static constexpr int BK = 64 / sizeof(S);      // K per block: 64 bytes per row
    static constexpr int LDK = BK + VE;            // padded LDS row (80 bytes)
    static constexpr int KS = BK / E::KSTEP;       // MFMA K-steps per block
    static constexpr int UV = (G_CM / 4) / VE;     // vectors per (k, gate) row segment
};

template <typename E, int MODE>
__global__ void __launch_bounds__(G_THREADS)
gemm_kernel(GemmParams p) {
    using S = typename E::store_t;
    using Src = typename E::src_t;  // element type of Bw (the caller's W or U)
    static_assert(sizeof(Src) == sizeof(S), "operand and source elements have one size");
    using F = typename E::frag_t;
    using TL = GemmTile<E>;
    constexpr int VE = TL::VE, BK = TL::BK, LDK = TL::LDK, KS = TL::KS, UV = TL::UV;
    __shared__ __attribute__((aligned(16))) S As[G_RN * LDK];
    __shared__ __attribute__((aligned(16))) S Bs[G_CM * LDK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int H = p.H, N4 = 4 * H, K = p.K;
    int nrows, row_base = 0;
    if (MODE == MODE_INPROJ) {
        nrows = p.meta->total_rows;
    } else {
        row_base = p.offsets[p.t];
        nrows = p.offsets[p.t + 1] - row_base;
    }
    const int ntc = (N4 + G_CM - 1) / G_CM;
    const int ntr = (nrows + G_RN - 1) / G_RN;
    const int ntiles = ntc * ntr;
    const S* __restrict__ A = static_cast<const S*>(p.A);
    const Src* __restrict__ Bw = static_cast<const Src*>(p.Bw);
    const int nkb = (K + BK - 1) / BK;

    for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int tr = tile / ntc, tc = tile - tr * ntc;
        const int r0 = tr * G_RN, c0 = tc * G_CM, ubase = c0 >> 2;

        // Per-thread source rows of the A tile (two 16-byte vectors per thread).
        const S* arow[2];
        bool arow_ok[2];
        int aseg[2], ar[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int v = tid + G_THREADS * j;
            ar[j] = v >> 2;
            aseg[j] = v & 3;
            const int r = r0 + ar[j];
            arow_ok[j] = r < nrows;
            long src = 0;
            if (arow_ok[j]) src = (MODE == MODE_INPROJ) ? (long)p.rowsrc[r] : (long)r;
            arow[j] = A + src * p.lda;
        }
        // B tile vectors: (kk, gate, seg) per thread.
        int bkk[2], bg[2], bseg[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int v = tid + G_THREADS * j;
            bseg[j] = v % UV;
            bg[j] = (v / UV) & 3;
            bkk[j] = v / (UV * 4);
        }

        S areg[2][VE];
        Src breg[2][VE];
        auto load_tiles = [&](int k0) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int k = k0 + aseg[j] * VE;
                if (arow_ok[j] && p.a_vec && k + VE <= K) {
                    const uint4 v = *reinterpret_cast<const uint4*>(arow[j] + k);
                    const S* vs = reinterpret_cast<const S*>(&v);
#pragma unroll
                    for (int e = 0; e < VE; ++e) areg[j][e] = vs[e];
                } else {
#pragma unroll
                    for (int e = 0; e < VE; ++e)
                        areg[j][e] = (arow_ok[j] && k + e < K) ? arow[j][k + e] : E::from_f32(0.0f);
                }
                const int kb = k0 + bkk[j];
                const int u = ubase + bseg[j] * VE;
                const Src* src = Bw + (long)kb * N4 + bg[j] * H + u;
                if (kb < K && p.b_vec && u + VE <= H) {
                    const uint4 v = *reinterpret_cast<const uint4*>(src);
                    const Src* vs = reinterpret_cast<const Src*>(&v);
#pragma unroll
                    for (int e = 0; e < VE; ++e) breg[j][e] = vs[e];
                } else {
#pragma unroll
                    for (int e = 0; e < VE; ++e)
                        breg[j][e] = (kb < K && u + e < H) ? src[e] : (Src)0.0f;
                }
            }
        };
        auto store_tiles = [&]() {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                S* dst = As + ar[j] * LDK + aseg[j] * VE;
#pragma unroll
                for (int e = 0; e < VE; ++e) dst[e] = areg[j][e];
#pragma unroll
                for (int e = 0; e < VE; ++e)
                    Bs[(4 * (bseg[j] * VE + e) + bg[j]) * LDK + bkk[j]] = E::from_src(breg[j][e]);
            }
        };

        f32x4_t acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

        load_tiles(0);
        __syncthreads();  // previous tile's readers are done with LDS
        store_tiles();
        __syncthreads();
        for (int kb = 0; kb < nkb; ++kb) {
            if (kb + 1 < nkb) load_tiles((kb + 1) * BK);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int koff = ks * E::KSTEP + (lane >> 4) * E::KPL;
                F af[4], bf[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    af[i] = E::load(Bs + (wm * 64 + i * 16 + (lane & 15)) * LDK + koff);
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    bf[j] = E::load(As + (wn * 64 + j * 16 + (lane & 15)) * LDK + koff);
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[i][j] = E::mfma(af[i], bf[j], acc[i][j]);
            }
            __syncthreads();
            if (kb + 1 < nkb) {
                store_tiles();
                __syncthreads();
            }
        }

        // Epilogue: lane holds gates 0..3 of unit u for one row.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int cp = c0 + wm * 64 + i * 16 + 4 * (lane >> 4);
            const int u = cp >> 2;
            if (u >= H) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = r0 + wn * 64 + j * 16 + (lane & 15);
                if (r >= nrows) continue;
                f32x4_t v = acc[i][j];
                if (MODE == MODE_INPROJ) {
#pragma unroll
                    for (int g = 0; g < 4; ++g) v[g] += p.bias[g * H + u];
                } else {
                    const f32x4_t a =
                        *reinterpret_cast<const f32x4_t*>(p.gx + (long)(row_base + r) * N4 + cp);
                    v += a;
                }
                *reinterpret_cast<f32x4_t*>(p.out + (long)r * N4 + cp) = v;
            }
        }
    }
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

hipError_t launch_inproj(const Dims& d, const void* x, const void* W, const float* b,
                         const Workspace& ws, int grid, hipStream_t s) {
    GemmParams p{};
    p.A = x;
    p.Bw = W;
    p.bias = b;
    p.out = ws.gx;
    p.meta = ws.meta;
    p.rowsrc = ws.rowsrc;
    p.K = d.D;
    p.lda = d.D;
    p.H = d.H;
    const int ve = d.bf16 ? 8 : 4;
    p.a_vec = (d.D % ve == 0) && aligned16(x);
    p.b_vec = (d.H % ve == 0) && aligned16(W);
    if (d.bf16)
        hipLaunchKernelGGL((gemm_kernel<EltBF16, MODE_INPROJ>), dim3(grid), dim3(G_THREADS), 0, s, p);
    else
        hipLaunchKernelGGL((gemm_kernel<EltF32, MODE_INPROJ>), dim3(grid), dim3(G_THREADS), 0, s, p);
    return hipGetLastError();
}

hipError_t launch_step_gemm(const Dims& d, int t, const void* U, const Workspace& ws, hipStream_t s) {
    GemmParams p{};
    p.A = ws.hx;
    p.Bw = U;
    p.gx = ws.gx;
    p.out = ws.z;
    p.offsets = ws.offsets;
    p.K = d.H;
    p.lda = d.hpad;
    p.H = d.H;
    p.t = t;
    const int ve = d.bf16 ? 8 : 4;
    p.a_vec = (d.hpad % ve == 0);
    p.b_vec = (d.H % ve == 0) && aligned16(U);
    const int grid = ((4 * d.H + G_CM - 1) / G_CM) * ((d.B + G_RN - 1) / G_RN);
    if (d.bf16)
        hipLaunchKernelGGL((gemm_kernel<EltH16, MODE_STEP>), dim3(grid), dim3(G_THREADS), 0, s, p);
    else
        hipLaunchKernelGGL((gemm_kernel<EltF32, MODE_STEP>), dim3(grid), dim3(G_THREADS), 0, s, p);
    return hipGetLastError();
}

}  // namespace ldyn
