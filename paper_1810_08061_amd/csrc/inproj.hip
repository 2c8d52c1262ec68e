// inproj.hip -- the input projection over all valid time steps, bf16 inputs.
//
// x does not depend on the recurrent state, so x[b, t] W + b for every valid
// (b, t) -- one row per sequence step, sum of lengths rows in all -- is one GEMM
// hoisted out of the time loop: Gx[r][c'] = x[rowsrc[r]] . Wt[c'] + b[col(c')],
// with c' the gate-interleaved column (4u + gate).
//
// W arrives as [D][4H] (N contiguous).  MFMA wants both operands contiguous
// along K, so a first kernel writes Wt[c'][k] (gate-interleaved rows, zero
// padded to whole tiles); the GEMM then loads both operands with 16-byte
// vector loads.  C^T = Wt x^T is formed so each lane's four results are the
// four gates of one (row, unit).
//
// Two GEMMs: inproj_dma_kernel (below; D a multiple of 8), whose operands
// reach LDS by DMA, and the fallback inproj_bf16_kernel for any D: tiles of
// 256 columns x 256 rows x 64 K, four waves of 128 x 128 each (8 x 8 MFMA
// 16x16x32 tiles), two LDS stages, the next K-block loaded into registers
// while the current one is multiplied, each result leaving as one 16-byte
// store.  Gx is stored non-temporally: the loop reads each row back only at
// its step, long after the GEMM, so its lines need not pass through the
// caches (measured with a 1.62 GB Gx: the GEMM 0.941 to 0.912 ms and the
// loop 4.77 to 4.755 ms; the workloads with 48 and 98 MB of Gx were not
// slower).
#include "launch.h"

namespace ldyn {

constexpr int IP_TILE = 256;            // rows and columns per tile
constexpr int IP_BK = 64;               // K per block
constexpr int IP_LDK = IP_BK + 8;       // padded LDS row: 144 bytes
constexpr int IP_THREADS = 256;
constexpr int IP_STAGE = 2 * IP_TILE * IP_LDK;  // bf16 elements per stage (A and B)
constexpr int IP_LDS_BYTES = 2 * IP_STAGE * 2;

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// Wt[c'][k] = W[k][col(c')] for c' < 4H, k < D; zero elsewhere (np x dp).
// A tile is 64 k by 64 c'; its 64 c' are 16 units times the four gates, so in
// a row of W they are four runs of 16 consecutive columns.  Each thread reads
// two 16-byte pieces of those runs (element by element when H is not a
// multiple of 8, W is not 16-byte aligned or the tile passes the edge of W),
// the tile turns through LDS, and each thread writes two 16-byte pieces of
// rows of Wt (dp is a multiple of 64).
__global__ void __launch_bounds__(256)
transpose_w_kernel(const __bf16* __restrict__ W, __bf16* __restrict__ Wt, int D, int H, int np, int dp) {
    constexpr int LDT = 64 + 8;  // bf16 per LDS row: 144 bytes, rows 16-byte aligned
    __shared__ __attribute__((aligned(16))) __bf16 tile[64][LDT];  // [c' in tile][k in tile]
    const int k0 = blockIdx.x * 64, c0 = blockIdx.y * 64, u0 = c0 / 4;
    const size_t H4 = 4 * (size_t)H;
    // a tile inside W, H a multiple of 8 and W 16-byte aligned: both pieces
    // by 16-byte loads, in flight together; otherwise element by element
    const bool vec = (H % 8) == 0 && (reinterpret_cast<uintptr_t>(W) & 15) == 0 && k0 + 64 <= D &&
                     u0 + 16 <= H;
    bf16x8_t v[2];
    if (vec) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int i = threadIdx.x + 256 * j;
            const int kl = i >> 3, g = (i >> 1) & 3, ub = u0 + 8 * (i & 1);  // row, gate, first unit
            v[j] = *reinterpret_cast<const bf16x8_t*>(W + (size_t)(k0 + kl) * H4 + (size_t)g * H + ub);
        }
    } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int i = threadIdx.x + 256 * j;
            const int kl = i >> 3, g = (i >> 1) & 3, ub = u0 + 8 * (i & 1);
            const int k = k0 + kl;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                v[j][e] = (k < D && ub + e < H) ? W[(size_t)k * H4 + (size_t)g * H + ub + e] : (__bf16)0.0f;
        }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int i = threadIdx.x + 256 * j;
        const int kl = i >> 3, g = (i >> 1) & 3, ub = u0 + 8 * (i & 1);
#pragma unroll
        for (int e = 0; e < 8; ++e) tile[4 * (ub - u0 + e) + g][kl] = v[j][e];
    }
    __syncthreads();
#pragma unroll
    for (int i = threadIdx.x; i < 512; i += 256) {
        const int cl = i >> 3, kp = 8 * (i & 7);
        const int cp = c0 + cl;
        if (cp < np && k0 + kp < dp)
            *reinterpret_cast<bf16x8_t*>(Wt + (size_t)cp * dp + k0 + kp) =
                *reinterpret_cast<const bf16x8_t*>(&tile[cl][kp]);
    }
}

struct InprojParams {
    const __bf16* x;       // [B*T][D]
    const __bf16* wt;      // [np][dp]
    const float* bias;     // [4H]
    float* gx;             // [rows][4H]
    const Meta* meta;
    const int32_t* rowsrc;
    int D, H, dp;
};

template <bool KFULL>
__global__ void __launch_bounds__(IP_THREADS, 1)
inproj_bf16_kernel(InprojParams p) {
    extern __shared__ __attribute__((aligned(16))) __bf16 smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;      // wave's 128 columns, 128 rows
    const int H = p.H, N4 = 4 * H, D = p.D;
    const int nrows = p.meta->total_rows;
    const int ntc = (N4 + IP_TILE - 1) / IP_TILE;
    const int ntr = (nrows + IP_TILE - 1) / IP_TILE;
    const int ntiles = ntc * ntr;
    const int nkb = (D + IP_BK - 1) / IP_BK;
    const int ldr = tid >> 3, chunk = tid & 7;     // this thread loads chunk of rows ldr + 32 i

    for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int tr = tile / ntc, tc = tile - tr * ntc;
        const int r0 = tr * IP_TILE, c0 = tc * IP_TILE;

        const __bf16* xrow[8];   // row starts of x
        const __bf16* wrow[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = min(r0 + ldr + 32 * i, nrows - 1);
            xrow[i] = p.x + (size_t)p.rowsrc[r] * D;
            wrow[i] = p.wt + (size_t)(c0 + ldr + 32 * i) * p.dp + chunk * 8;
        }
        u32x4_t ra[8], rb[8];
        auto gload = [&](int kb) {
            const int k = kb * IP_BK;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int kk = k + chunk * 8;  // first element of this thread's chunk
                if (KFULL) {
                    ra[i] = *reinterpret_cast<const u32x4_t*>(xrow[i] + kk);
                } else {
                    // ragged D: elementwise with addresses clamped into the row, zeros past D
                    __bf16 e[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const __bf16 v = xrow[i][min(kk + j, D - 1)];
                        e[j] = kk + j < D ? v : (__bf16)0.0f;
                    }
                    ra[i] = __builtin_bit_cast(u32x4_t, e);
                }
                rb[i] = *reinterpret_cast<const u32x4_t*>(wrow[i] + k);
            }
        };
        auto lstore = [&](int stage) {
            __bf16* sa = smem + stage * IP_STAGE;
            __bf16* sb = sa + IP_TILE * IP_LDK;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                *reinterpret_cast<u32x4_t*>(sa + (ldr + 32 * i) * IP_LDK + chunk * 8) = ra[i];
                *reinterpret_cast<u32x4_t*>(sb + (ldr + 32 * i) * IP_LDK + chunk * 8) = rb[i];
            }
        };

        f32x4_t acc[8][8];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

        gload(0);
        __syncthreads();  // the previous tile's readers are done with both stages
        lstore(0);
        __syncthreads();
        for (int kb = 0; kb < nkb; ++kb) {
            if (kb + 1 < nkb) gload(kb + 1);
            const __bf16* sa = smem + (kb & 1) * IP_STAGE;
            const __bf16* sb = sa + IP_TILE * IP_LDK;
#pragma unroll
            for (int ks = 0; ks < IP_BK / 32; ++ks) {
                const int koff = ks * 32 + (lane >> 4) * 8;
                bf16x8_t af[8], bf[8];
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    af[i] = *reinterpret_cast<const bf16x8_t*>(sb + (wm * 128 + i * 16 + (lane & 15)) * IP_LDK + koff);
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    bf[j] = *reinterpret_cast<const bf16x8_t*>(sa + (wn * 128 + j * 16 + (lane & 15)) * IP_LDK + koff);
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
            }
            if (kb + 1 < nkb) lstore((kb + 1) & 1);
            __syncthreads();
        }

        // epilogue: lane holds gates 0..3 of unit u for one row
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int cp = c0 + wm * 128 + i * 16 + 4 * (lane >> 4);
            const int u = cp >> 2;
            if (u >= H) continue;
            const f32x4_t bv = f32x4_t{p.bias[u], p.bias[H + u], p.bias[2 * H + u], p.bias[3 * H + u]};
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int r = r0 + wn * 128 + j * 16 + (lane & 15);
                if (r < nrows) __builtin_nontemporal_store(acc[i][j] + bv, reinterpret_cast<f32x4_t*>(p.gx + (size_t)r * N4 + cp));
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Variant fed by LDS DMA: both operand tiles go from memory straight into a
// two-stage LDS ring (buffer load with an LDS destination), K = 64 per stage:
// while one stage is multiplied the next is in flight, and no registers hold
// data in transit.  A DMA instruction writes 64 lanes x 16 bytes
// contiguously; with 128-byte operand rows that is 8 whole rows, and each
// lane fetches the 16-byte chunk that belongs at its position under the XOR
// swizzle chunk' = chunk ^ (row & 7), which spreads the MFMA fragment reads
// (16 rows, one chunk) over all banks.  x rows past D (the K tail) are
// fetched at an offset outside the buffer, which yields zeros.  Requires D a
// multiple of 8, x 16-byte aligned and under 2 GiB.
//
// Eight waves (two per SIMD) each own 128 columns x 64 rows of the 256 x 256
// tile, so one wave's LDS reads overlap the other's MFMAs; a wave reads both
// K-steps' fragments of a stage before its first MFMA.
constexpr int GD_TILE = 256;
constexpr int GD_BK = 64;
constexpr int GD_HALF = GD_TILE * GD_BK * 2;  // bytes of one operand tile per stage
constexpr int GD_STAGE = 2 * GD_HALF;
constexpr int GD_WAVES = 8;
constexpr int GD_OUT_LD = GD_TILE + 4;         // padded row of the output staging (floats)
constexpr int GD_LDS_BYTES =
    128 * GD_OUT_LD * 4 > 2 * GD_STAGE ? 128 * GD_OUT_LD * 4 : 2 * GD_STAGE;
static_assert(GD_BK == IP_BK, "the padded K of Wt is a whole number of stages");

struct InprojDmaParams {
    InprojParams b;
    unsigned x_bytes, wt_bytes;
};

// One LDS-DMA instruction: 16 bytes per lane from byte offset off of R into
// dst + 16 * lane.  (A plain function: the address-space cast is device-only.)
__device__ inline void dma16(__amdgpu_buffer_rsrc_t R, unsigned char* dst, unsigned off) {
    typedef __attribute__((address_space(3))) void* lds_ptr_t;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(R, (lds_ptr_t)dst, 16, off, 0, 0, 0);
}

// Workgroup barrier after this wave's LDS accesses have completed.  The
// kernel's waits for its LDS DMA are explicit; __syncthreads() would in
// addition wait for every outstanding vector memory operation -- the DMA of
// the stage in flight, and the stores of Gx -- and so drain the operand
// pipeline at every K-block.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__global__ void __launch_bounds__(GD_WAVES * 64, 1)
inproj_dma_kernel(InprojDmaParams q) {
    constexpr int RW = GD_TILE * 2 / GD_WAVES;  // rows per wave
    constexpr int JT = RW / 16;                 // row tiles per wave
    constexpr int QQ = 32 / GD_WAVES;           // DMA instructions per operand, stage and wave
    extern __shared__ __attribute__((aligned(16))) unsigned char gsm[];
    const InprojParams& p = q.b;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / (GD_WAVES / 2), wn = wave % (GD_WAVES / 2);  // wave's 128 columns, RW rows
    const int H = p.H, N4 = 4 * H, D = p.D;
    const int nrows = p.meta->total_rows;
    const int ntc = (N4 + GD_TILE - 1) / GD_TILE;
    const int ntiles = ntc * ((nrows + GD_TILE - 1) / GD_TILE);
    const int nkb = p.dp / GD_BK;
    const __amdgpu_buffer_rsrc_t Rx =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<__bf16*>(p.x), (short)0, (int)q.x_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t Rw =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<__bf16*>(p.wt), (short)0, (int)q.wt_bytes, 0x00020000);
    // Consecutive workgroups sit on different XCDs: give each XCD a run of
    // 32 consecutive tile numbers, and number the tiles so that such a run
    // is a block of 4 row tiles x 8 column tiles: each x block is then shared
    // by 8 workgroups of one L2 and each Wt block by 4.
    const int g = (gridDim.x & 7) == 0 ? (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3) : blockIdx.x;
    const int ntr = (nrows + GD_TILE - 1) / GD_TILE;
    const bool blocked = (ntc & 7) == 0;
    const int nnum = blocked ? (ntr + 3) / 4 * 4 * ntc : ntiles;

    for (int tile = g; tile < nnum; tile += gridDim.x) {
        int tr, tc;
        if (blocked) {
            const int sb = tile / (4 * ntc), t = tile - sb * 4 * ntc;
            tr = sb * 4 + ((t & 31) >> 3);
            tc = (t >> 5) * 8 + (t & 7);
            if (tr >= ntr) continue;
        } else {
            tr = tile / ntc;
            tc = tile - tr * ntc;
        }
        const int r0 = tr * GD_TILE, c0 = tc * GD_TILE;
        // this lane's DMA sources: rows 8 * (QQ * wave + qq) + (lane >> 3) of both tiles
        unsigned xoff[QQ], woff[QQ];
        int kchunk[QQ];
#pragma unroll
        for (int qq = 0; qq < QQ; ++qq) {
            const int r = 8 * (QQ * wave + qq) + (lane >> 3);
            const int c = (lane & 7) ^ (r & 7);
            const int row = min(r0 + r, nrows - 1);
            kchunk[qq] = 8 * c;
            xoff[qq] = ((unsigned)p.rowsrc[row] * (unsigned)D + 8u * c) * 2u;
            woff[qq] = ((unsigned)(c0 + r) * (unsigned)p.dp + 8u * c) * 2u;
        }
        auto issue = [&](int kb) {
            unsigned char* st = gsm + (kb & 1) * GD_STAGE;
#pragma unroll
            for (int qq = 0; qq < QQ; ++qq) {
                const bool in = kb * GD_BK + kchunk[qq] < D;
                dma16(Rx, st + (QQ * wave + qq) * 1024, in ? xoff[qq] + kb * GD_BK * 2u : 0x80000000u);
                dma16(Rw, st + GD_HALF + (QQ * wave + qq) * 1024, woff[qq] + kb * GD_BK * 2u);
            }
        };

        f32x4_t acc[8][JT];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < JT; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

        lds_barrier();  // every wave is done with the previous tile's stages
        issue(0);
        for (int kb = 0; kb < nkb; ++kb) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's DMAs of stage kb have landed
            lds_barrier();  // ... and every other wave's; all are done reading stage kb - 1
            if (kb + 1 < nkb) issue(kb + 1);
            const unsigned char* st = gsm + (kb & 1) * GD_STAGE;
            // both K-steps' fragments are read before any MFMA, so the second
            // step's reads are in flight while the first step multiplies
            bf16x8_t af[2][8], bfr[2][JT];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const int c = ks * 4 + (lane >> 4);
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int r = wm * 128 + i * 16 + (lane & 15);
                    af[ks][i] = *reinterpret_cast<const bf16x8_t*>(st + GD_HALF + r * 128 + 16 * (c ^ (r & 7)));
                }
#pragma unroll
                for (int j = 0; j < JT; ++j) {
                    const int r = wn * RW + j * 16 + (lane & 15);
                    bfr[ks][j] = *reinterpret_cast<const bf16x8_t*>(st + r * 128 + 16 * (c ^ (r & 7)));
                }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < JT; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[ks][i], bfr[ks][j], acc[i][j], 0, 0, 0);
        }

        // Epilogue through LDS, in two halves of 128 rows: the two waves of a
        // half park their quadrants as [row][column] (rows padded by 16 bytes),
        // then every wave writes whole 1 KB rows, lane l holding the four gates
        // of unit (c0 + 4 l) / 4.
        float* const out = reinterpret_cast<float*>(gsm);
        const int cl = 4 * lane, cp = c0 + cl;
        const bool col_ok = cp < N4;
        const int ub = col_ok ? cp >> 2 : 0;
        const f32x4_t bv = f32x4_t{p.bias[ub], p.bias[H + ub], p.bias[2 * H + ub], p.bias[3 * H + ub]};
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            lds_barrier();  // stages (or the previous half) no longer read
            if (wn * RW / 128 == half) {
                const int rl = wn * RW - half * 128;  // first row of this wave within the half
#pragma unroll
                for (int i = 0; i < 8; ++i)
#pragma unroll
                    for (int j = 0; j < JT; ++j)
                        *reinterpret_cast<f32x4_t*>(out + (rl + j * 16 + (lane & 15)) * GD_OUT_LD + wm * 128 + i * 16 +
                                                    4 * (lane >> 4)) = acc[i][j];
            }
            lds_barrier();
            for (int rr = wave; rr < 128; rr += GD_WAVES) {
                const int r = r0 + half * 128 + rr;
                if (r >= nrows) break;
                const f32x4_t v = *reinterpret_cast<const f32x4_t*>(out + rr * GD_OUT_LD + cl);
                if (col_ok) __builtin_nontemporal_store(v + bv, reinterpret_cast<f32x4_t*>(p.gx + (size_t)r * N4 + cp));
            }
        }
    }
}

int inproj_bf16_tiles_max(const Dims& d) {
    return (int)(((long long)d.B * d.T + IP_TILE - 1) / IP_TILE) * ((4 * d.H + IP_TILE - 1) / IP_TILE);
}

void inproj_bf16_wt_shape(const Dims& d, int* np, int* dp) {
    *np = (4 * d.H + IP_TILE - 1) / IP_TILE * IP_TILE;
    *dp = (d.D + IP_BK - 1) / IP_BK * IP_BK;
}

hipError_t inproj_bf16_setup() {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(inproj_bf16_kernel<true>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, IP_LDS_BYTES);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(inproj_dma_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, GD_LDS_BYTES);
    if (e != hipSuccess) return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(inproj_bf16_kernel<false>),
                               hipFuncAttributeMaxDynamicSharedMemorySize, IP_LDS_BYTES);
}

hipError_t launch_transpose_w(const Dims& d, const void* W, const Workspace& ws, hipStream_t s) {
    int np, dp;
    inproj_bf16_wt_shape(d, &np, &dp);
    hipLaunchKernelGGL(transpose_w_kernel, dim3(dp / 64, np / 64), dim3(256), 0, s,
                       static_cast<const __bf16*>(W), static_cast<__bf16*>(ws.wt), d.D, d.H, np, dp);
    return hipGetLastError();
}

hipError_t launch_inproj_bf16(const Dims& d, const void* x, const float* b, const Workspace& ws,
                              int grid, hipStream_t s) {
    int np, dp;
    inproj_bf16_wt_shape(d, &np, &dp);
    InprojParams p{static_cast<const __bf16*>(x), static_cast<const __bf16*>(ws.wt), b, ws.gx,
                   ws.meta, ws.rowsrc, d.D, d.H, dp};
    const bool aligned = (reinterpret_cast<uintptr_t>(x) & 15) == 0;
    const long long x_bytes = 2LL * d.B * d.T * d.D, wt_bytes = 2LL * np * dp;
    if (aligned && d.D % 8 == 0 && x_bytes < (1LL << 31) && wt_bytes < (1LL << 31)) {
        InprojDmaParams q{p, (unsigned)x_bytes, (unsigned)wt_bytes};
        hipLaunchKernelGGL(inproj_dma_kernel, dim3(grid), dim3(GD_WAVES * 64), GD_LDS_BYTES, s, q);
        return hipGetLastError();
    }
    const bool kfull = (d.D % IP_BK) == 0 && aligned;
    if (kfull)
        hipLaunchKernelGGL(inproj_bf16_kernel<true>, dim3(grid), dim3(IP_THREADS), IP_LDS_BYTES, s, p);
    else
        hipLaunchKernelGGL(inproj_bf16_kernel<false>, dim3(grid), dim3(IP_THREADS), IP_LDS_BYTES, s, p);
    return hipGetLastError();
}

}  // namespace ldyn
