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
// with bf16 data on a persistent handle the steps with few rows (the last
// ones, met first) instead run in one cooperative launch (bwd_loop_kernel,
// below).  After the last step the weight gradients are GEMMs over all
// compact rows (K = sum of lengths): dW = X^T dz, dU = H_prev^T dz,
// dx = dz W^T, and db = dz^T 1 a column sum, in gate-interleaved columns,
// permuted back to the caller's gate blocks at the end.  With bf16 data the
// three GEMMs take fp16 operands scaled by powers of two (fp32
// accumulation); with fp32 data they are fp32.
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
        dC[i] = dc_out ? dc_out[ib] : 0.0f;  // no cell state: no upstream gradient
    }
}

// The cell's backward for the rows of step t: one (row, unit) per thread; dz
// over z, dC <- dc_prev, and dH <- dh_direct (the GEMM then adds dz U^T).
template <int CELL>
__global__ void __launch_bounds__(256)
bwd_cell_kernel(float* __restrict__ gx, const float* __restrict__ save_h,
                const float* __restrict__ save_c, const float* __restrict__ dseq,
                const int32_t* __restrict__ perm, float* __restrict__ dH,
                float* __restrict__ dC, int t, int off, int act, int H, int T) {
    const long n = (long)act * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const long r = off + s;
        f32x4_t* zp = reinterpret_cast<f32x4_t*>(gx + r * 4 * H + 4 * u);
        float dh = dH[i];
        if (dseq) dh += dseq[((long)perm[s] * T + t) * H + u];
        float dcp, dhd;
        *zp = cell_backward<CELL>(*zp, save_h[r * H + u], save_c[r * H + u], dh, dC[i], dcp, dhd);
        dC[i] = dcp;
        dH[i] = dhd;
    }
}

// The same with bf16 data, one workgroup per row: the row's dz also goes to
// dz16 in fp16, scaled by a power of two that brings its largest magnitude
// into [2^13, 2^14), for the product dz U^T; dH of a row holds its gradient
// times srow (the scale of the dz it was last formed from; 1 at the start).
// A thread takes up to VU units 256 apart and issues all their loads before
// any store, so the row's reads are in flight together; for H <= 256 VU the
// row's dz and dh stay in registers until the scale is known.
constexpr int BWD_VU = 8;

template <int CELL>
__global__ void __launch_bounds__(256)
bwd_cell16_kernel(float* __restrict__ gx, const float* __restrict__ save_h,
                  const float* __restrict__ save_c, const float* __restrict__ dseq,
                  const int32_t* __restrict__ perm, float* __restrict__ dH,
                  float* __restrict__ dC, float* __restrict__ srow, _Float16* __restrict__ dz16,
                  int t, int off, int H, int T) {
    __shared__ unsigned red[4];
    const int s = blockIdx.x, tid = threadIdx.x;  // one workgroup per row of the step
    const long r = off + s;
    const float inv = 1.0f / srow[s];
    const float* dseq_row = dseq ? dseq + ((long)perm[s] * T + t) * H : nullptr;
    f32x4_t* const zrow = reinterpret_cast<f32x4_t*>(gx + r * 4 * H);
    float* const dh_row = dH + (long)s * H;
    float* const dc_row = dC + (long)s * H;
    unsigned m = 0;
    f32x4_t dz[BWD_VU];
    float dhd[BWD_VU];
    for (int u0 = 0; u0 < H; u0 += 256 * BWD_VU) {
        f32x4_t z[BWD_VU];
        float hp[BWD_VU], cp[BWD_VU], dh[BWD_VU], dc[BWD_VU];
#pragma unroll
        for (int j = 0; j < BWD_VU; ++j) {
            const int u = u0 + tid + 256 * j;
            if (u < H) {
                z[j] = zrow[u];
                hp[j] = save_h[r * H + u];
                cp[j] = save_c[r * H + u];
                dh[j] = dh_row[u] * inv;
                dc[j] = dc_row[u];
                if (dseq_row) dh[j] += dseq_row[u];
            }
        }
#pragma unroll
        for (int j = 0; j < BWD_VU; ++j) {
            const int u = u0 + tid + 256 * j;
            if (u < H) {
                float dcp;
                dz[j] = cell_backward<CELL>(z[j], hp[j], cp[j], dh[j], dc[j], dcp, dhd[j]);
                zrow[u] = dz[j];
                dc_row[u] = dcp;
                dh_row[u] = dhd[j];  // scaled below, once the row's scale is known
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    m = max(m, __float_as_uint(fabsf(dz[j][g])) & 0x7fffffffu);
            }
        }
    }
    for (int o = 32; o > 0; o >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, o));
    if ((tid & 63) == 0) red[tid >> 6] = m;
    __syncthreads();
    m = max(max(red[0], red[1]), max(red[2], red[3]));
    const float mf = __uint_as_float(m);
    float sc = 1.0f;
    if (mf > 0.0f && mf < 3.0e38f) {
        int e;
        (void)frexpf(mf, &e);
        sc = ldexpf(1.0f, min(14 - e, 126));
    }
    typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
    h4_t* const d16 = reinterpret_cast<h4_t*>(dz16 + (long)s * 4 * H);
    if (H <= 256 * BWD_VU) {  // the row is still in registers
#pragma unroll
        for (int j = 0; j < BWD_VU; ++j) {
            const int u = tid + 256 * j;
            if (u < H) {
                d16[u] = h4_t{(_Float16)(dz[j][0] * sc), (_Float16)(dz[j][1] * sc),
                              (_Float16)(dz[j][2] * sc), (_Float16)(dz[j][3] * sc)};
                dh_row[u] = dhd[j] * sc;
            }
        }
    } else {  // each thread reads back what it wrote
        for (int u = tid; u < H; u += 256) {
            const f32x4_t v = zrow[u];
            d16[u] = h4_t{(_Float16)(v[0] * sc), (_Float16)(v[1] * sc), (_Float16)(v[2] * sc),
                          (_Float16)(v[3] * sc)};
            dh_row[u] *= sc;
        }
    }
    if (tid == 0) srow[s] = sc;  // every thread read the old value before the barrier
}

// dh0, dc0: slot order -> batch order (dH divided by its row's scale when
// srow is given).
__global__ void __launch_bounds__(256)
bwd_state_out_kernel(const float* __restrict__ dH, const float* __restrict__ dC,
                     const float* __restrict__ srow, const int32_t* __restrict__ perm, float* dh0,
                     float* dc0, int B, int H) {
    const long n = (long)B * H;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const int s = (int)(i / H), u = (int)(i - (long)s * H);
        const long ib = (long)perm[s] * H + u;
        dh0[ib] = srow ? dH[i] / srow[s] : dH[i];
        if (dc0) dc0[ib] = dC[i];
    }
}

// srow = 1.
__global__ void bwd_ones_kernel(float* a, int n) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < n) a[i] = 1.0f;
}

// The workgroup's largest value of m (256 threads) into *out by one atomic
// maximum: many atomics on one address queue behind each other.
__device__ inline void block_max_to(unsigned m, unsigned* out) {
    __shared__ unsigned red[4];
    for (int o = 32; o > 0; o >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, o));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) atomicMax(out, max(max(red[0], red[1]), max(red[2], red[3])));
}

// x rows in the compact order, fp32, one wave per row (VEC: four elements
// per lane and load, D a multiple of 4 and x aligned to four elements).  With
// amax, the largest |x| of those rows (as bits) goes there too.
template <typename S, bool VEC>
__global__ void __launch_bounds__(256)
bwd_gather_x_kernel(const S* __restrict__ x, const int32_t* __restrict__ rowsrc,
                    const Meta* __restrict__ meta, float* __restrict__ xc, int D, unsigned* amax) {
    const long rows = meta->total_rows;
    const int lane = threadIdx.x & 63;
    unsigned m = 0;
    for (long r = blockIdx.x * 4L + (threadIdx.x >> 6); r < rows; r += gridDim.x * 4L) {
        const S* src = x + (long)rowsrc[r] * D;
        float* dst = xc + r * D;
        if constexpr (VEC) {
            typedef S s4_t __attribute__((ext_vector_type(4)));
#pragma unroll 4
            for (int k = lane; k < D / 4; k += 64) {
                const s4_t v = reinterpret_cast<const s4_t*>(src)[k];
                const f32x4_t f = f32x4_t{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
                reinterpret_cast<f32x4_t*>(dst)[k] = f;
#pragma unroll
                for (int e = 0; e < 4; ++e) m = max(m, __float_as_uint(f[e]) & 0x7fffffffu);
            }
        } else {
#pragma unroll 4
            for (int k = lane; k < D; k += 64) {
                const float f = (float)src[k];
                dst[k] = f;
                m = max(m, __float_as_uint(f) & 0x7fffffffu);
            }
        }
    }
    if (amax) block_max_to(m, amax);
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

// GRU and RNN gradients from the packed four-block layout (gate-interleaved
// columns c' = 4u + g) to the cell's own: block g of column j of the output
// comes from interleaved column 4u + src(g).  part: 0 the input side (W, b_ih
// or b), 1 the recurrent side (U, b_hh).
__device__ inline int unpack_src(int cell, int part, int g) {
    if (cell == CELL_RNN) return 0;
    if (g < 2) return g;               // r, u
    return part == 0 ? 3 : 2;          // n: input part in block 3, recurrent in block 2
}

__global__ void __launch_bounds__(256)
bwd_unpack_kernel(const float* __restrict__ il, float* out, int rows, int H, int cell, int part) {
    const int G = cell == CELL_GRU ? 3 * H : H;
    const long n = (long)rows * G;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
        const long k = i / G;
        const int j = (int)(i - k * G), g = j / H, u = j - g * H;
        out[i] = il[k * 4 * H + 4 * u + unpack_src(cell, part, g)];
    }
}

// dx [B][T][D], one wave per row (b, t): the compact row's dz W^T where b
// runs step t (t below its clamped length), zeros elsewhere; every element is
// written once.  The compact row of (b, t) is offsets[t] + the slot of b in
// the length sort, whose inverse the workgroup first builds in LDS.  VEC: four
// elements per lane and access (D a multiple of 4, dx 16-byte aligned).
template <bool VEC>
__global__ void __launch_bounds__(256)
bwd_dx_kernel(const float* __restrict__ dxc, const int32_t* __restrict__ perm,
              const int32_t* __restrict__ offsets, const int32_t* __restrict__ lengths, float* dx,
              int B, int T, int D) {
    extern __shared__ int32_t slot_of[];  // [B] batch row -> slot
    for (int i = threadIdx.x; i < B; i += 256) slot_of[perm[i]] = i;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const long n = (long)B * T;
    for (long q = blockIdx.x * 4L + (threadIdx.x >> 6); q < n; q += gridDim.x * 4L) {
        const int b = (int)(q / T), t = (int)(q - (long)b * T);
        const bool runs = t < min(max(lengths[b], 0), T);
        const float* src = dxc + (runs ? (long)(offsets[t] + slot_of[b]) * D : 0);
        float* dst = dx + q * D;
        if constexpr (VEC) {
            for (int k = lane; k < D / 4; k += 64)
                reinterpret_cast<f32x4_t*>(dst)[k] =
                    runs ? reinterpret_cast<const f32x4_t*>(src)[k] : f32x4_t{0.f, 0.f, 0.f, 0.f};
        } else {
            for (int k = lane; k < D; k += 64) dst[k] = runs ? src[k] : 0.0f;
        }
    }
}

// ---------------------------------------------------------------------------
// fp16 operands for the GEMMs of the backward with bf16 data: each operand is
// scaled by a power of two that brings its largest magnitude to [2^13, 2^14)
// (exact, and far from fp16 overflow; the host picks it from the largest
// magnitude), and the GEMM's alpha undoes the scales.

// Largest |a| of n floats (as bits): the bits of non-negative floats order as
// integers, so an integer atomic maximum gives the same result in any order.
// a is 16-byte aligned: four elements per load, then the tail.
__global__ void __launch_bounds__(256)
bwd_absmax_kernel(const float* __restrict__ a, long n, unsigned* out) {
    unsigned m = 0;
    const long n4 = n >> 2, stride = (long)gridDim.x * 256;
    long i = blockIdx.x * 256L + threadIdx.x;
    for (; i + 3 * stride < n4; i += 4 * stride) {  // four loads in flight
        f32x4_t v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = reinterpret_cast<const f32x4_t*>(a)[i + j * stride];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) m = max(m, __float_as_uint(v[j][e]) & 0x7fffffffu);
    }
    for (; i < n4; i += stride) {
        const f32x4_t v = reinterpret_cast<const f32x4_t*>(a)[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) m = max(m, __float_as_uint(v[e]) & 0x7fffffffu);
    }
    for (long i = 4 * n4 + blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256)
        m = max(m, __float_as_uint(a[i]) & 0x7fffffffu);
    block_max_to(m, out);
}

// db = dz^T 1 over all compact rows: the rows are cut into BWD_CS_CHUNKS
// ranges, a thread sums one group of four columns over one range in row
// order (partial sums, then bwd_colsum_finish_kernel over the ranges in
// order), and with CONV the same pass writes dz16 = fp16(dz * scale) for
// the weight-gradient GEMMs.
template <bool CONV>
__global__ void __launch_bounds__(256)
bwd_colsum_kernel(const float* __restrict__ dz, long rows, int n4, float* __restrict__ part,
                  _Float16* __restrict__ dz16, float scale) {
    const int cg = blockIdx.x * 256 + threadIdx.x;  // columns 4 cg .. 4 cg + 3
    if (cg >= n4) return;
    const long per = (rows + BWD_CS_CHUNKS - 1) / BWD_CS_CHUNKS;
    const long r0 = (long)blockIdx.y * per, r1 = r0 + per < rows ? r0 + per : rows;
    typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
    f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (long r = r0; r < r1; ++r) {
        const f32x4_t v = *reinterpret_cast<const f32x4_t*>(dz + r * 4 * n4 + 4 * cg);
        acc += v;
        if constexpr (CONV)
            *reinterpret_cast<h4_t*>(dz16 + r * 4 * n4 + 4 * cg) =
                h4_t{(_Float16)(v[0] * scale), (_Float16)(v[1] * scale), (_Float16)(v[2] * scale),
                     (_Float16)(v[3] * scale)};
    }
    *reinterpret_cast<f32x4_t*>(part + (size_t)blockIdx.y * 4 * n4 + 4 * cg) = acc;
}

__global__ void __launch_bounds__(256)
bwd_colsum_finish_kernel(const float* __restrict__ part, int ncols, float* __restrict__ out) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    if (c >= ncols) return;
    float s = 0.0f;
    for (int k = 0; k < BWD_CS_CHUNKS; ++k) s += part[(size_t)k * ncols + c];
    out[c] = s;
}

// dst = fp16(src * scale), n elements (both 16-byte aligned: four elements per
// access, then the tail).
__global__ void __launch_bounds__(256)
bwd_to_f16_kernel(const float* __restrict__ src, _Float16* dst, long n, float scale) {
    typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
    const long n4 = n >> 2;
    for (long i = blockIdx.x * 256L + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
        const f32x4_t v = reinterpret_cast<const f32x4_t*>(src)[i];
        reinterpret_cast<h4_t*>(dst)[i] =
            h4_t{(_Float16)(v[0] * scale), (_Float16)(v[1] * scale), (_Float16)(v[2] * scale),
                 (_Float16)(v[3] * scale)};
    }
    for (long i = 4 * n4 + blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256)
        dst[i] = (_Float16)(src[i] * scale);
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

hipError_t launch_bwd_cell(const Dims& d, int t, int off, int act, const float* save_h,
                           const float* save_c, const float* dseq, float* dH, float* dC,
                           const Workspace& ws, hipStream_t s) {
    if (act < 1) return hipSuccess;
    auto k = d.cell == CELL_GRU ? bwd_cell_kernel<CELL_GRU>
             : d.cell == CELL_RNN ? bwd_cell_kernel<CELL_RNN> : bwd_cell_kernel<CELL_LSTM>;
    hipLaunchKernelGGL(k, dim3(grid_of((long)act * d.H)), dim3(256), 0, s, ws.gx, save_h, save_c,
                       dseq, ws.perm, dH, dC, t, off, act, d.H, d.T);
    return hipGetLastError();
}

hipError_t launch_bwd_unpack(const Dims& d, const float* il, float* out, int rows, int part,
                             hipStream_t s) {
    const long n = (long)rows * (d.cell == CELL_GRU ? 3 : 1) * d.H;
    hipLaunchKernelGGL(bwd_unpack_kernel, dim3(grid_of(n)), dim3(256), 0, s, il, out, rows, d.H,
                       d.cell, part);
    return hipGetLastError();
}

hipError_t launch_bwd_state_out(const Dims& d, const float* dH, const float* dC, const float* srow,
                                float* dh0, float* dc0, const Workspace& ws, hipStream_t s) {
    hipLaunchKernelGGL(bwd_state_out_kernel, dim3(grid_of((long)d.B * d.H)), dim3(256), 0, s, dH,
                       dC, srow, ws.perm, dh0, dc0, d.B, d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_cell16(const Dims& d, int t, int off, int act, const float* save_h,
                             const float* save_c, const float* dseq, float* dH, float* dC,
                             float* srow, _Float16* dz16, const Workspace& ws, hipStream_t s) {
    auto k = d.cell == CELL_GRU ? bwd_cell16_kernel<CELL_GRU>
             : d.cell == CELL_RNN ? bwd_cell16_kernel<CELL_RNN> : bwd_cell16_kernel<CELL_LSTM>;
    if (act < 1) return hipSuccess;
    hipLaunchKernelGGL(k, dim3(act), dim3(256), 0, s, ws.gx, save_h, save_c, dseq, ws.perm, dH,
                       dC, srow, dz16, t, off, d.H, d.T);
    return hipGetLastError();
}

hipError_t launch_bwd_ones(float* a, int n, hipStream_t s) {
    hipLaunchKernelGGL(bwd_ones_kernel, dim3((n + 255) / 256), dim3(256), 0, s, a, n);
    return hipGetLastError();
}

hipError_t launch_bwd_gather_x(const Dims& d, const void* x, long rows, float* xc, unsigned* amax,
                               const Workspace& ws, hipStream_t s) {
    const long g4 = (rows + 3) / 4;
    const unsigned g = (unsigned)(g4 < 1 ? 1 : g4 > 1024 ? 1024 : g4);
    const uintptr_t xa = reinterpret_cast<uintptr_t>(x);
    if (d.bf16) {
        const __bf16* xs = static_cast<const __bf16*>(x);
        if (d.D % 4 == 0 && (xa & 7) == 0)
            hipLaunchKernelGGL((bwd_gather_x_kernel<__bf16, true>), dim3(g), dim3(256), 0, s, xs, ws.rowsrc,
                               ws.meta, xc, d.D, amax);
        else
            hipLaunchKernelGGL((bwd_gather_x_kernel<__bf16, false>), dim3(g), dim3(256), 0, s, xs, ws.rowsrc,
                               ws.meta, xc, d.D, amax);
    } else {
        const float* xs = static_cast<const float*>(x);
        if (d.D % 4 == 0 && (xa & 15) == 0)
            hipLaunchKernelGGL((bwd_gather_x_kernel<float, true>), dim3(g), dim3(256), 0, s, xs, ws.rowsrc,
                               ws.meta, xc, d.D, amax);
        else
            hipLaunchKernelGGL((bwd_gather_x_kernel<float, false>), dim3(g), dim3(256), 0, s, xs, ws.rowsrc,
                               ws.meta, xc, d.D, amax);
    }
    return hipGetLastError();
}

hipError_t launch_bwd_absmax(const float* a, long n, unsigned* out, hipStream_t s) {
    const unsigned g = grid_of(n / 4) < 1024 ? grid_of(n / 4) : 1024;
    hipLaunchKernelGGL(bwd_absmax_kernel, dim3(g), dim3(256), 0, s, a, n, out);
    return hipGetLastError();
}

hipError_t launch_bwd_colsum(const float* dz, long rows, int ncols, float* part, float* out,
                             _Float16* dz16, float scale, hipStream_t s) {
    const int n4 = ncols / 4;
    const dim3 grid((unsigned)((n4 + 255) / 256), BWD_CS_CHUNKS);
    if (dz16)
        hipLaunchKernelGGL(bwd_colsum_kernel<true>, grid, dim3(256), 0, s, dz, rows, n4, part, dz16, scale);
    else
        hipLaunchKernelGGL(bwd_colsum_kernel<false>, grid, dim3(256), 0, s, dz, rows, n4, part, dz16,
                           scale);
    hipLaunchKernelGGL(bwd_colsum_finish_kernel, dim3((unsigned)((ncols + 255) / 256)), dim3(256), 0, s,
                       part, ncols, out);
    return hipGetLastError();
}

hipError_t launch_bwd_to_f16(const float* src, _Float16* dst, long n, float scale, hipStream_t s) {
    hipLaunchKernelGGL(bwd_to_f16_kernel, dim3(grid_of(n)), dim3(256), 0, s, src, dst, n, scale);
    return hipGetLastError();
}

hipError_t launch_bwd_permute(const Dims& d, const float* il, float* out, int rows, hipStream_t s) {
    hipLaunchKernelGGL(bwd_permute_kernel, dim3(grid_of((long)rows * 4 * d.H)), dim3(256), 0, s, il,
                       out, rows, d.H);
    return hipGetLastError();
}

hipError_t launch_bwd_dx(const Dims& d, const float* dxc, long rows, const int32_t* lengths,
                         float* dx, const Workspace& ws, hipStream_t s) {
    (void)rows;
    const long g4 = ((long)d.B * d.T + 3) / 4;
    const unsigned g = (unsigned)(g4 < 1 ? 1 : g4 > 4096 ? 4096 : g4);
    const size_t lds = (size_t)d.B * sizeof(int32_t);
    if (d.D % 4 == 0 && (reinterpret_cast<uintptr_t>(dx) & 15) == 0)
        hipLaunchKernelGGL(bwd_dx_kernel<true>, dim3(g), dim3(256), lds, s, dxc, ws.perm, ws.offsets, lengths,
                           dx, d.B, d.T, d.D);
    else
        hipLaunchKernelGGL(bwd_dx_kernel<false>, dim3(g), dim3(256), lds, s, dxc, ws.perm, ws.offsets, lengths,
                           dx, d.B, d.T, d.D);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// The reverse loop in one cooperative launch (bf16 data, persistent handles).
//
// Workgroup g owns the 8 units [8 g, 8 g + 8) and keeps in LDS the rows of U
// of those units (gate-interleaved columns, fp16, times su) as MFMA
// A-fragments of 32 columns each: 8 x 4H values, 128 KB at H = 2048, which
// leaves the registers free for a whole row tile of the exchanged dz.  Step t
// (from the last down to t_end, then once more for dh entering t_end - 1):
//   * product: dh of the rows that ran step t+1 and of the owned units,
//     sum_j dz_{t+1}[s][j] U[u][j] over all 4H columns, from the step's dz
//     that every workgroup published (fp16; each row's 32 columns from one
//     workgroup scaled by that workgroup's power of two, undone after the
//     MFMA of those columns); the waves split the columns and their
//     partial sums meet in LDS;
//   * cell: the owned (row, unit) pairs of the rows that run step t take dh
//     (plus the carried term and the output sequence's gradient), their z
//     and saved state, give dz (kept in fp32 for the weight gradients and
//     published in fp16 under the block's scale), dc and the carried term;
//   * a grid barrier; the published dz alternates between two buffers.
// The carried dh and dc live in dH, dC ([B][H], slot order): in, the upstream
// gradients of the final state; out, the complete dh entering step t_end - 1
// (dh0 when t_end is 0) and the carried dc at that point.
struct BwdLoopParams {
    const _Float16* u16;     // [H][4H] U, gate-interleaved columns, times su
    float* gx;               // [rows][4H] z in, dz (fp32) out
    const float* save_h;     // [rows][H] the state each step started from
    const float* save_c;
    const float* dseq;       // [B][T][H] gradient of the output sequence, or null
    const int32_t* perm;     // [B] slot -> batch row
    const int32_t* offsets;  // [T + 1] first compact row of each step
    Meta* meta;              // max_len in, timeout status out
    float* dH;               // [B][H] carried dh: in d_out_h, out dh0 (slot order)
    float* dC;               // [B][H] carried dc: in d_out_c, out dc0
    _Float16* dzx;           // [2][bpad][kp] published dz (fp16, scaled per row and block)
    float* dzs;              // [2][bpad][nblk] the scales (powers of two)
    unsigned* bar;           // [9 * 64] barrier counters, zero at the launch
    unsigned long long timeout_ticks;
    float alpha_u;           // 1 / su
    int B, H, T, bpad, groups, kp, nblk;
    int t_end;               // steps max_len - 1 down to t_end; then dh of step t_end - 1
};

constexpr int BL_WAVES = 8;
constexpr int BL_NTC = 4;  // row tiles per chunk
constexpr int BL_SC1 = 16;  // buffer-instruction cache policy: device scope

typedef unsigned bl_u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned bl_u32x4 __attribute__((ext_vector_type(4)));

template <int KSW, int CELL>
__global__ void __launch_bounds__(BL_WAVES * 64, 1)
bwd_loop_kernel(BwdLoopParams p) {
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int lds_ok;
    const int tid = threadIdx.x, l = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = blockIdx.x;
    const int H = p.H, H4 = 4 * H, KP = p.kp, NB = p.nblk, bpad = p.bpad;
    constexpr int KSA = BL_WAVES * KSW;  // K-steps of 32 columns over the padded 4H
    // LDS: U fragments [KSA][32 lanes][8 halves], then the partial sums
    // [BL_WAVES][BL_NTC][32 lanes][4]
    _Float16* const ufr = reinterpret_cast<_Float16*>(lds);
    float* const part = lds + KSA * 32 * 8 / 2;
    const __amdgpu_buffer_rsrc_t Ru = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<_Float16*>(p.u16), (short)0, (int)((size_t)H * H4 * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t Rz = __builtin_amdgcn_make_buffer_rsrc(
        p.dzx, (short)0, (int)((size_t)2 * bpad * KP * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t Rs = __builtin_amdgcn_make_buffer_rsrc(
        p.dzs, (short)0, (int)((size_t)2 * bpad * NB * 4), 0x00020000);
    constexpr unsigned OOB = 0x80000000u;  // past every buffer: loads give zero

    // Fragment slot q (0..31) of K-step kg: unit 8 g + q % 8, columns
    // 32 kg + 8 (q / 8) .. + 7; lane l of an A-fragment takes slot
    // (l / 16) * 8 + l % 16 when l % 16 < 8 (units 8..15 of the 16-row tile
    // are zero).
    for (int e = tid; e < KSA * 32; e += BL_WAVES * 64) {
        const int kg = e >> 5, q = e & 31;
        const int u = 8 * g + (q & 7), col = 32 * kg + 8 * (q >> 3);
        const bool in = u < H && col < H4;
        const bl_u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(
            Ru, in ? (unsigned)((u * H4 + col) * 2) : OOB, 0, 0);
        *reinterpret_cast<bl_u32x4*>(ufr + (size_t)e * 8) = v;
    }
    __syncthreads();
    const bool alane = (l & 15) < 8;
    const int aslot = (l >> 4) * 8 + (l & 15);

    const int max_len = p.meta->max_len;
    auto act_of = [&](int t) { return p.offsets[t + 1] - p.offsets[t]; };
    const int t_end = p.t_end;
    int k = 0;
    for (int t = max_len - 1; t >= t_end - 1; --t, ++k) {
        const bool last = t < t_end;  // only the product: dh entering step t_end - 1
        const int actp = t + 1 < max_len ? act_of(t + 1) : 0;  // rows with dz_{t+1}
        const int actc = last ? 0 : act_of(t);                // rows that run step t
        const int rows = last ? actp : actc;
        const int nt = (rows + 15) >> 4;
        const unsigned pin = (unsigned)((t + 1) & 1), pout = (unsigned)((t + 2) & 1);
        // The cell's inputs for this thread's pair of the first chunk depend
        // on no other workgroup: loaded now, they travel during the product.
        const int ul = tid & 7, u = 8 * g + ul;
        const bool uin = u < H;
        const int s_pre = tid >> 3;
        const bool pre = !last && uin && s_pre < min(rows, BL_NTC * 16);
        f32x4_t z_pre = f32x4_t{0.f, 0.f, 0.f, 0.f};
        float hp_pre = 0.f, cp_pre = 0.f, dh_pre = 0.f, dc_pre = 0.f, ds_pre = 0.f;
        if (pre) {
            const size_t r = (size_t)p.offsets[t] + s_pre, su = (size_t)s_pre * H + u;
            z_pre = *reinterpret_cast<const f32x4_t*>(p.gx + r * H4 + 4 * u);
            hp_pre = p.save_h[r * H + u];
            cp_pre = p.save_c[r * H + u];
            dh_pre = p.dH[su];
            dc_pre = p.dC[su];
            if (p.dseq) ds_pre = p.dseq[((size_t)p.perm[s_pre] * p.T + t) * H + u];
        }
        for (int ntc0 = 0; ntc0 < nt; ntc0 += BL_NTC) {
            const int nchunk = min(BL_NTC, nt - ntc0);
            // ---- product: this wave's KSW K-steps of each row tile, the
            // tile's dz fragments and scales all loaded before its MFMAs
            for (int j = 0; j < nchunk; ++j) {
                const int s = (ntc0 + j) * 16 + (l & 15);
                const bool live = s < actp;
                const unsigned row = pin * (unsigned)bpad + (unsigned)s;
                f16x8_t b[KSW];
#pragma unroll
                for (int ks = 0; ks < KSW; ++ks) {
                    const int col = 32 * (w * KSW + ks) + 8 * (l >> 4);
                    b[ks] = __builtin_bit_cast(f16x8_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                            Rz, live ? (row * KP + col) * 2u : OOB, 0, BL_SC1));
                }
                float inv[KSW];
                if constexpr (KSW % 4 == 0) {
#pragma unroll
                    for (int k4 = 0; k4 < KSW; k4 += 4) {
                        const bl_u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(
                            Rs, live ? (row * NB + w * KSW + k4) * 4u : OOB, 0, BL_SC1);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float sc = __uint_as_float(v[e]);
                            inv[k4 + e] = sc > 0.0f ? 1.0f / sc : 0.0f;
                        }
                    }
                } else {
#pragma unroll
                    for (int ks = 0; ks < KSW; ++ks) {
                        const float sc = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                            Rs, live ? (row * NB + w * KSW + ks) * 4u : OOB, 0, BL_SC1));
                        inv[ks] = sc > 0.0f ? 1.0f / sc : 0.0f;
                    }
                }
                f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSW; ++ks) {
                    const int kg = w * KSW + ks;
                    f16x8_t a = f16x8_t{};
                    if (alane) a = *reinterpret_cast<const f16x8_t*>(ufr + ((size_t)kg * 32 + aslot) * 8);
                    const f32x4_t tmp = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                        a, b[ks], f32x4_t{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                    acc += tmp * inv[ks];
                }
                // lanes 0..31 hold the 8 real units (rows 4 (l / 16) + i of the tile)
                if (l < 32) *reinterpret_cast<f32x4_t*>(part + ((w * BL_NTC + j) * 32 + l) * 4) = acc;
            }
            __syncthreads();
            // ---- cell: the owned pairs of the chunk's rows; 8 lanes per row
            {
                const int rend = min((ntc0 + nchunk) * 16, rows);
                for (int s = ntc0 * 16 + (tid >> 3); s < rend; s += BL_WAVES * 8) {
                    const bool have = pre && ntc0 == 0;  // s is s_pre: one pass per chunk
                    float dh = 0.0f;
                    if (s < actp) {
                        const int j = (s >> 4) - ntc0, ln = 16 * (ul >> 2) + (s & 15), i = ul & 3;
                        float sum = 0.0f;
#pragma unroll
                        for (int ww = 0; ww < BL_WAVES; ++ww) sum += part[((ww * BL_NTC + j) * 32 + ln) * 4 + i];
                        dh = sum * p.alpha_u;
                    }
                    const size_t su = (size_t)s * H + u;
                    if (uin) dh += have ? dh_pre : p.dH[su];
                    if (last) {  // dh entering step t_end - 1 (dh0 when t_end is 0)
                        if (uin) p.dH[su] = dh;
                        continue;
                    }
                    f32x4_t dz = f32x4_t{0.f, 0.f, 0.f, 0.f};
                    if (uin) {
                        const size_t r = (size_t)p.offsets[t] + s;
                        f32x4_t* zp = reinterpret_cast<f32x4_t*>(p.gx + r * H4 + 4 * u);
                        float dcp, dhd;
                        if (have) {
                            dh += ds_pre;
                            dz = cell_backward<CELL>(z_pre, hp_pre, cp_pre, dh, dc_pre, dcp, dhd);
                        } else {
                            if (p.dseq) dh += p.dseq[((size_t)p.perm[s] * p.T + t) * H + u];
                            dz = cell_backward<CELL>(*zp, p.save_h[r * H + u], p.save_c[r * H + u], dh,
                                                     p.dC[su], dcp, dhd);
                        }
                        *zp = dz;
                        p.dC[su] = dcp;
                        p.dH[su] = dhd;
                    }
                    // the block's scale: its largest magnitude into [2^13, 2^14)
                    unsigned m = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) m = max(m, __float_as_uint(fabsf(dz[e])) & 0x7fffffffu);
                    for (int o = 4; o > 0; o >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, o));
                    const float mf = __uint_as_float(m);
                    float sc = 1.0f;
                    if (mf > 0.0f && mf < 3.0e38f) {
                        int e;
                        (void)frexpf(mf, &e);
                        sc = ldexpf(1.0f, min(14 - e, 126));
                    }
                    typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
                    const h4_t hv = h4_t{(_Float16)(dz[0] * sc), (_Float16)(dz[1] * sc),
                                         (_Float16)(dz[2] * sc), (_Float16)(dz[3] * sc)};
                    const unsigned row = pout * (unsigned)bpad + (unsigned)s;
                    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(bl_u32x2, hv), Rz,
                                                          (row * KP + 32 * g + 4 * ul) * 2u, 0, BL_SC1);
                    if (ul == 0)
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(sc), Rs, (row * NB + g) * 4u, 0,
                                                              BL_SC1);
                }
            }
            __syncthreads();  // the partial sums are read before the next chunk writes them
        }
        if (!last && !grid_barrier_bounded(p.bar, p.groups, k, p.timeout_ticks, p.meta, &lds_ok)) return;
    }
}

// K-steps per wave: 32 columns each over 4H, a power of two, 32 at the most
// (H = 2048); H even so 8-column groups do not straddle rows of U.
int bwd_loop_ksw(int H) {
    if (H < 16 || H > 2048 || (H & 1)) return 0;
    const int ks = (H + 7) / 8;
    int ksw = 1;
    while (ksw * BL_WAVES < ks) ksw *= 2;
    return ksw;
}

static int bwd_loop_lds_bytes(int ksw) {
    return BL_WAVES * ksw * 32 * 16 + BL_WAVES * BL_NTC * 32 * 16;
}

typedef void (*bwd_loop_fn)(BwdLoopParams);

static bwd_loop_fn bwd_loop_pick(int ksw, int cell) {
#define BL_CELLS(K)                                                                         \
    if (ksw == K)                                                                           \
        return cell == CELL_GRU ? bwd_loop_kernel<K, CELL_GRU>                              \
               : cell == CELL_RNN ? bwd_loop_kernel<K, CELL_RNN> : bwd_loop_kernel<K, CELL_LSTM>;
    BL_CELLS(1) BL_CELLS(2) BL_CELLS(4) BL_CELLS(8) BL_CELLS(16) BL_CELLS(32)
#undef BL_CELLS
    return nullptr;
}

// Sizes of the exchange: columns per published row and scale blocks per row
// (one block of 32 columns per workgroup).
void bwd_loop_shape(int H, int* kp, int* nblk) {
    const int ksw = bwd_loop_ksw(H);
    *kp = 32 * BL_WAVES * ksw;
    *nblk = *kp / 32;
}

// Workgroups (one per CU, all resident) the loop can run with, or 0.
int bwd_loop_fits(const Dims& d, int num_cus) {
    const int ksw = bwd_loop_ksw(d.H);
    if (!ksw || !d.bf16 || d.bpad > 512) return 0;
    const int groups = (d.H + 7) / 8;
    if (groups > num_cus) return 0;
    bwd_loop_fn f = bwd_loop_pick(ksw, d.cell);
    if (!f) return 0;
    const int lds = bwd_loop_lds_bytes(ksw);
    int n = 0;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(f),
                                                     BL_WAVES * 64, lds) != hipSuccess) {
        (void)hipGetLastError();  // not an error of a later call: the per-step path serves
        return 0;
    }
    return n >= 1 ? groups : 0;
}

hipError_t launch_bwd_loop(const Dims& d, const _Float16* u16, float alpha_u, const float* save_h,
                           const float* save_c, const float* dseq, float* dH, float* dC,
                           _Float16* dzx, float* dzs, unsigned* bar, unsigned long long timeout_ticks,
                           int t_end, const Workspace& ws, hipStream_t s) {
    const int ksw = bwd_loop_ksw(d.H);
    bwd_loop_fn f = bwd_loop_pick(ksw, d.cell);
    if (!f) return hipErrorInvalidValue;
    int kp, nblk;
    bwd_loop_shape(d.H, &kp, &nblk);
    BwdLoopParams p{};
    p.u16 = u16;
    p.gx = ws.gx;
    p.save_h = save_h;
    p.save_c = save_c;
    p.dseq = dseq;
    p.perm = ws.perm;
    p.offsets = ws.offsets;
    p.meta = ws.meta;
    p.dH = dH;
    p.dC = dC;
    p.dzx = dzx;
    p.dzs = dzs;
    p.bar = bar;
    p.timeout_ticks = timeout_ticks;
    p.alpha_u = alpha_u;
    p.B = d.B;
    p.H = d.H;
    p.T = d.T;
    p.bpad = d.bpad;
    p.groups = (d.H + 7) / 8;
    p.kp = kp;
    p.nblk = nblk;
    p.t_end = t_end;
    void* args[] = {&p};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(f), dim3(p.groups),
                                      dim3(BL_WAVES * 64), args, (unsigned)bwd_loop_lds_bytes(ksw), s);
}

}  // namespace ldyn
