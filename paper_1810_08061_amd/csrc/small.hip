// small.hip -- the whole forward in one workgroup, one launch (H <= 32).
//
// When the 4H gate columns fit the 8 gate tiles of one workgroup, nothing
// needs a grid: the loop bound is reduced in LDS, each step forms
// z = x_t W + h U + b with MFMA (W and U slices held in registers, each wave
// owning two gate tiles over the full K = D + H, so no cross-wave reduction),
// applies the gates to the rows with t < L[b] (the per-row select of the
// paper's loop, Section 9 "RNN cells"), and passes h to the next step through
// LDS.  x for step t+1 is fetched while step t computes.  Rows stay in batch
// order; finished rows are simply not updated.  With bf16 data, x W takes bf16
// operands and h U fp16 operands (U widened from bf16), as in the persistent
// loop.
#include "launch.h"

namespace ldyn {

constexpr int SM_WAVES = 4;
constexpr int SM_THREADS = 64 * SM_WAVES;
constexpr int SM_MT = 2;  // gate tiles per wave: 4 waves x 2 x 16 columns = 4H <= 128

struct SmallParams {
    const void* x;
    const int32_t* lengths;
    const void* W;
    const void* U;
    const float* b;
    const float* h0;
    const float* c0;
    float* out_h;
    float* out_c;
    float* seq;  // [B][T][H] output sequence (valid steps only), or null
    Meta* meta;
    int B, D, H, T;
    int cell;  // CellKind (only the LSTM has a cell state)
    // termination from the state (stop_v null: none): a row ends after a step
    // that leaves v . h + c > 0; steps[b] receives the steps it ran
    const float* stop_v;
    float stop_c;
    int32_t* steps;
};

// E: element type of x and W; EH: of the recurrent operands (U, h).
template <typename E, typename EH, int KD, int KH, int NT>
__global__ void __launch_bounds__(SM_THREADS, 1)
small_kernel(SmallParams p) {
    using S = typename E::store_t;
    using F = typename E::frag_t;
    using SH = typename EH::store_t;
    using FH = typename EH::frag_t;
    static_assert(E::KSTEP == EH::KSTEP && E::KPL == EH::KPL, "one fragment shape");
    constexpr int HP = KH * EH::KSTEP;      // padded hidden width of the LDS h rows
    constexpr int HS = HP + 16 / sizeof(SH);  // row stride (16-byte pad)
    __shared__ __attribute__((aligned(16))) SH hs[2][NT * 16 * HS];
    __shared__ int len[NT * 16];
    __shared__ int maxlen, bad;
    __shared__ int ended[NT * 16];  // termination from the state: 1 once the row ended
    __shared__ int ran[2];          // some row ran at step t (slot t & 1)

    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const int B = p.B, D = p.D, H = p.H, T = p.T, H4 = 4 * H;
    const S* X = static_cast<const S*>(p.x);
    const S* W = static_cast<const S*>(p.W);
    const typename EH::src_t* U = static_cast<const typename EH::src_t*>(p.U);

    if (tid == 0) {
        maxlen = 0;
        bad = 0;
        ran[0] = 0;
        ran[1] = 0;
    }
    __syncthreads();
    for (int i = tid; i < NT * 16; i += SM_THREADS) {
        int v = 0;
        if (i < B) {
            v = p.lengths[i];
            if (v < 0 || v > T) {
                atomicOr(&bad, 1);
                v = v < 0 ? 0 : T;
            }
            atomicMax(&maxlen, v);
        }
        len[i] = v;
        ended[i] = 0;
        if (p.stop_v && i < B) p.steps[i] = v;  // a row that never ends runs to its cap
    }
    // h0 -> LDS (operand type); padding rows and columns are zero in both buffers
    for (int i = tid; i < NT * 16 * HS; i += SM_THREADS) {
        const int n = i / HS, k = i - n * HS;
        hs[0][i] = EH::from_f32((n < B && k < H) ? p.h0[(size_t)n * H + k] : 0.0f);
        hs[1][i] = EH::from_f32(0.0f);
    }

    // A-fragments of W^T and U^T for this wave's two gate tiles (clamped loads).
    F wf[SM_MT][KD];
    FH uf[SM_MT][KH];
    float bias[SM_MT][4];
#pragma unroll
    for (int mt = 0; mt < SM_MT; ++mt) {
        const int cp = (w * SM_MT + mt) * 16 + (l & 15);
        const bool uok = (cp >> 2) < H;
        const int col = uok ? gate_col(cp, H) : 0;
#pragma unroll
        for (int ks = 0; ks < KD; ++ks) {
            F f = E::zero();
#pragma unroll
            for (int e = 0; e < E::KPL; ++e) {
                const int k = ks * E::KSTEP + (l >> 4) * E::KPL + e;
                const S v = W[(size_t)min(k, D - 1) * H4 + col];
                if constexpr (E::KPL == 1) f = (uok && k < D) ? v : 0.0f;
                else f[e] = (uok && k < D) ? v : E::from_f32(0.0f);
            }
            wf[mt][ks] = f;
        }
#pragma unroll
        for (int ks = 0; ks < KH; ++ks) {
            FH f = EH::zero();
#pragma unroll
            for (int e = 0; e < EH::KPL; ++e) {
                const int k = ks * EH::KSTEP + (l >> 4) * EH::KPL + e;
                const SH v = EH::from_src(U[(size_t)min(k, H - 1) * H4 + col]);
                if constexpr (EH::KPL == 1) f = (uok && k < H) ? v : 0.0f;
                else f[e] = (uok && k < H) ? v : EH::from_f32(0.0f);
            }
            uf[mt][ks] = f;
        }
        // this lane's four gates belong to unit (cp0 >> 2) with cp0 = tile base + 4 * (l >> 4)
        const int u = ((w * SM_MT + mt) * 16 + 4 * (l >> 4)) >> 2;
#pragma unroll
        for (int g = 0; g < 4; ++g) bias[mt][g] = u < H ? p.b[g * H + u] : 0.0f;
    }

    // Owned state: lane holds (row nt*16 + (l & 15), unit of gate tile mt).
    float cst[SM_MT][NT], hst[SM_MT][NT];
#pragma unroll
    for (int mt = 0; mt < SM_MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int n = nt * 16 + (l & 15);
            const int u = ((w * SM_MT + mt) * 16 + 4 * (l >> 4)) >> 2;
            const bool ok = n < B && u < H;
            cst[mt][nt] = ok && p.cell == CELL_LSTM ? p.c0[(size_t)n * H + u] : 0.0f;
            hst[mt][nt] = ok ? p.h0[(size_t)n * H + u] : 0.0f;
        }
    __syncthreads();
    const int ml = maxlen;

    // x fragments of one step: lane holds row nt*16 + (l & 15), K slice of D.
    F xf[NT][KD], xn[NT][KD];
    auto load_x = [&](F (&dst)[NT][KD], int t) {
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int n = nt * 16 + (l & 15);
            const size_t row = (size_t)min(n, B - 1) * T + min(t, T - 1);
#pragma unroll
            for (int ks = 0; ks < KD; ++ks) {
                F f = E::zero();
#pragma unroll
                for (int e = 0; e < E::KPL; ++e) {
                    const int k = ks * E::KSTEP + (l >> 4) * E::KPL + e;
                    const S v = X[row * D + min(k, D - 1)];
                    if constexpr (E::KPL == 1) f = k < D ? v : 0.0f;
                    else f[e] = k < D ? v : E::from_f32(0.0f);
                }
                dst[nt][ks] = f;
            }
        }
    };
    if (ml > 0) load_x(xf, 0);

    int iters = 0;  // termination from the state: steps in which some row ran
    int t = 0;
    for (; t < ml; ++t) {
        const SH* hcur = hs[t & 1];
        SH* hnext = hs[(t + 1) & 1];
        if (p.stop_v) {
            // Halting scores of h_t (the operand in LDS, k in order): a row
            // that ran step t-1 and scores > 0 has ended.  Every lane of a row
            // computes the same score; lane (row, unit 0) records it.
            if (t > 0) {
                if (ran[(t - 1) & 1] == 0) break;  // no row ran at step t-1: none runs again
                iters = t;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) {
                    const int n = nt * 16 + (l & 15);
                    float sc = 0.f;
                    for (int k = 0; k < H; ++k) sc += p.stop_v[k] * EH::to_f32(hcur[n * HS + k]);
                    const bool ends = n < B && t - 1 < len[n] && !ended[n] && sc + p.stop_c > 0.f;
                    __syncthreads();  // every lane has read ended[] before it changes
                    if (ends && w == 0 && (l >> 4) == 0) {
                        ended[n] = 1;
                        p.steps[n] = t;
                    }
                }
            }
            if (tid == 0) ran[t & 1] = 0;
            __syncthreads();
        }
        if (t + 1 < ml) load_x(xn, t + 1);
        f32x4_t acc[SM_MT][NT];
#pragma unroll
        for (int mt = 0; mt < SM_MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KD; ++ks)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int mt = 0; mt < SM_MT; ++mt) acc[mt][nt] = E::mfma(wf[mt][ks], xf[nt][ks], acc[mt][nt]);
#pragma unroll
        for (int ks = 0; ks < KH; ++ks)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const FH hf = EH::load(hcur + (nt * 16 + (l & 15)) * HS + ks * EH::KSTEP + (l >> 4) * EH::KPL);
#pragma unroll
                for (int mt = 0; mt < SM_MT; ++mt) acc[mt][nt] = EH::mfma(uf[mt][ks], hf, acc[mt][nt]);
            }
#pragma unroll
        for (int mt = 0; mt < SM_MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int n = nt * 16 + (l & 15);
                const int u = ((w * SM_MT + mt) * 16 + 4 * (l >> 4)) >> 2;
                if (u >= H) continue;
                if (t < len[n] && !ended[n]) {  // len[n] = 0 for padding rows
                    if (p.stop_v) ran[t & 1] = 1;
                    f32x4_t z = acc[mt][nt];
#pragma unroll
                    for (int g = 0; g < 4; ++g) z[g] += bias[mt][g];
                    float c = cst[mt][nt], h = hst[mt][nt];
                    apply_cell(p.cell, z, c, h);
                    cst[mt][nt] = c;
                    hst[mt][nt] = h;
                    if (p.seq) p.seq[((size_t)n * T + t) * H + u] = h;  // output at step t
                }
                hnext[n * HS + u] = EH::from_f32(hst[mt][nt]);
            }
        __syncthreads();
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int ks = 0; ks < KD; ++ks) xf[nt][ks] = xn[nt][ks];
    }

#pragma unroll
    for (int mt = 0; mt < SM_MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            const int n = nt * 16 + (l & 15);
            const int u = ((w * SM_MT + mt) * 16 + 4 * (l >> 4)) >> 2;
            if (n < B && u < H) {
                p.out_h[(size_t)n * H + u] = hst[mt][nt];
                p.out_c[(size_t)n * H + u] = cst[mt][nt];
            }
        }
    if (tid == 0) {
        int total = 0;
        for (int i = 0; i < B; ++i) total += len[i];
        p.meta->max_len = ml;
        p.meta->total_rows = total;
        p.meta->status = bad ? STATUS_BAD_LENGTHS : 0;
        // a loop that ran to ml: did some row run in its last step?
        if (p.stop_v && t == ml && ml > 0 && ran[(ml - 1) & 1] != 0) iters = ml;
        p.meta->iters = p.stop_v ? iters : ml;
    }
}

typedef void (*small_fn)(SmallParams);
struct SmallVariant { int bf16, kd, kh, nt; small_fn f; };
#define SV(BF, ET, EH, KD, KH, NT) {BF, KD, KH, NT, small_kernel<ET, EH, KD, KH, NT>}
static const SmallVariant kSmall[] = {
    // fp32: K-step 4; D <= 64, H <= 32; B <= 16 or 64
    SV(0, EltF32, EltF32, 4, 8, 1), SV(0, EltF32, EltF32, 16, 8, 1), SV(0, EltF32, EltF32, 4, 8, 4),
    SV(0, EltF32, EltF32, 16, 8, 4),
    // bf16 data (fp16 recurrent operands): K-step 32; D <= 128, H <= 32
    SV(1, EltBF16, EltH16, 1, 1, 1), SV(1, EltBF16, EltH16, 4, 1, 1), SV(1, EltBF16, EltH16, 1, 1, 4),
    SV(1, EltBF16, EltH16, 4, 1, 4),
};
#undef SV

// Smallest variant covering (D, H, B); fills *kd, *nt.  Returns false if none.
bool small_pick(int bf16, int B, int D, int H, int* kd, int* nt) {
    const int kstep = bf16 ? 32 : 4;
    const int kdn = (D + kstep - 1) / kstep, khn = (H + kstep - 1) / kstep;
    const int ntn = (B + 15) / 16;
    int best = -1;
    for (int i = 0; i < (int)(sizeof(kSmall) / sizeof(kSmall[0])); ++i) {
        const SmallVariant& v = kSmall[i];
        if (v.bf16 != bf16 || v.kd < kdn || v.kh < khn || v.nt < ntn) continue;
        if (best < 0 || v.kd * v.nt < kSmall[best].kd * kSmall[best].nt) best = i;
    }
    if (best < 0) return false;
    *kd = kSmall[best].kd;
    *nt = kSmall[best].nt;
    return true;
}

hipError_t launch_small(const Dims& d, int kd, int nt, const void* x, const int32_t* lengths,
                        const void* W, const void* U, const float* b, const float* h0,
                        const float* c0, float* out_h, float* out_c, float* seq,
                        const StopArgs* stop, const Workspace& ws, hipStream_t s) {
    small_fn f = nullptr;
    for (const SmallVariant& v : kSmall)
        if (v.bf16 == d.bf16 && v.kd == kd && v.nt == nt) f = v.f;
    if (!f) return hipErrorInvalidValue;
    SmallParams p{x, lengths, W, U, b, h0, c0, out_h, out_c, seq, ws.meta, d.B, d.D, d.H, d.T, d.cell,
                  stop ? stop->v : nullptr, stop ? stop->c : 0.0f, stop ? stop->steps : nullptr};
    hipLaunchKernelGGL(f, dim3(1), dim3(SM_THREADS), 0, s, p);
    return hipGetLastError();
}

}  // namespace ldyn
