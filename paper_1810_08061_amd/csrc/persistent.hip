// persistent.hip -- the LSTM time loop run on the device in one persistent kernel.
//
// The staged loop of the paper (Section 9 "RNN cells"; Appendix A) executes
// its whole body, every step, without returning to the host.  Here that loop
// is a persistent grid of `groups` workgroups, one per CU, all co-resident
// (cooperative launch).  Workgroup g owns 4*MT hidden units, i.e. 16*MT
// gate-interleaved columns of U, and keeps that slice of U in registers as
// MFMA A-fragments for the whole loop.  Per step t:
//   1. prefetch Gx[t] (input projection + bias) for the (row, unit) pairs it owns;
//   2. wait at the grid barrier until every workgroup has published h_t;
//   3. the four waves split K = H: each forms partial C^T = U_slice^T h_t^T for
//      the active rows (slots [0, active(t)) after the length sort);
//   4. partials meet in LDS; the owning wave adds them and Gx, applies the gate
//      non-linearities, and updates c and h, which live in its registers;
//      finished rows are not touched (the per-row select of the paper);
//   5. it writes its slice of h_{t+1} (MFMA operand type) and publishes it.
// The loop bound max_len and active(t) are read on the device; when every row
// is done the loop ends.  A grid of one workgroup synchronises with
// __syncthreads only.
#include "launch.h"

namespace ldyn {

constexpr int P_WAVES = 4;               // waves per workgroup; they split K
constexpr int P_THREADS = 64 * P_WAVES;
constexpr int P_LDS_TILES = 32;          // (row tile, gate tile) partials per wave in LDS

struct PersistParams {
    const void* U;
    const float* h0;
    const float* c0;
    float* out_h;
    float* out_c;
    const float* gx;
    void* hx;
    unsigned* flags;
    Meta* meta;
    const int32_t* perm;
    const int32_t* offsets;
    int B, H, hpad, bpad, groups, ksw;
    unsigned epoch;
    unsigned long long timeout_ticks;
};

// Logical workgroup index: consecutive workgroups are dispatched to different
// XCDs (round robin over 8); give the workgroups of one XCD adjacent unit
// ranges so the columns of U and Gx they read share L2 lines.
__device__ inline int logical_group(int bid, int groups) {
    if ((groups & 7) != 0) return bid;
    return (bid & 7) * (groups >> 3) + (bid >> 3);
}

// Grid barrier on per-workgroup arrival values.  Workgroup g publishes
// "h_k is written" by storing epoch + k + 1 into flags[g]; waiting for h_k
// means every flag is at least that value.  Values grow across forwards
// (epoch advances by T_max + 1 per forward), so no reset is needed.
__device__ inline void grid_publish(const PersistParams& p, int g, unsigned value) {
    // Each wave makes its own stores visible at device scope first.
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_store(p.flags + g, value, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}

// Returns false if the wait exceeded its bound (status flagged, loop abandoned).
__device__ inline bool grid_wait(const PersistParams& p, unsigned value, int* lds_ok) {
    if (threadIdx.x < 64) {
        const int lane = threadIdx.x;
        const unsigned long long t0 = wall_clock64();
        bool ok = true;
        while (true) {
            bool mine = true;
            for (int i = lane; i < p.groups; i += 64)
                mine &= __hip_atomic_load(p.flags + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= value;
            if (__all(mine)) break;
            if (wall_clock64() - t0 > p.timeout_ticks) {
                ok = false;
                if (lane == 0)
                    __hip_atomic_fetch_or(&p.meta->status, STATUS_TIMEOUT, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        if (lane == 0) *lds_ok = ok;
    }
    __syncthreads();
    return *lds_ok;
}

template <typename E, int MT, int KSWMAX, int NST>
__global__ void __launch_bounds__(P_THREADS, 1)
persistent_kernel(PersistParams p) {
    using S = typename E::store_t;
    using F = typename E::frag_t;
    constexpr int NTC = P_LDS_TILES / MT;  // row tiles per LDS chunk
    extern __shared__ __attribute__((aligned(16))) float lds[];  // [P_WAVES][NTC][MT][64][4]
    __shared__ int lds_ok;

    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const int single = p.groups == 1;
    const int g = logical_group(blockIdx.x, p.groups);
    const int H = p.H, H4 = 4 * H, hpad = p.hpad;
    const int u0 = g * 4 * MT;
    const int kw0 = w * p.ksw * E::KSTEP;
    const int B = p.B, ntmax = (B + 15) >> 4;
    S* hx0 = static_cast<S*>(p.hx);
    const size_t hx_stride = (size_t)p.bpad * hpad;

    // ---- U slice -> registers (A-fragments of U^T; rows = gate-interleaved columns).
    const S* U = static_cast<const S*>(p.U);
    F afrag[MT][KSWMAX];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int cp = (u0 + mt * 4) * 4 + (l & 15);  // global gate-interleaved column
        const int u = cp >> 2;
        const int col = gate_col(cp, H);
#pragma unroll
        for (int ks = 0; ks < KSWMAX; ++ks) {
            F f = E::zero();
            if (ks < p.ksw && u < H) {
                const int kb = kw0 + ks * E::KSTEP + (l >> 4) * E::KPL;
                if constexpr (E::KPL == 1) {
                    if (kb < H) f = U[(size_t)kb * H4 + col];
                } else {
#pragma unroll
                    for (int e = 0; e < E::KPL; ++e)
                        if (kb + e < H) f[e] = U[(size_t)(kb + e) * H4 + col];
                }
            }
            afrag[mt][ks] = f;
        }
    }

    // ---- Owned state: pair q = i*P_WAVES + w -> row tile q / MT, gate tile q % MT.
    // c lives in registers; h is written to out_h whenever it changes (rows
    // that never run keep h0, which is copied here).
    float cst[NST];
#pragma unroll
    for (int i = 0; i < NST; ++i) {
        const int q = i * P_WAVES + w, nt = q / MT, mt = q % MT;
        const int s = nt * 16 + (l & 15), u = u0 + mt * 4 + (l >> 4);
        cst[i] = 0.f;
        if (nt < ntmax && s < B && u < H) {
            const size_t ib = (size_t)p.perm[s] * H + u;
            const float hv = p.h0[ib];
            cst[i] = p.c0[ib];
            hx0[(size_t)s * hpad + u] = E::from_f32(hv);
            p.out_h[ib] = hv;  // exact aliasing out_h == h0 is allowed: same element, same lane
        }
    }

    // Gx[t] for the owned pairs, prefetched while the barrier wait is pending.
    f32x4_t gxv[NST];
    auto prefetch_gx = [&](int t) {
        const int off = p.offsets[t];
        const int act = p.offsets[t + 1] - off;
#pragma unroll
        for (int i = 0; i < NST; ++i) {
            const int q = i * P_WAVES + w, nt = q / MT, mt = q % MT;
            const int s = nt * 16 + (l & 15), u = u0 + mt * 4 + (l >> 4);
            gxv[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
            if (s < act && u < H)
                gxv[i] = *reinterpret_cast<const f32x4_t*>(p.gx + (size_t)(off + s) * H4 + 4 * u);
        }
    };

    const int max_len = p.meta->max_len;
    bool alive = true;
    if (max_len > 0) {
        prefetch_gx(0);
        if (single) {
            __syncthreads();
        } else {
            grid_publish(p, g, p.epoch + 1u);
            alive = grid_wait(p, p.epoch + 1u, &lds_ok);
        }
    }

    for (int t = 0; t < max_len && alive; ++t) {
        const int act = p.offsets[t + 1] - p.offsets[t];
        const int nt_act = (act + 15) >> 4;
        const S* hcur = hx0 + (size_t)(t & 1) * hx_stride;
        S* hnext = hx0 + (size_t)((t + 1) & 1) * hx_stride;

        for (int ntc0 = 0; ntc0 < nt_act; ntc0 += NTC) {
            const int nchunk = min(NTC, nt_act - ntc0);
            // partial products over this wave's K range
            for (int j = 0; j < nchunk; ++j) {
                const int row = (ntc0 + j) * 16 + (l & 15);
                const S* hrow = hcur + (size_t)row * hpad + kw0 + (l >> 4) * E::KPL;
                f32x4_t acc[MT];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSWMAX; ++ks) {
                    if (ks < p.ksw) {
                        const F bf = E::load(hrow + ks * E::KSTEP);
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt) acc[mt] = E::mfma(afrag[mt][ks], bf, acc[mt]);
                    }
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    *reinterpret_cast<f32x4_t*>(lds + ((((w * NTC + j) * MT + mt) * 64 + l) << 2)) = acc[mt];
            }
            __syncthreads();
            // reduce, gates, state update, own slice of h_{t+1}
#pragma unroll
            for (int i = 0; i < NST; ++i) {
                const int q = i * P_WAVES + w, nt = q / MT, mt = q % MT;
                const int j = nt - ntc0;
                if (j < 0 || j >= nchunk) continue;
                const int s = nt * 16 + (l & 15), u = u0 + mt * 4 + (l >> 4);
                if (s >= act || u >= H) continue;
                f32x4_t z = gxv[i];
#pragma unroll
                for (int ww = 0; ww < P_WAVES; ++ww)
                    z += *reinterpret_cast<const f32x4_t*>(lds + ((((ww * NTC + j) * MT + mt) * 64 + l) << 2));
                float c = cst[i], h;
                lstm_cell(z, c, h);
                cst[i] = c;
                hnext[(size_t)s * hpad + u] = E::from_f32(h);
                p.out_h[(size_t)p.perm[s] * H + u] = h;
            }
            __syncthreads();
        }
        if (t + 1 < max_len) {
            if (single) {
                prefetch_gx(t + 1);
            } else {
                grid_publish(p, g, p.epoch + (unsigned)(t + 2));
                prefetch_gx(t + 1);
                alive = grid_wait(p, p.epoch + (unsigned)(t + 2), &lds_ok);
            }
        }
    }

    // ---- final cell state, batch order
#pragma unroll
    for (int i = 0; i < NST; ++i) {
        const int q = i * P_WAVES + w, nt = q / MT, mt = q % MT;
        const int s = nt * 16 + (l & 15), u = u0 + mt * 4 + (l >> 4);
        if (nt < ntmax && s < B && u < H) p.out_c[(size_t)p.perm[s] * H + u] = cst[i];
    }
}

// ---------------------------------------------------------------------------
// Variants: (element type, gate tiles per workgroup, K-step capacity per wave,
// owned pairs per wave).  Register arrays are sized by the last two, so the
// plan picks the smallest variant that covers the problem.
typedef void (*persist_fn)(PersistParams);

struct Variant { int bf16, mt, kswmax, nst; persist_fn f; };

#define PV(BF, ET, MT, KS, NS) {BF, MT, KS, NS, persistent_kernel<ET, MT, KS, NS>}
static const Variant kVariants[] = {
    // one workgroup, H <= 32
    PV(0, EltF32, 8, 2, 2), PV(0, EltF32, 8, 2, 8), PV(0, EltF32, 8, 2, 16),
    PV(1, EltBF16, 8, 1, 2), PV(1, EltBF16, 8, 1, 8), PV(1, EltBF16, 8, 1, 16),
    // four hidden units per workgroup
    PV(0, EltF32, 1, 16, 2), PV(0, EltF32, 1, 16, 8), PV(0, EltF32, 1, 16, 16),
    PV(0, EltF32, 1, 64, 2), PV(0, EltF32, 1, 64, 8), PV(0, EltF32, 1, 64, 16),
    PV(1, EltBF16, 1, 4, 2), PV(1, EltBF16, 1, 4, 8), PV(1, EltBF16, 1, 4, 16),
    PV(1, EltBF16, 1, 8, 2), PV(1, EltBF16, 1, 8, 8), PV(1, EltBF16, 1, 8, 16),
    // eight hidden units per workgroup (H up to 2048 on 256 CUs)
    PV(1, EltBF16, 2, 16, 8), PV(1, EltBF16, 2, 16, 16),
};
#undef PV

static persist_fn find_variant(int bf16, int mt, int kswmax, int nst) {
    for (const Variant& v : kVariants)
        if (v.bf16 == bf16 && v.mt == mt && v.kswmax == kswmax && v.nst == nst) return v.f;
    return nullptr;
}

bool persistent_pick_variant(int bf16, int mt, int ksw, int nstate, int* kswmax, int* nst) {
    int best_k = 0, best_n = 0;
    for (const Variant& v : kVariants) {
        if (v.bf16 != bf16 || v.mt != mt || v.kswmax < ksw || v.nst < nstate) continue;
        if (best_k == 0 || v.kswmax < best_k || (v.kswmax == best_k && v.nst < best_n)) {
            best_k = v.kswmax;
            best_n = v.nst;
        }
    }
    if (best_k == 0) return false;
    *kswmax = best_k;
    *nst = best_n;
    return true;
}

int persistent_blocks_per_cu(int bf16, int mt, int kswmax, int nst, int lds_bytes) {
    persist_fn f = find_variant(bf16, mt, kswmax, nst);
    if (!f) return 0;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes) != hipSuccess)
        return 0;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(f),
                                                     P_THREADS, lds_bytes) != hipSuccess)
        return 0;
    return n;
}

hipError_t launch_persistent(const Dims& d, const PersistentConfig& pc, const void* U,
                             const float* h0, const float* c0, float* out_h, float* out_c,
                             const Workspace& ws, hipStream_t s) {
    persist_fn f = find_variant(d.bf16, pc.mt, pc.kswmax, pc.nst);
    if (!f) return hipErrorInvalidValue;
    PersistParams p{};
    p.U = U;
    p.h0 = h0;
    p.c0 = c0;
    p.out_h = out_h;
    p.out_c = out_c;
    p.gx = ws.gx;
    p.hx = ws.hx;
    p.flags = ws.flags;
    p.meta = ws.meta;
    p.perm = ws.perm;
    p.offsets = ws.offsets;
    p.B = d.B;
    p.H = d.H;
    p.hpad = d.hpad;
    p.bpad = d.bpad;
    p.groups = pc.groups;
    p.ksw = pc.ksw;
    p.epoch = pc.epoch;
    p.timeout_ticks = pc.timeout_ticks;
    void* args[] = {&p};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(f), dim3(pc.groups),
                                      dim3(P_THREADS), args, (unsigned)pc.lds_bytes, s);
}

}  // namespace ldyn
