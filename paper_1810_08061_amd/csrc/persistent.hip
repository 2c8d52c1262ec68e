// persistent.hip -- the LSTM time loop run on the device in one persistent kernel.
//
// The staged loop of the paper (Section 9 "RNN cells"; Appendix A) executes
// its whole body, every step, without returning to the host.  Here that loop
// is a persistent grid of `groups` workgroups, one per CU, all co-resident
// (cooperative launch).  Workgroup g owns 4*MT hidden units, i.e. 16*MT
// gate-interleaved columns of U, and keeps that slice of U in registers as
// MFMA A-fragments for the whole loop.  Per step t:
//   1. the KW waves split K = H; each forms partial C^T = U_slice^T h_t^T for
//      the active rows (slots [0, active(t)) after the length sort), one
//      16-row tile at a time, loading the h fragments of the next tiles while
//      the current tile's MFMAs run;
//   2. partials meet in LDS; the wave that owns a row tile adds them and the
//      prefetched Gx[t] (input projection + bias), applies the gate
//      non-linearities and updates c and h (in its registers); finished rows
//      are not touched (the per-row select of the paper);
//   3. the owner stores the tile's rows of this workgroup's slice of h_{t+1}
//      and marks the same segments of the buffer that will take h_{t+3} as
//      not yet written; Gx[t+1] goes to LDS by DMA.
// The loop bound max_len and active(t) are read on the device; when every row
// is done the loop ends.
//
// Exchange of h between workgroups (they sit on different XCDs, whose L2
// caches are not coherent with each other): h is stored and loaded with
// device-scope cache policy (sc1), so stores are written through to the
// coherence point and loads are served from it, with no L2 write-back or
// invalidate.  There is one grid barrier, at the start (it makes h_0 and the
// first marks visible); after it the steps synchronise through the data.  h
// lives in a ring of four buffers, and a segment not yet written for the
// coming step holds the all-ones pattern, a NaN that the stores never
// produce.  A reader polls its first row tile of h_t until no active row
// holds the marker and uses later tiles as loaded; a marker that slipped into
// an active row shows up as a NaN pre-activation, and the chunk is then redone
// with every tile polled.  Every wait is bounded (then ERR_TIMEOUT).
#include "launch.h"

namespace ldyn {

constexpr int P_LDS_KB = 144;           // dynamic LDS for partial sums and the Gx prefetch
constexpr int P_MAX_ROWS = 512;         // batch rows the variants hold (8 owned row tiles per wave)
constexpr int P_SC1 = 16;               // buffer-instruction cache policy: device scope

struct PersistParams {
    const void* U;
    const float* h0;
    const float* c0;
    float* out_h;
    float* out_c;
    const float* gx;
    void* hx;
    unsigned* bar;          // [0]: global counter, [64 * (1 + x)]: group counter x (256 bytes apart)
    Meta* meta;
    const int32_t* perm;
    const int32_t* offsets;
    int B, H, hpad, bpad, groups;
    unsigned long long timeout_ticks;
    unsigned long long* trace;  // [T + 1][4] timestamps from workgroup 0, or null
    float* seq;                 // output sequence [B][T][H] (fp32), or null
    // Termination from the state (variants with STOP): a row ends after a step
    // that leaves v . h + c > 0; steps[b] receives the steps row b ran.
    const float* stop_v;        // [H]
    float stop_c;
    int32_t* steps;             // [B], batch order; written by workgroup 0
    const int32_t* lengths;     // [B] caps (clamped to [0, T] here)
    int T;
    // Forward for training (variants with SAVE): each step keeps, per compact
    // row, the pre-activations z in place of the row's Gx and the state the
    // step started from in save_h, save_c ([rows][H], fp32).
    float* save_h;
    float* save_c;
};

// What a variant of the loop does besides the plain forward.
enum LoopMode { LM_PLAIN = 0, LM_STOP = 1, LM_SAVE = 2 };

// Logical workgroup index: consecutive workgroups are dispatched to different
// XCDs (round robin over 8); give the workgroups of one XCD adjacent unit
// ranges so the columns of U and Gx they read share L2 lines.
__device__ inline int logical_group(int bid, int groups) {
    if ((groups & 7) != 0) return bid;
    return (bid & 7) * (groups >> 3) + (bid >> 3);
}

__device__ inline void drain_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Data written before this kernel started and only read by it, seen through
// the constant address space: wave-uniform reads of it become scalar loads,
// which do not queue behind the vector loads in flight.
typedef const __attribute__((address_space(4))) int32_t const_i32;

// Barrier k (k = 0, 1, ...), split in two so work can be issued between the
// arrival and the wait.  Arrival happens only after every wave of the
// workgroup has drained its stores.
__device__ inline void grid_arrive(const PersistParams& p, int k) {
    drain_stores();
    __syncthreads();
    if (threadIdx.x == 0 && p.groups > 1) {
        const int x = blockIdx.x & 7;
        const unsigned members = (unsigned)((p.groups - x + 7) >> 3);
        const unsigned old = __hip_atomic_fetch_add(p.bar + 64 * (1 + x), 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        if (old + 1u == (unsigned)(k + 1) * members)
            __hip_atomic_fetch_add(p.bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// Returns false if the wait exceeded its bound (the timeout status bit is set
// and the caller abandons the loop).
__device__ inline bool grid_wait(const PersistParams& p, int k, int* lds_ok) {
    if (threadIdx.x == 0) {
        int ok = 1;
        if (p.groups > 1) {
            const int ngroups = p.groups < 8 ? p.groups : 8;
            const unsigned want = (unsigned)(k + 1) * (unsigned)ngroups;
            const unsigned long long t0 = wall_clock64();
            while (__hip_atomic_load(p.bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < want) {
                if (wall_clock64() - t0 > p.timeout_ticks) {
                    ok = 0;
                    __hip_atomic_fetch_or(&p.meta->status, STATUS_TIMEOUT, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        *lds_ok = ok;
    }
    __syncthreads();
    return *lds_ok;
}

// Device-scope loads/stores of the operand buffer through a buffer resource.
// An operand slot whose value for the coming step has not arrived yet holds
// the all-ones pattern (a NaN).  operand() never produces it: a NaN h that
// would convert to it is stored as the canonical quiet NaN instead.
template <typename E> struct HxIO;
// 16-bit operands (bf16 or fp16): T the element, V eight of them, QNAN the
// canonical quiet NaN's bits.
template <typename T, typename V, unsigned short QNAN> struct HxIO16 {
    __device__ static inline V load(__amdgpu_buffer_rsrc_t R, unsigned byte_off) {
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(R, byte_off, 0, P_SC1);
        return __builtin_bit_cast(V, v);
    }
    __device__ static inline T operand(float h) {
        const unsigned short b = __builtin_bit_cast(unsigned short, (T)h);
        return __builtin_bit_cast(T, b == 0xffffu ? QNAN : b);
    }
    __device__ static inline void store(__amdgpu_buffer_rsrc_t R, unsigned byte_off, float h) {
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, operand(h)), R, byte_off, 0,
                                              P_SC1);
    }
    // true if any of the KSW fragments holds the marker in one of its elements
    template <int KSW>
    __device__ static inline bool has_marker(const V* f) {
        typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        u16x2 m = {0, 0};
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks) {
            const u32x4 v = __builtin_bit_cast(u32x4, f[ks]);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const unsigned d = v[j];  // (a bit_cast of the subscript itself reads element 0)
                m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x2, d));
            }
        }
        return m[0] == 0xffffu || m[1] == 0xffffu;
    }
};
template <> struct HxIO<EltH16> : HxIO16<_Float16, f16x8_t, 0x7e00> {};

template <> struct HxIO<EltF32> {
    __device__ static inline float load(__amdgpu_buffer_rsrc_t R, unsigned byte_off) {
        return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(R, byte_off, 0, P_SC1));
    }
    __device__ static inline float operand(float h) {
        const unsigned b = __float_as_uint(h);
        return __uint_as_float(b == 0xffffffffu ? 0x7fc00000u : b);
    }
    __device__ static inline void store(__amdgpu_buffer_rsrc_t R, unsigned byte_off, float h) {
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(operand(h)), R, byte_off, 0, P_SC1);
    }
    template <int KSW>
    __device__ static inline bool has_marker(const float* f) {
        unsigned m = 0;
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks) m = max(m, __float_as_uint(f[ks]));
        return m == 0xffffffffu;
    }
};

// K index (relative to the wave's K range) of the first value lane l holds for
// MFMA K-step ks.  bf16: 8 consecutive k per lane per step.  fp32 with at
// least four steps: each lane holds 4 consecutive k for a group of four
// steps (one 16-byte load feeds four MFMAs); the A- and B-fragments use the
// same assignment, so the sum over k is unchanged.
template <typename E, int KSW>
__device__ inline int kslot(int ks, int l) {
    if constexpr (E::KPL == 1 && KSW >= 4) return 16 * (ks >> 2) + 4 * (l >> 4) + (ks & 3);
    else return ks * E::KSTEP + (l >> 4) * E::KPL;
}

// The operand buffer holds h in MFMA fragment order rather than row-major:
// 16-row tiles, each cut along k into 1 KB blocks of 64 sixteen-byte chunks;
// chunk q * 16 + r of a block holds row r of the tile and the q-th run of
// 16 / sizeof(element) consecutive k.  Lane l's fragment of one K-step (or,
// for fp32, of a group of four K-steps) is chunk l of one block, so a wave's
// load is 1 KB of consecutive addresses (every lane quad hits one 64-byte
// segment), and a workgroup's row segment of UPW <= 16 bytes stays inside
// one chunk.  Byte offset of h[s][k] within one half of the buffer:
template <typename E>
__device__ inline unsigned hx_off(int s, int k, int hpad) {
    constexpr int CK = 16 / (int)sizeof(typename E::store_t);  // elements per chunk
    constexpr int KB = 4 * CK;                                 // k per block
    const int blk = (s >> 4) * (hpad / KB) + k / KB;
    const int chunk = ((k % KB) / CK) * 16 + (s & 15);
    return (unsigned)(blk * 64 + chunk) * 16u + (unsigned)(k % CK) * (unsigned)sizeof(typename E::store_t);
}

// Dynamic LDS of one workgroup during the loop: partial sums of NTC row tiles
// ([KW][NTC][MT][64 lanes][4 floats]) followed by the prefetched Gx of G of
// each wave's owned row tiles ([G][MT][KW][64 lanes][4 floats]).  When the
// Gx of every owned tile fits next to the partial sums, all are staged at
// once; otherwise (G < NOT) a chunk is G * KW row tiles, so it holds exactly
// G owned tiles of each wave, and the Gx of an owned tile goes into the slot
// of the tile G before it once that one is committed.  For eight waves of two
// gate tiles this makes a chunk 8 row tiles instead of 7 (two chunks per
// step at 256 rows instead of three).
template <int MT, int KW, int NST>
struct PLayout {
    static constexpr int NOT = NST / MT;                        // owned row tiles per wave
    static constexpr int GMAX = P_LDS_KB / (KW * MT * (KW + 1));
    static constexpr int G = NOT <= GMAX ? NOT : GMAX;          // owned tiles with a Gx slot
    static constexpr int GX_KB = G * MT * KW;
    static constexpr int NTC = NOT <= GMAX ? (P_LDS_KB - GX_KB) / (KW * MT) : G * KW;  // row tiles per chunk
    static constexpr int GX_OFF = NTC * KW * MT * 256;          // in floats
    static constexpr int BYTES = (NTC * KW * MT + GX_KB) * 1024;
    static_assert(GMAX >= 1, "no room for the Gx of one owned tile");
};

template <typename E, int MT, int KSW, int KW, int NST, int CELL, int LMODE>
__global__ void __launch_bounds__(KW * 64, 1)
persistent_kernel(PersistParams p) {
    constexpr bool STOP = LMODE == LM_STOP;
    constexpr bool SAVE = LMODE == LM_SAVE;
    using S = typename E::store_t;
    using F = typename E::frag_t;
    using IO = HxIO<E>;
    using LY = PLayout<MT, KW, NST>;
    constexpr int NTC = LY::NTC;
    static_assert(NTC >= 1, "partial buffer too small");
    static_assert(NST % MT == 0, "a wave owns whole row tiles");
    constexpr int NOT = NST / MT;  // row tiles owned per wave
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int lds_ok, lds_abort, lds_nan;
    constexpr int UPW = 4 * MT;                      // hidden units per workgroup
    constexpr int SEG_BYTES = UPW * (int)sizeof(S);  // one row of this workgroup's h slice
    static_assert(SEG_BYTES == 8 || SEG_BYTES == 16, "h row segment must be 8 or 16 bytes");
    // per-wave gather of one owned row tile's h before its row segments are stored
    __shared__ __attribute__((aligned(16))) S hstage[KW][16 * UPW];
    // STOP: the read-out v in operand precision over the padded K range, each
    // wave's partial halting scores of the chunk's row tiles, and whether any
    // row ran at step t (slot t & 1)
    constexpr int VST = STOP ? KW * KSW * E::KSTEP : 1;
    __shared__ __attribute__((aligned(16))) S vst[VST];
    __shared__ float s_part[STOP ? KW : 1][STOP ? NTC : 1][16];
    __shared__ int lds_run[2];
    // slot -> batch row, for the output sequence's row addresses
    __shared__ int perm_s[P_MAX_ROWS];

    // tid and l are re-read through empty asm statements at the top of each
    // step and chunk, so values derived from them (addresses, row indices)
    // are recomputed where used instead of being kept live across the loop.
    int tid = threadIdx.x, l = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    float* const gxs = lds + LY::GX_OFF + w * 256;  // this wave's Gx slots, 1 KB per owned pair
    const int g = logical_group(blockIdx.x, p.groups);
    const int H = p.H, H4 = 4 * H, hpad = p.hpad;
    const int u0 = g * 4 * MT;
    const int kw0 = w * KSW * E::KSTEP;
    const int B = p.B, ntmax = (B + 15) >> 4;
    const unsigned hx_part = (unsigned)(p.bpad * hpad) * (unsigned)sizeof(S);  // one of four buffers
    const __amdgpu_buffer_rsrc_t R =
        __builtin_amdgcn_make_buffer_rsrc(p.hx, (short)0, (int)(4u * hx_part), 0x00020000);
    if (tid == 0) {
        lds_abort = 0;
        lds_nan = 0;
        lds_run[0] = 0;
        lds_run[1] = 0;
    }
    if constexpr (STOP) {
        for (int k = tid; k < VST; k += KW * 64) vst[k] = E::from_f32(k < H ? p.stop_v[k] : 0.0f);
    }
    if (p.seq)  // read after the prologue's barriers
        for (int i = tid; i < B; i += KW * 64) perm_s[i] = p.perm[i];
    F afrag[MT][KSW];

    // ---- U slice -> registers (A-fragments of U^T; rows = gate-interleaved columns).
    // The slice is staged through LDS transposed, ust[c'][k], with rows padded
    // by 16 bytes (spreads the 2/4-byte writes over banks, keeps the 16-byte
    // fragment reads aligned).  Out-of-range k and units stage as zeros.
    {
        using Src = typename E::src_t;
        const Src* U = static_cast<const Src*>(p.U);
        S* ust = reinterpret_cast<S*>(lds);
        constexpr int NCOL = 16 * MT, UPG = 4 * MT;  // columns, units per gate segment
        const int stride = hpad + 16 / (int)sizeof(S);
        const int total = hpad * NCOL;
        auto src_of = [&](int e, bool& ok) {
            const int k = e / NCOL, c = e - k * NCOL;
            const int gate = c / UPG, uu = c - gate * UPG;
            ok = k < H && u0 + uu < H;
            return ok ? (size_t)k * H4 + gate * H + u0 + uu : (size_t)0;
        };
        auto dst_of = [&](int e) {
            const int k = e / NCOL, c = e - k * NCOL;
            const int gate = c / UPG, uu = c - gate * UPG;
            return (4 * uu + gate) * stride + k;
        };
        auto stage = [&](int e) {
            bool ok;
            const S v = E::from_src(U[src_of(e, ok)]);
            ust[dst_of(e)] = ok ? v : E::from_f32(0.0f);
        };
        constexpr int ROUND = KW * 64 * 8;
        const int full = total / ROUND * ROUND;
        for (int e0 = 0; e0 < full; e0 += ROUND) {  // unguarded: eight loads in flight per thread
            Src v[8];
            bool ok[8];
#pragma unroll
            for (int r = 0; r < 8; ++r) v[r] = U[src_of(e0 + r * KW * 64 + tid, ok[r])];
#pragma unroll
            for (int r = 0; r < 8; ++r)
                ust[dst_of(e0 + r * KW * 64 + tid)] = ok[r] ? E::from_src(v[r]) : E::from_f32(0.0f);
        }
        for (int e = full + tid; e < total; e += KW * 64) stage(e);
        __syncthreads();
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int ks = 0; ks < KSW; ++ks)
                afrag[mt][ks] = E::load(ust + (mt * 16 + (l & 15)) * stride + kw0 + kslot<E, KSW>(ks, l));
        __syncthreads();  // the LDS is reused for partial sums
    }

    const int max_len = p.meta->max_len;
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    // One row's segment of this workgroup's h slice (UPW units), device scope.
    auto seg_store = [&](unsigned off, const S* v) {
        if constexpr (SEG_BYTES == 16)
            __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4*>(v), R, off, 0, P_SC1);
        else
            __builtin_amdgcn_raw_buffer_store_b64(*reinterpret_cast<const u32x2*>(v), R, off, 0, P_SC1);
    };
    auto seg_mark = [&](unsigned off) {
        if constexpr (SEG_BYTES == 16)
            __builtin_amdgcn_raw_buffer_store_b128(u32x4{~0u, ~0u, ~0u, ~0u}, R, off, 0, P_SC1);
        else
            __builtin_amdgcn_raw_buffer_store_b64(u32x2{~0u, ~0u}, R, off, 0, P_SC1);
    };
    // Wave w owns row tiles a * KW + w (a < NOT) with all MT gate tiles of this
    // workgroup: pair i = a * MT + mt.  It alone computes, stores and marks
    // their rows of this workgroup's h slice (lanes 0..15 hold the 16 rows), so
    // the marks of a segment and its later data come from the same wave.
    // Marks rows [0, rows) of the owned tiles in one buffer as not yet written.
    auto mark_owned = [&](unsigned part, int rows) {
        int lo = l;
        asm volatile("" : "+v"(lo));
#pragma unroll
        for (int a = 0; a < NOT; ++a) {
            const int s = (a * KW + w) * 16 + lo;
            if (lo < 16 && s < rows) seg_mark(part + hx_off<E>(s, u0, hpad));
        }
    };

    // ---- Owned state.  c and h live in registers and reach out_c / out_h
    // once, after the loop.  h_0 goes to buffer 0 as whole row segments (the
    // padding units of a ragged last workgroup as zeros).
    float cst[NST], hst[NST];
#pragma unroll
    for (int a = 0; a < NOT; ++a) {
        const int nt = a * KW + w;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int i = a * MT + mt;
            const int s = nt * 16 + (l & 15), u = u0 + mt * 4 + (l >> 4);
            cst[i] = 0.f;
            hst[i] = 0.f;
            if (nt < ntmax && s < B && u < H) {
                const size_t ib = (size_t)p.perm[s] * H + u;
                hst[i] = p.h0[ib];  // read before the final write: exact aliasing out_h == h0 is allowed
                if constexpr (CELL == CELL_LSTM) cst[i] = p.c0[ib];
            }
            hstage[w][(l & 15) * UPW + mt * 4 + (l >> 4)] = IO::operand(hst[i]);
        }
        __builtin_amdgcn_wave_barrier();
        if (nt < ntmax && l < 16 && nt * 16 + l < B) seg_store(hx_off<E>(nt * 16 + l, u0, hpad), &hstage[w][l * UPW]);
        __builtin_amdgcn_wave_barrier();
        if constexpr (STOP) {
            // a row that never ends early runs to its cap
            if (g == 0 && nt < ntmax && l < 16 && nt * 16 + l < B) {
                const int b = p.perm[nt * 16 + l];
                p.steps[b] = min(max(p.lengths[b], 0), p.T);
            }
        }
    }

    // Gx[t] of one owned tile goes straight from memory into this wave's LDS
    // slots (no registers held while it is in flight); lanes of rows that are
    // not active fetch row 0 instead, which is never read.
    auto prefetch_tile = [&](int a, int off, int act) {
        int lo = l;
        asm volatile("" : "+v"(lo));
        const int nt = a * KW + w;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const int s = nt * 16 + (lo & 15), u = u0 + mt * 4 + (lo >> 4);
            const bool ok = s < act && u < H;
            const float* src = p.gx + (ok ? (size_t)(off + s) * H4 + 4 * u : 0);
            __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)(gxs + ((a % LY::G) * MT + mt) * KW * 256),
                                             16, 0, 0);
        }
    };

    // Row offsets of steps t .. t+3 travel in registers; the one for t+4 is
    // loaded a step ahead.
    const_i32* const offs = (const_i32*)p.offsets;
    auto offset_at = [&](int t) { return offs[min(t, max_len)]; };
    int o0 = offset_at(0), o1 = offset_at(1), o2 = offset_at(2), o3 = offset_at(3);

    // h_0 sits in buffer 0 and buffers 1 and 2 are marked for h_1 and h_2; one
    // grid barrier (which drains every store) makes all of it visible.  After
    // that the steps synchronise through the data.
    mark_owned(hx_part, o2 - o1);
    mark_owned(2u * hx_part, o3 - o2);
    bool alive = true;
    if (max_len > 0) {
        grid_arrive(p, 0);
#pragma unroll
        for (int a = 0; a < LY::G; ++a)
            if ((a * KW + w) * 16 < o1 - o0) prefetch_tile(a, o0, o1 - o0);
        alive = grid_wait(p, 0, &lds_ok);
    }

    // fp32 lanes take 4 consecutive k for a group of four K-steps (one 16-byte
    // load); bf16 lanes take 8 consecutive k per K-step.  Either way a load is
    // one 1 KB block of the fragment-ordered buffer.
    static_assert(E::KPL == 8 || KSW % 4 == 0, "fp32 variants need whole groups of four K-steps");
    constexpr bool GROUPED = E::KPL == 1;
    constexpr int KB = GROUPED ? 16 : 32;  // k per 1 KB block
    const unsigned lane_off = (unsigned)(kw0 / KB) * 1024u + (unsigned)l * 16u;
    const unsigned tile_bytes = (unsigned)(16 * hpad) * (unsigned)sizeof(S);
    unsigned stopped = 0;  // STOP: bit a set once the lane's row of owned tile a has ended
    int iters = 0;         // STOP: steps in which some row ran
    int t = 0;
    for (; t < max_len && alive; ++t) {
        asm volatile("" : "+v"(tid), "+v"(l));
        const bool tr = p.trace && blockIdx.x == 0 && tid == 0;
        if (tr) p.trace[4 * t] = wall_clock64();
        const int o4 = offset_at(t + 4);  // used next step
        const int act = o1 - o0, act1 = o2 - o1;
        const int nt_act = (act + 15) >> 4;
        const unsigned cur = (unsigned)(t & 3) * hx_part;        // h_t
        const unsigned nxt = (unsigned)((t + 1) & 3) * hx_part;  // h_{t+1}
        // The owners of the previous step's row tiles may still be reading its
        // partial sums.
        __syncthreads();
        if constexpr (STOP) {
            // Every workgroup takes the same decisions from the same h, so all
            // leave together: once no row ran at step t-1, none runs again
            // (ended rows stay ended, caps only shrink the active prefix).
            if (t > 0) {
                if (lds_run[(t - 1) & 1] == 0) break;
                iters = t;
            }
            if (tid == 0) lds_run[t & 1] = 0;
        }

        constexpr int FRAG_REGS = KSW * (int)sizeof(F) / 4;
        // VGPRs per lane with KW / 4 waves per SIMD (less the halting score's with STOP)
        constexpr int REG_BUDGET = (KW <= 8 ? 256 : 2048 / KW) - (STOP ? 16 : 0);
        constexpr int DEPTH = (MT + 3) * FRAG_REGS < REG_BUDGET / 2    ? 3
                              : (MT + 2) * FRAG_REGS <= REG_BUDGET / 2 ? 2
                                                                       : 1;
        F f0[KSW], f1[DEPTH >= 2 ? KSW : 1], f2[DEPTH == 3 ? KSW : 1];
        // Lanes whose row of the tile is not active read row 0's chunk of
        // their k-run instead of their own: it lies in the same 64-byte
        // segment as the active rows' chunks, so the load moves no extra
        // lines, and the value only reaches the products of the inactive row,
        // which are never used.
        auto tile_base = [&](int nt) {
            const unsigned skip = (l & 15) >= act - nt * 16 ? (unsigned)(l & 15) * 16u : 0u;
            return cur + (unsigned)nt * tile_bytes + lane_off - skip;
        };
        auto load_tile = [&](F* f, int nt) {
            const unsigned base = tile_base(nt);
            if constexpr (GROUPED) {
                typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
                for (int ks = 0; ks < KSW; ks += 4) {
                    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(R, base + (ks >> 2) * 1024u, 0, P_SC1);
#pragma unroll
                    for (int j = 0; j < 4; ++j) f[ks + j] = __uint_as_float(v[j]);
                }
            } else {
#pragma unroll
                for (int ks = 0; ks < KSW; ++ks) f[ks] = IO::load(R, base + ks * 1024u);
            }
        };

        bool aborted = false;
        for (int ntc0 = 0; ntc0 < nt_act; ntc0 += NTC) {
            asm volatile("" : "+v"(tid), "+v"(l));
            const int nchunk = min(NTC, nt_act - ntc0);
            // Bounded waits: past the deadline the wave gives up, flags the
            // workgroup and the status, and the loop ends after this chunk.
            auto expired = [&](unsigned long long t0) {
                if (wall_clock64() - t0 <= p.timeout_ticks) return false;
                if (l == 0) {
                    lds_abort = 1;
                    __hip_atomic_fetch_or(&p.meta->status, STATUS_TIMEOUT, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                }
                return true;
            };
            // Reloads tile j until its active rows hold no marker.
            auto poll_tile = [&](F* f, int j) {
                const bool mine = ntc0 * 16 + j * 16 + (l & 15) < act;
                if (__builtin_amdgcn_ballot_w64(mine && IO::template has_marker<KSW>(f)) == 0) return;
                const unsigned long long t0 = wall_clock64();
                do {
                    if (expired(t0)) return;
                    __builtin_amdgcn_s_sleep(1);
                    load_tile(f, ntc0 + j);
                } while (__builtin_amdgcn_ballot_w64(mine && IO::template has_marker<KSW>(f)) != 0);
            };
            // Tile j's products with each K-step's fragment reloaded from tile
            // j+1 right after its MFMAs (one register set in flight).
            auto mma_roll = [&](F* f, int j) {
                f32x4_t acc[MT];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
                f32x4_t sacc = f32x4_t{0.f, 0.f, 0.f, 0.f};
                const unsigned next = tile_base(ntc0 + j + 1);
#pragma unroll
                for (int ks = 0; ks < KSW; ++ks) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) acc[mt] = E::mfma(afrag[mt][ks], f[ks], acc[mt]);
                    if constexpr (STOP) sacc = E::mfma(E::load(vst + kw0 + kslot<E, KSW>(ks, l)), f[ks], sacc);
                    if constexpr (GROUPED) {
                        if ((ks & 3) == 3) {
                            typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
                            const u32x4 v =
                                __builtin_amdgcn_raw_buffer_load_b128(R, next + (ks >> 2) * 1024u, 0, P_SC1);
#pragma unroll
                            for (int e = 0; e < 4; ++e) f[ks - 3 + e] = __uint_as_float(v[e]);
                        }
                    } else {
                        f[ks] = IO::load(R, next + ks * 1024u);
                    }
                }
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    *reinterpret_cast<f32x4_t*>(lds + ((((w * NTC + j) * MT + mt) * 64 + l) << 2)) = acc[mt];
                if constexpr (STOP) {
                    if (l < 16) s_part[w][j][l] = sacc[0];
                }
            };
            // Partial products of row tile j of the chunk into its LDS slot.
            auto mma_tile = [&](const F* f, int j) {
                f32x4_t acc[MT];
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < KSW; ++ks)
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) acc[mt] = E::mfma(afrag[mt][ks], f[ks], acc[mt]);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    *reinterpret_cast<f32x4_t*>(lds + ((((w * NTC + j) * MT + mt) * 64 + l) << 2)) = acc[mt];
                if constexpr (STOP) {
                    // halting score: every row of the A operand is v, so lane l
                    // gets this wave's partial v . h of row (l & 15) of the tile
                    f32x4_t sacc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KSW; ++ks)
                        sacc = E::mfma(E::load(vst + kw0 + kslot<E, KSW>(ks, l)), f[ks], sacc);
                    if (l < 16) s_part[w][j][l] = sacc[0];
                }
                // keep the reload of this register set after its MFMAs, so the
                // set is reused rather than renamed
                __builtin_amdgcn_sched_barrier(0);
            };

            // The chunk's first tile is polled until complete: that is where
            // a workgroup waits for the others.  Later tiles are nearly always
            // complete by then and are used as loaded.  A marker is a NaN, so
            // one that slipped into an active row shows up as a NaN in that
            // row's pre-activations; the chunk is then redone with every tile
            // polled.  (A NaN that the redo reproduces comes from the data and
            // is kept.)
            bool exact = false;
            float cn[NST], hn[NST];  // state update of this chunk, kept until it is verified
            unsigned ends = 0;       // STOP: owned tiles whose lane row ends before step t
            for (;;) {
                if (!exact) {
                    stress_delay(t, 1 + ntc0);
                    load_tile(f0, ntc0);
                    poll_tile(f0, 0);
                    if (tr && ntc0 == 0) p.trace[4 * t + 3] = wall_clock64();
                    if (nchunk == 1) {
                        mma_tile(f0, 0);
                    } else if constexpr (DEPTH == 1) {
                        for (int j = 0; j + 1 < nchunk; ++j) mma_roll(f0, j);
                        mma_tile(f0, nchunk - 1);
                    } else if (nchunk == 2 || DEPTH == 2) {
                        load_tile(f1, ntc0 + 1);
                        int j = 0;
                        for (; j + 3 < nchunk; j += 2) {
                            mma_tile(f0, j);
                            load_tile(f0, ntc0 + j + 2);
                            mma_tile(f1, j + 1);
                            load_tile(f1, ntc0 + j + 3);
                        }
                        if (nchunk - j == 2) {  // 2 or 3 tiles left, the first two loaded
                            mma_tile(f0, j);
                            mma_tile(f1, j + 1);
                        } else {
                            mma_tile(f0, j);
                            load_tile(f0, ntc0 + j + 2);
                            mma_tile(f1, j + 1);
                            mma_tile(f0, j + 2);
                        }
                    } else if constexpr (DEPTH == 3) {
                        load_tile(f1, ntc0 + 1);
                        load_tile(f2, ntc0 + 2);
                        int j = 0;
                        for (; j + 5 < nchunk; j += 3) {
                            mma_tile(f0, j);
                            load_tile(f0, ntc0 + j + 3);
                            mma_tile(f1, j + 1);
                            load_tile(f1, ntc0 + j + 4);
                            mma_tile(f2, j + 2);
                            load_tile(f2, ntc0 + j + 5);
                        }
                        const int rest = nchunk - j;  // 3, 4 or 5 tiles, the first three loaded
                        if (rest == 3) {
                            mma_tile(f0, j);
                            mma_tile(f1, j + 1);
                            mma_tile(f2, j + 2);
                        } else if (rest == 4) {
                            mma_tile(f0, j);
                            load_tile(f0, ntc0 + j + 3);
                            mma_tile(f1, j + 1);
                            mma_tile(f2, j + 2);
                            mma_tile(f0, j + 3);
                        } else {
                            mma_tile(f0, j);
                            load_tile(f0, ntc0 + j + 3);
                            mma_tile(f1, j + 1);
                            load_tile(f1, ntc0 + j + 4);
                            mma_tile(f2, j + 2);
                            mma_tile(f0, j + 3);
                            mma_tile(f1, j + 4);
                        }
                    }
                } else {
                    for (int j = 0; j < nchunk; ++j) {
                        load_tile(f0, ntc0 + j);
                        poll_tile(f0, j);
                        mma_tile(f0, j);
                    }
                }
                __syncthreads();
                if (lds_abort) {  // read by every wave between the same two barriers
                    aborted = true;
                    break;
                }
                if (tr && ntc0 == 0 && !exact) p.trace[4 * t + 1] = wall_clock64();
                // pre-activations of the owned pairs of this chunk.  The lane id
                // passes through an empty asm so the per-pair indices are
                // recomputed here rather than kept live across the loop.
                int lo = l;
                asm volatile("" : "+v"(lo));
                // this wave's Gx prefetch has landed, and so have its marks and
                // h stores of earlier steps
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                bool nan = false;
                ends = 0;
#pragma unroll
                for (int a = 0; a < NOT; ++a) {
                    const int j = a * KW + w - ntc0;
                    if (j < 0 || j >= nchunk) continue;
                    if constexpr (STOP) {
                        // halting score of the row's h_t: the waves' partials in
                        // a fixed order, then c; positive after step t-1 ends it
                        float sum = 0.f;
#pragma unroll
                        for (int ww = 0; ww < KW; ++ww) sum += s_part[ww][j][lo & 15];
                        if (t > 0 && sum + p.stop_c > 0.f) ends |= 1u << a;
                    }
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const int i = a * MT + mt;
                        // all partial reads first, then a tree sum (the reads overlap)
                        f32x4_t pv[KW + 1];
#pragma unroll
                        for (int ww = 0; ww < KW; ++ww)
                            pv[ww] = *reinterpret_cast<const f32x4_t*>(lds + ((((ww * NTC + j) * MT + mt) * 64 + lo) << 2));
                        pv[KW] = *reinterpret_cast<const f32x4_t*>(gxs + ((a % LY::G) * MT + mt) * KW * 256 + 4 * lo);
#pragma unroll
                        for (int span = 1; span <= KW; span *= 2)
#pragma unroll
                            for (int b = 0; b + span <= KW; b += 2 * span) pv[b] += pv[b + span];
                        const f32x4_t z = pv[0];
                        const int s = (j + ntc0) * 16 + (lo & 15);
                        const bool live = s < act;
                        if constexpr (SAVE) {
                            // z in place of this pair's Gx (its prefetch has landed);
                            // a redo pass stores again, last
                            const int u = u0 + mt * 4 + (lo >> 4);
                            if (live && u < H)
                                *reinterpret_cast<f32x4_t*>(const_cast<float*>(p.gx) + (size_t)(o0 + s) * H4 + 4 * u) = z;
                        }
                        nan |= live & ((z[0] != z[0]) | (z[1] != z[1]) | (z[2] != z[2]) | (z[3] != z[3]));
                        float c = cst[i], h = hst[i];
                        apply_cell(CELL, z, c, h);  // CELL is a template argument: no branch
                        cn[i] = c;
                        hn[i] = h;
                    }
                }
                // a one-tile chunk was polled in full: nothing left to verify
                if (exact || nchunk == 1) break;
                if (__builtin_amdgcn_ballot_w64(nan) != 0 && l == 0) lds_nan = 1;
                __syncthreads();
                const bool redo = lds_nan != 0;
                if (!redo) break;
                __syncthreads();  // every wave has read the flag
                if (tid == 0) lds_nan = 0;
                exact = true;
            }
            if (aborted) break;
            // Commit the owned tiles of the chunk and store their rows of h_{t+1}.
            {
                int lo = l;
                asm volatile("" : "+v"(lo));
#pragma unroll
                for (int a = 0; a < NOT; ++a) {
                    const int nt = a * KW + w;
                    const int j = nt - ntc0;
                    if (j < 0 || j >= nchunk) continue;
                    bool runs = true;
                    if constexpr (STOP) {
                        const int s = nt * 16 + (lo & 15);
                        if (((ends & ~stopped) >> a) & 1) {  // ends now: it ran t steps
                            if (g == 0 && lo < 16 && s < act) p.steps[p.perm[s]] = t;
                        }
                        stopped |= ends & (1u << a);
                        runs = !((stopped >> a) & 1);
                        if (runs && s < act) lds_run[t & 1] = 1;
                    }
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt) {
                        const int i = a * MT + mt;
                        const int s = nt * 16 + (lo & 15), u = u0 + mt * 4 + (lo >> 4);
                        if constexpr (SAVE) {
                            if (s < act && u < H) {  // the state this step started from
                                p.save_h[(size_t)(o0 + s) * H + u] = hst[i];
                                p.save_c[(size_t)(o0 + s) * H + u] = cst[i];
                            }
                        }
                        if (s < act && u < H && runs) {
                            cst[i] = cn[i];
                            hst[i] = hn[i];
                        }
                    }
                    // 16-bit operands: each lane stores its own elements of
                    // h_{t+1} (padding units of a ragged last workgroup as
                    // zeros); a reader checks every element for the marker, so a
                    // segment may arrive in parts.  fp32 operands: the tile's
                    // rows are gathered in this wave's staging slot and each
                    // active row leaves as one segment store (for fp32 the
                    // per-element stores made the loop 12% slower).
                    stress_delay(t, 64 + a);
                    if constexpr (E::KPL == 1) {
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt) {
                            const int u = u0 + mt * 4 + (lo >> 4);
                            hstage[w][(lo & 15) * UPW + mt * 4 + (lo >> 4)] =
                                u < H ? IO::operand(hst[a * MT + mt]) : E::from_f32(0.0f);
                        }
                        __builtin_amdgcn_wave_barrier();
                        if (lo < 16 && nt * 16 + lo < act)
                            seg_store(nxt + hx_off<E>(nt * 16 + lo, u0, hpad), &hstage[w][lo * UPW]);
                        __builtin_amdgcn_wave_barrier();
                    } else {
#pragma unroll
                        for (int mt = 0; mt < MT; ++mt) {
                            const int s = nt * 16 + (lo & 15), u = u0 + mt * 4 + (lo >> 4);
                            if (s < act) IO::store(R, nxt + hx_off<E>(s, u, hpad), u < H ? hst[a * MT + mt] : 0.0f);
                        }
                    }
                    if constexpr (LY::G < NOT) {
                        // the Gx of owned tile a + G (next chunk) into this tile's
                        // slot, which the gate math of the chunk has read
                        if (a + LY::G < NOT && ((a + LY::G) * KW + w) * 16 < act) prefetch_tile(a + LY::G, o0, act);
                    }
                    if (p.seq) {
                        // the output sequence: h of (row, unit) after step t, fp32,
                        // at out_seq[b][t] (a row that has ended keeps storing its
                        // state; the zeros written after the loop replace it)
                        const int s = nt * 16 + (lo & 15);
                        if (s < act) {
                            float* const row = p.seq + ((size_t)perm_s[s] * p.T + t) * H + u0;
#pragma unroll
                            for (int mt = 0; mt < MT; ++mt) {
                                const int u = u0 + mt * 4 + (lo >> 4);
                                if (u < H) row[mt * 4 + (lo >> 4)] = hst[a * MT + mt];
                            }
                        }
                    }
                }
            }
        }
        if (aborted) {
            alive = false;
            break;
        }
        if (tr) p.trace[4 * t + 2] = wall_clock64();
        // Gx[t+1] of the owned tiles, into the slots the gate math has read; it
        // is in flight while h_{t+1} arrives.  (Issued only now: the gate math
        // of a later chunk waits for every load of this wave.)
        if (t + 1 < max_len) {
#pragma unroll
            for (int a = 0; a < LY::G; ++a)
                if ((a * KW + w) * 16 < act1) prefetch_tile(a, o1, act1);
        }
        // Buffer (t+3) mod 4 still holds h_{t-1}.  This workgroup has seen rows
        // [0, act(t)) of every workgroup's h_t, so every workgroup has finished
        // reading h_{t-1} in those rows, which include every row active at t+3.
        // The marks drain before this wave's h_{t+2} stores of the same
        // segments (the wait before the gate math), so a reader that saw a
        // segment of h_{t+2} then sees its mark in buffer (t+3) mod 4.
        stress_delay(t, 128);
        mark_owned((unsigned)((t + 3) & 3) * hx_part, o4 - o3);
        o0 = o1;
        o1 = o2;
        o2 = o3;
        o3 = o4;
    }

    // Nothing of this wave may still be in flight when it ends (a loop left
    // early has a Gx prefetch into LDS outstanding).
    drain_stores();
    if constexpr (STOP) {
        // a loop that ran to max_len: did some row run in its last step?
        __syncthreads();
        if (alive && t == max_len && max_len > 0 && lds_run[(max_len - 1) & 1] != 0) iters = max_len;
        if (g == 0 && tid == 0) p.meta->iters = iters;
    }
    if (p.trace && blockIdx.x == 0 && tid == 0) p.trace[4 * max_len] = wall_clock64();
    // ---- final state, batch order
#pragma unroll
    for (int i = 0; i < NST; ++i) {
        const int nt = (i / MT) * KW + w, mt = i % MT;
        const int s = nt * 16 + (l & 15), u = u0 + mt * 4 + (l >> 4);
        if (nt < ntmax && s < B && u < H) {
            const size_t ib = (size_t)p.perm[s] * H + u;
            p.out_c[ib] = cst[i];
            p.out_h[ib] = hst[i];
        }
    }
}

// ---------------------------------------------------------------------------
// Variants: (element type, gate tiles per workgroup, K-steps per wave, waves,
// owned pairs per wave).  Register arrays are sized by these, so the plan
// picks the variant whose K-steps equal the problem's (rounded up to a power
// of two; the padding of the operand buffer is zero) and the smallest state
// capacity that covers the batch.
typedef void (*persist_fn)(PersistParams);

// f[cell][mode]: the variant compiled for each CellKind and LoopMode, so the
// gate step has no branch on either (a uniform branch on the cell there cost
// about 4% of the loop).
struct Variant { int bf16, mt, ksw, kw, nst, lds_bytes; persist_fn f[3][3]; };

#define PV_CELL(ET, MT, KS, KW, NS, C)                                                       \
    {persistent_kernel<ET, MT, KS, KW, NS, C, LM_PLAIN>, persistent_kernel<ET, MT, KS, KW, NS, C, LM_STOP>, \
     persistent_kernel<ET, MT, KS, KW, NS, C, LM_SAVE>}
#define PV(BF, ET, MT, KS, KW, NS)                                             \
    {BF, MT, KS, KW, NS, PLayout<MT, KW, NS>::BYTES,                            \
     {PV_CELL(ET, MT, KS, KW, NS, CELL_LSTM), PV_CELL(ET, MT, KS, KW, NS, CELL_GRU), \
      PV_CELL(ET, MT, KS, KW, NS, CELL_RNN)}}
#define PV_NST(BF, ET, MT, KS, KW) PV(BF, ET, MT, KS, KW, 2), PV(BF, ET, MT, KS, KW, 8)
static const Variant kVariants[] = {
    PV_NST(0, EltF32, 1, 4, 4),
    PV_NST(0, EltF32, 1, 8, 4), PV_NST(0, EltF32, 1, 16, 4), PV_NST(0, EltF32, 1, 32, 4),
    PV_NST(0, EltF32, 1, 64, 4),
    PV_NST(1, EltH16, 1, 1, 4), PV_NST(1, EltH16, 1, 2, 4), PV_NST(1, EltH16, 1, 4, 4),
    PV_NST(1, EltH16, 1, 8, 4),
    PV(1, EltH16, 2, 8, 8, 4), PV(1, EltH16, 2, 8, 8, 8),
};
#undef PV_NST
#undef PV
#undef PV_CELL

static persist_fn find_variant(int bf16, int mt, int ksw, int kw, int nst, int cell, int mode) {
    if (cell < CELL_LSTM || cell > CELL_RNN || mode < LM_PLAIN || mode > LM_SAVE) return nullptr;
    for (const Variant& v : kVariants)
        if (v.bf16 == bf16 && v.mt == mt && v.ksw == ksw && v.kw == kw && v.nst == nst)
            return v.f[cell][mode];
    return nullptr;
}

bool persistent_pick_variant(int bf16, int mt, int kw, int ksw, int nstate, int* nst) {
    int best = 0;
    for (const Variant& v : kVariants) {
        if (v.bf16 != bf16 || v.mt != mt || v.kw != kw || v.ksw != ksw || v.nst < nstate) continue;
        if (best == 0 || v.nst < best) best = v.nst;
    }
    if (best == 0) return false;
    *nst = best;
    return true;
}

// Dynamic LDS: the partial-sum chunks, or the staged U slice if larger.
int persistent_lds_bytes(int bf16, int mt, int kw, int nst, int hpad) {
    const int esz = bf16 ? 2 : 4;
    const int staged = 16 * mt * (hpad + 16 / esz) * esz;  // the U slice before the loop
    int loop = 0;
    for (const Variant& v : kVariants)
        if (v.bf16 == bf16 && v.mt == mt && v.kw == kw && v.nst == nst) loop = v.lds_bytes;
    return staged > loop ? staged : loop;
}

int persistent_blocks_per_cu(int bf16, int mt, int ksw, int kw, int nst, int lds_bytes, int cell,
                             int mode) {
    persist_fn f = find_variant(bf16, mt, ksw, kw, nst, cell, mode);
    if (!f) return 0;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes) != hipSuccess)
        return 0;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(f), kw * 64,
                                                     lds_bytes) != hipSuccess)
        return 0;
    return n;
}

hipError_t launch_persistent(const Dims& d, const PersistentConfig& pc, const void* U,
                             const float* h0, const float* c0, float* out_h, float* out_c,
                             const Workspace& ws, hipStream_t s) {
    const int mode = pc.stop ? LM_STOP : pc.save_h ? LM_SAVE : LM_PLAIN;
    persist_fn f = find_variant(d.bf16, pc.mt, pc.ksw, pc.kw, pc.nst, d.cell, mode);
    if (!f || (pc.seq && d.B > P_MAX_ROWS)) return hipErrorInvalidValue;
    PersistParams p{};
    p.U = U;
    p.h0 = h0;
    p.c0 = c0;
    p.out_h = out_h;
    p.out_c = out_c;
    p.gx = ws.gx;
    p.hx = ws.hx;
    p.bar = ws.bar;
    p.meta = ws.meta;
    p.perm = ws.perm;
    p.offsets = ws.offsets;
    p.B = d.B;
    p.H = d.H;
    p.hpad = d.hpad;
    p.bpad = d.bpad;
    p.groups = pc.groups;
    p.timeout_ticks = pc.timeout_ticks;
    p.trace = pc.trace;
    p.seq = pc.seq;
    p.T = d.T;
    p.save_h = pc.save_h;
    p.save_c = pc.save_c;
    if (pc.stop) {
        p.stop_v = pc.stop->v;
        p.stop_c = pc.stop->c;
        p.steps = pc.stop->steps;
        p.lengths = pc.stop->lengths;
        p.T = d.T;
    }
    void* args[] = {&p};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(f), dim3(pc.groups),
                                      dim3(pc.kw * 64), args, (unsigned)pc.lds_bytes, s);
}

}  // namespace ldyn
