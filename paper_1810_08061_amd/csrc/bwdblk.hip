// bwdblk.hip -- the whole reverse loop of the backward pass in one cooperative
// launch, for bf16 data on persistent handles with H a multiple of 256.
//
// Backpropagation through the masked loop of the paper's Section 9 "RNN
// cells" experiment.  Going back from the last step, the rows of step t are
// the prefix [0, active(t)) of the length sort, and each step takes
//   dh_t = dz_{t+1} U^T  (the rows that ran step t+1; U is [H][4H] with
//                          gate-interleaved columns 4u + gate)
// then the cell's backward for the rows of step t, which gives dz_t.
//
// Workgroup (kb, cb), one of H / 8, keeps in registers, as MFMA A-fragments,
// the block of U of the 32 hidden units [32 kb, 32 kb + 32) and the H gate
// columns [H cb, H cb + H): one of four column blocks, 128 KB at H = 2048,
// the size of the forward loop's slice.  Per step t:
//   * product: the block's share of dh_t for the rows that ran step t+1, the
//     sum over its H columns of dz_{t+1} U^T, from the fp16 dz of those
//     columns (each row's 32-column block scaled by the power of two its
//     writer chose, undone after that block's MFMA); the waves split the
//     columns, their partial sums meet in LDS, and the workgroup's sums for
//     its 32 units are published as its share;
//   * cell: the 8 units [32 kb + 8 cb, + 8) of the rows of step t take dh =
//     the four siblings' shares (kb, 0..3) in order (plus the carried term
//     and the output sequence's gradient); the cell's backward gives dz (kept
//     in fp32 over z for the weight gradients, published in fp16 under its
//     row block's scale), dc and the carried term.  A thread takes the same
//     (row, unit) pairs in every step, so where the batch pads to at most 256
//     rows their carried dh and dc stay in LDS for the whole loop, and a
//     step loads the cell's z and c (from HBM) right after publishing its
//     shares, while the siblings' shares are still on their way.
// Neither exchange has a barrier.  A value not yet written for its step
// holds the all-ones marker (a NaN that the writers never publish), and the
// reader polls for it: the product polls the first row tile of each chunk of
// dz (a marker that slipped into a later tile is a NaN in the sums, and the
// chunk is redone with every tile polled), the cell polls the shares.  Each
// exchange cycles through four slots by step.  A workgroup that has read all
// its siblings' shares of step t knows that every workgroup has finished the
// product of step t+1 (each sibling read dz_{t+1} from every writer of its
// column block, and the four column blocks cover all workgroups), so it puts
// the marker back into its blocks of the slots of the shares of step t+1 and
// of dz_{t+2}; it drains those stores before it publishes anything more, so
// a reader that has seen its later data sees the marks.
// A workgroup reads a quarter of each row's dz (4 KB of fp16 at H = 2048, as
// much as the forward loop reads of h per row), where one holding all 4H
// columns of a few units would read all of it; the exchange of the shares is
// the price.
// After the last step, one more product gives dh entering step 0: dH
// receives dh0 (slot order, unscaled) and dC dc0.
#include "launch.h"

namespace ldyn {

constexpr int BB_WAVES = 8;
constexpr int BB_NCB = 4;     // column blocks of U
constexpr int BB_UNITS = 32;  // hidden units (rows of U) per block
constexpr int BB_NTC = 8;     // row tiles per chunk of the product
constexpr int BB_SC1 = 16;    // buffer-instruction cache policy: device scope
constexpr int BB_RING = 4;    // slots of each exchange (dz and the shares of dh), by step
constexpr int BB_LDS_BYTES = BB_WAVES * BB_NTC * 2 * 64 * 16;  // the waves' partial sums
// With at most 256 padded rows (one row set per thread, 4 rows), the carried
// dh and dc of each thread's (row, unit) pairs stay in LDS for the whole
// loop: [2][4][512 threads] floats after the partial sums.
constexpr int BB_RES_ROWS = 4 * BB_WAVES * 8;
constexpr int BB_RES_BYTES = 2 * 4 * BB_WAVES * 64 * 4;
// Each thread's largest |dz| so far (float bits), after the partial sums.
constexpr int BB_AMAX_BYTES = BB_WAVES * 64 * 4;

typedef unsigned bb_u32x2 __attribute__((ext_vector_type(2)));
// Data written before the kernel started and only read by it (the step
// offsets), seen through the constant address space: scalar loads.
typedef const __attribute__((address_space(4))) int32_t bb_const_i32;
typedef unsigned bb_u32x4 __attribute__((ext_vector_type(4)));

struct BwdBlockParams {
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
    // Published dz in MFMA fragment order: [4 slots][bpad / 16 row tiles][4H / 32
    // column blocks][64 chunks of 16 bytes], chunk q * 16 + r holding row r
    // of the tile and columns 8 q .. 8 q + 7 of the block (fp16, each row's
    // block scaled by its own power of two); a wave's load of one block is
    // 1 KB of consecutive bytes.
    _Float16* dzx;
    float* dzs;              // [4 slots][bpad / 16][4H / 32][16 rows] the scales
    // shares of dh: [4 slots][4 column blocks][H / 32 unit blocks][bpad][32]
    float* pdh;
    unsigned* amax;          // largest |dz| over all rows, float bits (atomic maximum)
    unsigned long long timeout_ticks;
    // [T + 1][4] timestamps of workgroup 0, or null: per step t (at 4 t) its
    // start, its shares published, its cells done (the siblings' shares
    // awaited), the marks issued; at 4 max_len the product for dh0
    unsigned long long* trace;
    float alpha_u;           // 1 / su
    int B, H, T, bpad, groups;
};

// A chunk length as a type, for code unrolled per length.
template <int N> struct BbLen { static constexpr int value = N; };

template <int KSW, int CELL, bool RES>
__global__ void __launch_bounds__(BB_WAVES * 64, 1)
bwd_block_kernel(BwdBlockParams p) {
    // [BB_WAVES][BB_NTC][2][64][4] partial sums, each thread's largest |dz|, then
    // (RES) the carried dh and dc
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ int lds_nan, lds_abort;
    // tid and l are re-read through empty asm statements at the top of each
    // step, so that addresses derived from them are recomputed where used
    // rather than kept live across the step (which made the variants with
    // the largest U blocks spill)
    int tid = threadIdx.x, l = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int H = p.H, H4 = 4 * H, NKB = H / BB_UNITS, NBLK = H / 8;
    const unsigned bpad = (unsigned)p.bpad;
    // Consecutive workgroups are dispatched to different XCDs (round robin
    // over 8): number them so that the workgroups of one XCD share a column
    // block, whose dz they then read through one L2.
    const int g = (p.groups & 7) == 0 ? (blockIdx.x & 7) * (p.groups >> 3) + (blockIdx.x >> 3)
                                      : (int)blockIdx.x;
    const int cb = g / NKB, kb = g - cb * NKB;
    const int k0 = kb * BB_UNITS, c0 = cb * H;
    const int ks0 = w * KSW;  // this wave's first 32-column step within the block

    // U block -> registers: lane l of afrag[kt][ks] holds row k0 + 16 kt + (l & 15),
    // columns c0 + 32 (ks0 + ks) + 8 (l >> 4) .. + 8.
    f16x8_t afrag[2][KSW];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks)
            afrag[kt][ks] = *reinterpret_cast<const f16x8_t*>(
                p.u16 + (size_t)(k0 + 16 * kt + (l & 15)) * H4 + c0 + 32 * (ks0 + ks) + 8 * (l >> 4));

    const __amdgpu_buffer_rsrc_t Rz = __builtin_amdgcn_make_buffer_rsrc(
        p.dzx, (short)0, (int)((size_t)BB_RING * bpad * H4 * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t Rs = __builtin_amdgcn_make_buffer_rsrc(
        p.dzs, (short)0, (int)((size_t)BB_RING * bpad * NBLK * 4), 0x00020000);
    const __amdgpu_buffer_rsrc_t Rp = __builtin_amdgcn_make_buffer_rsrc(
        p.pdh, (short)0, (int)((size_t)BB_RING * BB_NCB * bpad * H * 4), 0x00020000);
    const unsigned NTP = bpad / 16;  // row tiles of one slot of the dz exchange
    // byte offset of the share of dh of (slot, column block c, row s, unit k)
    // in pdh
    auto share_off = [&](unsigned par, unsigned c, unsigned s, unsigned k) {
        return ((((par * BB_NCB + c) * (unsigned)NKB + (k >> 5)) * bpad + s) * 32u + (k & 31u)) * 4u;
    };

    // One row tile's dz fragments of this wave's columns and their scales
    // (inverted where the tile is multiplied, so that nothing waits for the
    // loads here).  Rows of the tile that did not run step t+1 hold values of
    // an earlier step: they reach only those rows' sums, which are not
    // published.
    auto load_tile = [&](f16x8_t* b, float* sc, unsigned pin, int nt) {
        const unsigned tb = (pin * NTP + (unsigned)nt) * (unsigned)NBLK + (unsigned)(c0 / 32 + ks0);
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks)
            b[ks] = __builtin_bit_cast(f16x8_t, __builtin_amdgcn_raw_buffer_load_b128(
                                                    Rz, (tb + (unsigned)ks) * 1024u + (unsigned)l * 16u, 0, BB_SC1));
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks)
            sc[ks] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                Rs, ((tb + (unsigned)ks) * 16u + (unsigned)(l & 15)) * 4u, 0, BB_SC1));
    };
    // Tile j of the chunk: this wave's partial sums of dh (rows of the tile,
    // the block's 32 units) into its LDS slot.
    auto mma_tile = [&](const f16x8_t* b, const float* sc, int j) {
        f32x4_t acc[2] = {f32x4_t{0.f, 0.f, 0.f, 0.f}, f32x4_t{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks) {
            const float inv = __builtin_amdgcn_rcpf(sc[ks]);  // a power of two: exact
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
                acc[kt] += __builtin_amdgcn_mfma_f32_16x16x32_f16(afrag[kt][ks], b[ks],
                                                                  f32x4_t{0.f, 0.f, 0.f, 0.f}, 0, 0, 0) *
                           inv;
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
            *reinterpret_cast<f32x4_t*>(lds + ((((w * BB_NTC + j) * 2 + kt) * 64 + l) << 2)) = acc[kt];
    };

    // Whether an active row of a loaded tile still holds the marker (all-ones
    // halves of dz or an all-ones scale: values not yet written for the
    // step).  Rows past actp may hold anything; their sums are not used.
    auto marked = [&](const f16x8_t* b, const float* sc, int nt, int actp) {
        const bool live = nt * 16 + (l & 15) < actp;
        bool m = false;
#pragma unroll
        for (int ks = 0; ks < KSW; ++ks) {
            const bb_u32x4 v = __builtin_bit_cast(bb_u32x4, b[ks]);
#pragma unroll
            for (int e = 0; e < 4; ++e) m |= (v[e] & 0xffffu) == 0xffffu || (v[e] >> 16) == 0xffffu;
            m |= __float_as_uint(sc[ks]) == 0xffffffffu;
        }
        return __builtin_amdgcn_ballot_w64(live && m) != 0;
    };
    // Reloads tile nt until its active rows hold no marker; false past the
    // deadline (the timeout status is set).
    auto poll_tile = [&](f16x8_t* b, float* sc, unsigned pin, int nt, int actp) {
        if (!marked(b, sc, nt, actp)) return true;
        const unsigned long long t0 = wall_clock64();
        do {
            if (wall_clock64() - t0 > p.timeout_ticks) {
                if (l == 0)
                    __hip_atomic_fetch_or(&p.meta->status, STATUS_TIMEOUT, __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
                return false;
            }
            __builtin_amdgcn_s_sleep(1);
            load_tile(b, sc, pin, nt);
        } while (marked(b, sc, nt, actp));
        return true;
    };

    const unsigned blk = (unsigned)((k0 + 8 * cb) >> 3);  // this workgroup's 32-column block of dz
    const int32_t* const off = p.offsets;
    const int max_len = p.meta->max_len;
    // RES: thread tid's carried dh and dc of row (tid >> 3) + 64 i, unit
    // k0 + 8 cb + (tid & 7), at [i][tid] (the rows and the unit of its cell
    // pairs, the same in every step)
    unsigned* const lds_am = reinterpret_cast<unsigned*>(lds + BB_LDS_BYTES / 4);
    float* const lds_dh = lds + (BB_LDS_BYTES + BB_AMAX_BYTES) / 4;
    float* const lds_dc = lds_dh + 4 * BB_WAVES * 64;
    lds_am[tid] = 0u;
    if constexpr (RES) {
        const int uc = k0 + 8 * cb + (tid & 7);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int s = (tid >> 3) + i * BB_WAVES * 8;
            lds_dh[i * BB_WAVES * 64 + tid] = s < p.B ? p.dH[(size_t)s * H + uc] : 0.0f;
            lds_dc[i * BB_WAVES * 64 + tid] = s < p.B ? p.dC[(size_t)s * H + uc] : 0.0f;
        }
    }
    // Step offsets off[t - 2] .. off[t + 2] travel in registers (scalars); the
    // one for the step after next is loaded a step ahead.  Indices are
    // clamped into [0, max_len]; the values they give outside the loop's
    // range are not used.
    const bb_const_i32* const offc = (const bb_const_i32*)off;
    auto off_at = [&](int i) { return offc[max(min(i, max_len), 0)]; };
    int o_m2 = off_at(max_len - 3), o_m1 = off_at(max_len - 2), o_0 = off_at(max_len - 1),
        o_p1 = off_at(max_len), o_p2 = off_at(max_len + 1);
    for (int t = max_len - 1; t >= -1; --t) {
        const int o_next = off_at(t - 3);  // off[t - 3]: off[t - 2] of the next step
        asm volatile("" : "+v"(tid), "+v"(l));
        // this thread's cell pairs: 8 lanes per row, one unit each
        const int ul = tid & 7, u = k0 + 8 * cb + ul;
        const bool last = t < 0;  // only the product: dh entering step 0
        const int actp = t + 1 < max_len ? o_p2 - o_p1 : 0;  // rows with dz_{t+1}
        const int actc = last ? 0 : o_p1 - o_0;             // rows that run step t
        // slots: dz_{t+1} read, and dz_t and the shares of step t written
        const unsigned pin = (unsigned)((t + 1) & (BB_RING - 1)), pout = (unsigned)(t & (BB_RING - 1));
        // step trace: stamps kept in scalar registers, stored after the step
        const bool tr = p.trace && blockIdx.x == 0 && w == 0;
        const int ti = last ? max_len : t;
        unsigned long long ts[4] = {0, 0, 0, 0};
        if (tr) ts[0] = wall_clock64();

        // ---- product: the block's share of dh_t, into pdh[cb].  dz_{t+1}
        // arrives without a barrier: each chunk's first tile is polled until
        // its active rows hold no marker (that is where a workgroup waits for
        // the others); later tiles are nearly always complete by then and are
        // used as loaded.  A marker that slipped into an active row is a NaN
        // in that row's sums (an all-ones half is a NaN, and so is an all-ones
        // scale), and the chunk is then redone with every tile polled; a NaN
        // that the redo reproduces comes from the data and is kept.
        const int ntp = (actp + 15) >> 4;
        __syncthreads();  // every wave is done with the last step's flags
        if (tid == 0) {
            lds_nan = 0;
            lds_abort = 0;
        }
        __syncthreads();
        // The cell's inputs (fresh rows from HBM every step) are loaded as
        // soon as the product's last chunk is published, so that their latency
        // passes during the wait for the siblings' shares (rows (tid >> 3) +
        // 64 i, clamped, as in the cell).
        const bool early = RES && !last && ntp > 0;
        f32x4_t zv[4];  // the cell's z, h and c of rows (tid >> 3) + 64 i
        float hp[4], cp[4];
        int ntc0 = 0, nchunk = 0;
        {
            // The waves' partial sums in order, for the (at most two) entries
            // (tile j, unit tile kt, lane ln) of this thread; lane ln holds
            // units 16 kt + 4 (ln >> 4) .. + 3 of row (ln & 15).  Returns
            // whether an active row's sum is a NaN.  They are published only
            // once verified: a sibling reads them as soon as they arrive.
            static_assert(BB_NTC * 128 <= 2 * BB_WAVES * 64, "two entries per thread");
            f32x4_t sums[2];
            auto reduce = [&]() {
                bool nan = false;
                int tq = tid;  // (addresses recomputed here, not kept live across the step)
                asm volatile("" : "+v"(tq));
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int e = tq + q * BB_WAVES * 64;
                    if (e < nchunk * 128) {
                        const int j = e >> 7, kt = (e >> 6) & 1, ln = e & 63;
                        f32x4_t sum = *reinterpret_cast<const f32x4_t*>(lds + (((j * 2 + kt) * 64 + ln) << 2));
#pragma unroll
                        for (int ww = 1; ww < BB_WAVES; ++ww)
                            sum += *reinterpret_cast<const f32x4_t*>(
                                lds + ((((ww * BB_NTC + j) * 2 + kt) * 64 + ln) << 2));
                        sums[q] = sum;
                        if ((ntc0 + j) * 16 + (ln & 15) < actp)
                            nan |= (sum[0] != sum[0]) | (sum[1] != sum[1]) | (sum[2] != sum[2]) | (sum[3] != sum[3]);
                    }
                }
                return nan;
            };
            // (after a redo the sums are formed again from the partial sums,
            // which are still in LDS, rather than kept in registers across it)
            auto publish = [&](bool again) {
                if (again) (void)reduce();
                int tq = tid;
                asm volatile("" : "+v"(tq));
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    const int e = tq + q * BB_WAVES * 64;
                    const int j = e >> 7, kt = (e >> 6) & 1, ln = e & 63;
                    const int s = (ntc0 + j) * 16 + (ln & 15);
                    if (e < nchunk * 128 && s < actp) {
                        // an all-ones word (the marker) goes out as the canonical quiet NaN
                        bb_u32x4 v = __builtin_bit_cast(bb_u32x4, sums[q]);
#pragma unroll
                        for (int x = 0; x < 4; ++x) v[x] = v[x] == 0xffffffffu ? 0x7fc00000u : v[x];
                        const unsigned k = (unsigned)(k0 + 16 * kt + 4 * (ln >> 4));
                        __builtin_amdgcn_raw_buffer_store_b128(v, Rp, share_off(pout, (unsigned)cb, (unsigned)s, k), 0,
                                                               BB_SC1);
                    }
                }
            };
            // Straight-line code per chunk length: DEPTH tiles are in flight,
            // and a tile's register set is reloaded with the tile DEPTH ahead
            // as soon as its products are formed.  (With conditional loads the
            // compiler waits for all loads in flight before every product, and
            // a wave then has one tile in flight.)  Reloading the polled first
            // tile instead of using it cost a load round trip per chunk.
            f16x8_t bp[KSW];  // the chunk's first tile, polled
            float sp[KSW];
            auto chunk = [&](auto len) {
                constexpr int N = decltype(len)::value;
                constexpr int DEPTH = KSW >= 8 ? 2 : 4;
                constexpr int D0 = N < DEPTH ? N : DEPTH;
                f16x8_t b[DEPTH][KSW];
                float sc[DEPTH][KSW];
#pragma unroll
                for (int ks = 0; ks < KSW; ++ks) {
                    b[0][ks] = bp[ks];
                    sc[0][ks] = sp[ks];
                }
#pragma unroll
                for (int j = 1; j < D0; ++j) load_tile(b[j], sc[j], pin, ntc0 + j);
#pragma unroll
                for (int j = 0; j < N; ++j) {
                    mma_tile(b[j % DEPTH], sc[j % DEPTH], j);
                    if (j + DEPTH < N) load_tile(b[j % DEPTH], sc[j % DEPTH], pin, ntc0 + j + DEPTH);
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            // The chunk's sums checked, redone if a marker slipped in, and
            // published; false if a wait ran out.  After publishing its last
            // chunk, a step loads the cell's inputs.
            auto finish = [&](bool last_chunk) {
                __syncthreads();
                if (lds_abort) return false;  // read by every wave between the same two barriers
                if (reduce()) lds_nan = 1;
            __syncthreads();
            const bool redo = lds_nan != 0;  // (read by every wave between the same two barriers)
            if (redo) {
                // a marker slipped into a tile used as loaded: once more with
                // every tile polled (a NaN then is the data's, and is kept)
                __syncthreads();  // every wave has read the flag and its sums
                if (tid == 0) lds_nan = 0;
                for (int j = 0; j < nchunk; ++j) {
                    f16x8_t b[KSW];
                    float sc[KSW];
                    load_tile(b, sc, pin, ntc0 + j);
                    if (!poll_tile(b, sc, pin, ntc0 + j, actp)) lds_abort = 1;
                    mma_tile(b, sc, j);
                }
                __syncthreads();
                if (lds_abort) return false;
            }
            publish(redo);  // (the checked sums, or, after a redo, the new ones)
            if (last_chunk && early) {
                int tq = tid;
                asm volatile("" : "+v"(tq));
                const int uq = k0 + 8 * cb + (tq & 7);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const size_t r = (size_t)o_0 + min((tq >> 3) + i * BB_WAVES * 8, actc - 1);
                    zv[i] = *reinterpret_cast<const f32x4_t*>(p.gx + r * H4 + 4 * uq);
                    hp[i] = p.save_h[r * H + uq];
                    cp[i] = p.save_c[r * H + uq];
                }
            }
            __syncthreads();  // the partial sums are read before the next chunk writes them
            return true;
            };
            for (; ntc0 < ntp; ntc0 += BB_NTC) {
                nchunk = min(BB_NTC, ntp - ntc0);
                // the first tile is polled; the pipeline starts from it, its
                // loads complete, while the next tiles are loaded
                stress_delay(t, 1 + ntc0);
                load_tile(bp, sp, pin, ntc0);
                if (!poll_tile(bp, sp, pin, ntc0, actp)) lds_abort = 1;
                switch (nchunk) {
                    case 1: chunk(BbLen<1>{}); break;
                    case 2: chunk(BbLen<2>{}); break;
                    case 3: chunk(BbLen<3>{}); break;
                    case 4: chunk(BbLen<4>{}); break;
                    case 5: chunk(BbLen<5>{}); break;
                    case 6: chunk(BbLen<6>{}); break;
                    case 7: chunk(BbLen<7>{}); break;
                    default: chunk(BbLen<BB_NTC>{}); break;
                }
                if (ntc0 + BB_NTC >= ntp) break;  // the last chunk is finished below
                if (!finish(false)) return;
            }
            if (ntp > 0 && !finish(true)) return;
        }
        if (tr) ts[1] = wall_clock64();

        // ---- cell: this workgroup's 8 units of the rows of step t, four rows
        // per thread at a time with all their loads issued before any use
        // (rows past the end load row rows - 1 and store nothing).  The
        // siblings' shares arrive without a barrier: they are polled until no
        // active row's share holds the marker.
        const int rows = last ? actp : actc;
        bool drained = false;
        for (int sb = tid >> 3; sb < rows; sb += 4 * BB_WAVES * 8) {
            float share[4][BB_NCB], dhc[4], dcc[4], ds[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int s = min(sb + i * BB_WAVES * 8, rows - 1);
                // rows without a product read a row that has one (or row 0),
                // and the sum is not used
                const unsigned sp = (unsigned)min(s, max(actp - 1, 0));
#pragma unroll
                for (int c = 0; c < BB_NCB; ++c)
                    share[i][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                        Rp, share_off(pout, (unsigned)c, sp, (unsigned)u), 0, BB_SC1));
                const size_t su = (size_t)s * H + u;
                dhc[i] = RES ? lds_dh[i * BB_WAVES * 64 + tid] : p.dH[su];
                if (!last) {  // (loaded while the shares are polled)
                    const size_t r = (size_t)o_0 + s;
                    if (!early) {
                        zv[i] = *reinterpret_cast<const f32x4_t*>(p.gx + r * H4 + 4 * u);
                        hp[i] = p.save_h[r * H + u];
                        cp[i] = p.save_c[r * H + u];
                    }
                    dcc[i] = RES ? lds_dc[i * BB_WAVES * 64 + tid] : p.dC[su];
                    ds[i] = p.dseq ? p.dseq[((size_t)p.perm[s] * p.T + t) * H + u] : 0.0f;
                }
            }
            auto shares_marked = [&]() {
                bool m = false;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int c = 0; c < BB_NCB; ++c)
                        m |= sb + i * BB_WAVES * 8 < actp && __float_as_uint(share[i][c]) == 0xffffffffu;
                return __builtin_amdgcn_ballot_w64(m) != 0;
            };
            if (shares_marked()) {
                const unsigned long long t0 = wall_clock64();
                do {
                    if (wall_clock64() - t0 > p.timeout_ticks) {
                        if (l == 0)
                            __hip_atomic_fetch_or(&p.meta->status, STATUS_TIMEOUT, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
                        return;  // the other workgroups' waits for this one end at their bounds
                    }
                    __builtin_amdgcn_s_sleep(1);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const unsigned sp =
                            (unsigned)min(min(sb + i * BB_WAVES * 8, rows - 1), max(actp - 1, 0));
#pragma unroll
                        for (int c = 0; c < BB_NCB; ++c)
                            share[i][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                                Rp, share_off(pout, (unsigned)c, sp, (unsigned)u), 0, BB_SC1));
                    }
                } while (shares_marked());
            }
            unsigned am = 0;  // largest |dz| of this thread's rows in the pass
            if (!drained) {
                // The marks this workgroup stored after its last cell (below)
                // complete before it publishes anything more, so a workgroup
                // that sees its later data also sees those marks.
                __builtin_amdgcn_s_waitcnt(0x0F70);
                drained = true;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int s = sb + i * BB_WAVES * 8;
                if (s < rows) {
                    float sum = 0.0f;
#pragma unroll
                    for (int c = 0; c < BB_NCB; ++c) sum += share[i][c];
                    float dh = (s < actp ? sum * p.alpha_u : 0.0f) + dhc[i];
                    const size_t su = (size_t)s * H + u;
                    if (last) {  // dh entering step 0: dh0
                        if constexpr (RES) lds_dh[i * BB_WAVES * 64 + tid] = dh;
                        else p.dH[su] = dh;
                        continue;
                    }
                    dh += ds[i];
                    const size_t r = (size_t)o_0 + s;
                    float dcp, dhd;
                    const f32x4_t dz = cell_backward<CELL>(zv[i], hp[i], cp[i], dh, dcc[i], dcp, dhd);
                    *reinterpret_cast<f32x4_t*>(p.gx + r * H4 + 4 * u) = dz;
                    if constexpr (RES) {
                        lds_dc[i * BB_WAVES * 64 + tid] = dcp;
                        lds_dh[i * BB_WAVES * 64 + tid] = dhd;
                    } else {
                        p.dC[su] = dcp;
                        p.dH[su] = dhd;
                    }
                    // the row block's scale: its largest magnitude into [2^13, 2^14)
                    unsigned m = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e) m = max(m, __float_as_uint(fabsf(dz[e])) & 0x7fffffffu);
                    for (int o = 4; o > 0; o >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, o));
                    am = max(am, m);
                    const float mf = __uint_as_float(m);
                    float sc = 1.0f;
                    if (mf > 0.0f && mf < 3.0e38f) {
                        int ex;
                        (void)frexpf(mf, &ex);
                        sc = ldexpf(1.0f, min(14 - ex, 126));
                    }
                    // fp16, an all-ones half (the marker) replaced by the canonical quiet NaN
                    unsigned short hb[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const unsigned short b16 = __builtin_bit_cast(unsigned short, (_Float16)(dz[e] * sc));
                        hb[e] = b16 == 0xffffu ? (unsigned short)0x7e00u : b16;
                    }
                    typedef unsigned short h4_t __attribute__((ext_vector_type(4)));
                    const h4_t hv = h4_t{hb[0], hb[1], hb[2], hb[3]};
                    // columns 4u .. 4u + 3: chunk (u & 7) / 2 of the block, its
                    // first or second half
                    const unsigned tb = (pout * NTP + (unsigned)(s >> 4)) * (unsigned)NBLK + blk;
                    stress_delay(t, 300 + i);
                    __builtin_amdgcn_raw_buffer_store_b64(
                        __builtin_bit_cast(bb_u32x2, hv), Rz,
                        tb * 1024u + ((unsigned)(ul >> 1) * 16u + (unsigned)(s & 15)) * 16u + (unsigned)(ul & 1) * 8u, 0,
                        BB_SC1);
                    if (ul == 0)
                        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(sc), Rs,
                                                              (tb * 16u + (unsigned)(s & 15)) * 4u, 0, BB_SC1);
                }
            }
            lds_am[tid] = max(lds_am[tid], am);
            if constexpr (RES) break;  // at most 256 rows: one pass (and no loop for the compiler)
        }
        if (tr) ts[2] = wall_clock64();
        // This workgroup has read every sibling's shares of step t, so every
        // sibling has finished its product of step t; each of those read dz_{t+1}
        // from every writer of its column block, so every workgroup has
        // finished its cell of step t+1 and its product of step t+1 (reading
        // dz_{t+2}).  The marker therefore goes back into this workgroup's
        // blocks of the slots of the shares of step t+1 and of dz_{t+2}, for
        // the rows of step t-2, which are written there next (at steps t-3 and
        // t-2).  The drain before this workgroup's next stores orders the
        // marks before them.
        if (t >= 2) {
            stress_delay(t, 200);
            const int rows_m = o_m1 - o_m2;
            const unsigned zslot = (unsigned)((t + 2) & (BB_RING - 1));
            const unsigned pslot = (unsigned)((t + 1) & (BB_RING - 1));
            for (int e = tid; e < rows_m * 4; e += BB_WAVES * 64) {
                const int sm = e >> 2, q = e & 3;
                const unsigned tb = (zslot * NTP + (unsigned)(sm >> 4)) * (unsigned)NBLK + blk;
                __builtin_amdgcn_raw_buffer_store_b128(bb_u32x4{~0u, ~0u, ~0u, ~0u}, Rz,
                                                       tb * 1024u + ((unsigned)q * 16u + (unsigned)(sm & 15)) * 16u, 0,
                                                       BB_SC1);
                if (q == 0)
                    __builtin_amdgcn_raw_buffer_store_b32(~0u, Rs, (tb * 16u + (unsigned)(sm & 15)) * 4u, 0, BB_SC1);
            }
            for (int e = tid; e < rows_m * 8; e += BB_WAVES * 64) {  // 8 x 16 bytes per row
                const int sm = e >> 3, q = e & 7;
                __builtin_amdgcn_raw_buffer_store_b128(bb_u32x4{~0u, ~0u, ~0u, ~0u}, Rp,
                                                       share_off(pslot, (unsigned)cb, (unsigned)sm,
                                                                 (unsigned)(k0 + 4 * q)),
                                                       0, BB_SC1);
            }
        }
        if (tr) {
            ts[3] = wall_clock64();
            if (l == 0)
#pragma unroll
                for (int e = 0; e < 4; ++e) p.trace[4 * ti + e] = ts[e];
        }
        o_p2 = o_p1;
        o_p1 = o_0;
        o_0 = o_m1;
        o_m1 = o_m2;
        o_m2 = o_next;
    }
    if constexpr (RES) {
        const int uc = k0 + 8 * cb + (tid & 7);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int s = (tid >> 3) + i * BB_WAVES * 8;
            if (s < p.B) {
                p.dH[(size_t)s * H + uc] = lds_dh[i * BB_WAVES * 64 + tid];
                p.dC[(size_t)s * H + uc] = lds_dc[i * BB_WAVES * 64 + tid];
            }
        }
    }
    {  // the largest |dz|: one atomic maximum per workgroup
        unsigned m = lds_am[tid];
        for (int o = 32; o > 0; o >>= 1) m = max(m, (unsigned)__shfl_xor((int)m, o));
        __syncthreads();  // every slot has been read
        if (l == 0) lds_am[w] = m;
        __syncthreads();
        if (tid == 0) {
            for (int ww = 1; ww < BB_WAVES; ++ww) m = max(m, lds_am[ww]);
            atomicMax(p.amax, m);
        }
    }
    // nothing of this wave in flight when it ends
    __builtin_amdgcn_s_waitcnt(0x0F70);
}

typedef void (*bwd_block_fn)(BwdBlockParams);

static bwd_block_fn bwd_block_pick(int H, int cell, bool res) {
#define BB_CELLS(K, R)                                                                           \
    if (H == 256 * K && res == R)                                                                \
        return cell == CELL_GRU ? bwd_block_kernel<K, CELL_GRU, R>                               \
               : cell == CELL_RNN ? bwd_block_kernel<K, CELL_RNN, R> : bwd_block_kernel<K, CELL_LSTM, R>;
    BB_CELLS(1, true) BB_CELLS(2, true) BB_CELLS(4, true) BB_CELLS(8, true)
    BB_CELLS(1, false) BB_CELLS(2, false) BB_CELLS(4, false) BB_CELLS(8, false)
#undef BB_CELLS
    return nullptr;
}

static int bwd_block_lds(const Dims& d) {
    return BB_LDS_BYTES + BB_AMAX_BYTES + (d.bpad <= BB_RES_ROWS ? BB_RES_BYTES : 0);
}

int bwd_block_fits(const Dims& d, int num_cus) {
    if (!d.bf16 || d.H % 256 != 0 || d.H > 2048 || d.bpad > 512) return 0;
    const int groups = d.H / 8;
    if (groups > num_cus) return 0;
    bwd_block_fn f = bwd_block_pick(d.H, d.cell, d.bpad <= BB_RES_ROWS);
    if (!f) return 0;
    int n = 0;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(f), hipFuncAttributeMaxDynamicSharedMemorySize,
                            bwd_block_lds(d)) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(f), BB_WAVES * 64,
                                                     bwd_block_lds(d)) != hipSuccess) {
        (void)hipGetLastError();  // not an error of a later call: another path serves
        return 0;
    }
    return n >= 1 ? groups : 0;
}

hipError_t launch_bwd_block(const Dims& d, const _Float16* u16, float alpha_u, const float* save_h,
                            const float* save_c, const float* dseq, float* dH, float* dC, _Float16* dzx,
                            float* dzs, float* pdh, unsigned* amax_dz, unsigned long long timeout_ticks,
                            unsigned long long* trace, const Workspace& ws, hipStream_t s) {
    bwd_block_fn f = bwd_block_pick(d.H, d.cell, d.bpad <= BB_RES_ROWS);
    if (!f || d.bpad > 512) return hipErrorInvalidValue;
    BwdBlockParams p{};
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
    p.pdh = pdh;
    p.amax = amax_dz;
    p.timeout_ticks = timeout_ticks;
    p.trace = trace;
    p.alpha_u = alpha_u;
    p.B = d.B;
    p.H = d.H;
    p.T = d.T;
    p.bpad = d.bpad;
    p.groups = d.H / 8;
    void* args[] = {&p};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(f), dim3(p.groups), dim3(BB_WAVES * 64),
                                      args, (unsigned)bwd_block_lds(d), s);
}

}  // namespace ldyn
