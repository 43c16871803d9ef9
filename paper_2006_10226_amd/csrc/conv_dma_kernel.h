// Implicit-GEMM quantized conv2d / dense with operands streamed straight
// into LDS (gfx950 buffer loads with the LDS-direct bit), for channel
// counts that are a multiple of 64.
//
// Arithmetic as in conv_mfma.hip (Jain et al., Sec. II-B Eq. (3), Sec.
// III-B/C): term 1 on int8 MFMA over x' = x - 128 (uint8 inputs) or x
// (int8), terms 2 and 4 and the bias folded into ChanRec.bconst, term 3
// from the window sums, requantize of Eq. (5) in the epilogue.
//
// What differs is the data path.  Every K-step is a 64-byte channel slice
// of one filter tap (C % 64 == 0), so each 16-byte chunk of the gather has
// the address  x + pixel_base(m) + tap_offset(r, s) + cc + 16 * q  and is
// fetched by one lane of a buffer load whose destination is LDS: a wave
// writes 1 KB (16 rows x 64 bytes) per instruction, lane L landing at byte
// 16 * L, so each lane fetches the chunk that the XOR swizzle places there.
// No registers hold staged tiles, so NS stages (NS - 1 of them in flight)
// cover the memory latency, with one barrier per K-step.
//
// Two consequences of skipping the registers:
//   * the uint8 -> int8 flip (XOR 0x80 per byte) is applied to the
//     activation fragments after they are read from LDS;
//   * a tap outside the image is fetched from an out-of-range offset, which
//     the hardware answers with zero bytes, i.e. x = 0 instead of the
//     padding value zp_x.  The difference, zp_x times the sum of the
//     weights of the outside taps, depends only on which taps are outside
//     (the pixel's border class) and the channel; the plan tabulates it
//     and the epilogue adds it (store_tile).
#pragma once

#include "conv_common.h"

#include <type_traits>

namespace qnn {

using namespace conv;

namespace dma {

// s_waitcnt with only the vector-memory count set (gfx9 encoding: vmcnt
// low bits 3:0 and high bits 15:14, expcnt 6:4 and lgkmcnt 11:8 at their
// no-wait maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier for the stage ring: this wave's LDS-direct loads up to
// the stage about to be read have landed (vmcnt N) and its LDS reads of the
// stage about to be overwritten have returned (lgkmcnt 0) before it
// arrives.  A plain __syncthreads would also wait for the loads still in
// flight (they write LDS), draining the pipeline at every K-step.
template <int N>
__device__ __forceinline__ void stage_barrier()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Swizzle of 64-byte LDS rows: physical chunk = logical chunk ^ sw64(row).
// Measured on gfx950 (bank-conflict counter): with it, the 64 lanes of an
// operand read (row L % 16, chunk L / 16) are conflict free.
__device__ __forceinline__ int sw64(int row)
{
    return (row >> 1) & 3;
}

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, int8_t *lds_dst, int voff, int soff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void *)lds_dst, 16, voff, soff, 0,
                                             0);
}

}  // namespace dma

using namespace dma;

template <int WTC, int WTP>
constexpr int dma_occupancy()
{
    return WTC * WTP >= 128 * 64 ? 1 : 2;
}

// SHORT: reductions of at most NS K-steps (1x1 convolutions with few input
// channels).  All NS stages are issued at once into their own buffers (no
// ring), so the LDS footprint is only NS stages and more workgroups stay
// resident to cover the memory latency of these one-pass tiles.
// KS = 2 (ring form only): two groups of WC x WP waves share the tile and
// take alternate K-steps, each through its own half of the ring (NS / 2
// stages); the second group's partial sums are added through LDS before
// the first group's epilogue.  For tiles too few to fill the chip this
// puts two waves on each SIMD and twice the MFMA work behind each barrier.
// FUSE: the epilogue applies the residual add (store_tile).
template <int TC, int TP, int WC, int WP, int NS, bool FLIP, bool SHORT, int KS = 1, bool SPLIT = false,
          bool FUSE = false>
__global__ void __launch_bounds__(WC *WP * 64 * KS, (KS > 1 ? 1 : dma_occupancy<TC / WC, TP / WP>()))
    conv_dma_kernel(ConvArgs a)
{
    constexpr int NW = WC * WP;     // waves of one group
    constexpr int BK = 64;
    constexpr int WTC = TC / WC, WTP = TP / WP;
    constexpr int FC = WTC / 16, FP = WTP / 16;
    constexpr int STAGE = (TC + TP) * BK;
    constexpr int LA = TC / (16 * NW);   // 1 KB weight blocks per wave per stage
    constexpr int LB = TP / (16 * NW);   // 1 KB activation blocks per wave per stage
    constexpr int LPS = LA + LB;         // loads per lane per stage
    constexpr int NSG = NS / KS;        // ring stages of one group
    constexpr int LDS_BYTES = NS * STAGE > TP * (TC + 16) ? NS * STAGE : TP * (TC + 16);
    static_assert(TC % (16 * NW) == 0 && TP % (16 * NW) == 0, "every wave loads whole 16-row blocks");
    static_assert((NS & (NS - 1)) == 0 && (NSG & (NSG - 1)) == 0, "stage counts are powers of two");
    static_assert(KS == 1 || KS == 2, "one or two K-step groups");
    static_assert(KS == 1 || (!SHORT && NW * FC * FP * 1024 <= LDS_BYTES), "split groups: ring form, partials fit");
    static_assert(LPS * (SHORT ? NS - 1 : NSG - 2) < 64, "vmcnt range");
    static_assert(SHORT || NSG >= 4, "the fragment prefetch needs stage k + 1 to land one step early");
    static_assert(!SPLIT || (!SHORT && KS == 1), "split reductions: ring form, one K-step group");
    static_assert(!FUSE || !SPLIT, "the fused add has no split-reduction form");

    __shared__ __attribute__((aligned(1024))) int8_t lds[LDS_BYTES];
    // the tile's channel records, fetched at the start for the epilogue
    __shared__ __attribute__((aligned(16))) ChanRec recs[TC];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave_id = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int grp = KS == 1 ? 0 : wave_id / NW;         // K-step group: steps grp, grp + KS, ...
    const int wave = KS == 1 ? wave_id : wave_id % NW;   // wave inside its group
    const int wc = wave / WP, wpos = wave % WP;

    // XCD x (workgroups dealt round-robin) takes the x-th eighth of the
    // work list; consecutive tiles are the channel tiles of one pixel tile.
    // Split reduction (a.ksplit = S > 1, ring form): a work unit is one of
    // the S parts of a tile's K-steps, and the S parts of a tile are
    // consecutive units, so they run on one XCD at the same time.
    const int S = SPLIT ? a.ksplit : 1;
    const int units = a.ntiles * S;
    const int chunk = (units + 7) >> 3;
    const int xcd = blockIdx.x & 7;
    const int unit = xcd * chunk + (blockIdx.x >> 3);
    if (unit >= min(units, (xcd + 1) * chunk))
        return;
    const int tile = SPLIT ? unit / S : unit;
    const int part = SPLIT ? unit - tile * S : 0;
    // this unit's K-steps: [kbeg, kbeg + nk)
    const int kbeg = SPLIT ? (int)((long long)part * a.nk / S) : 0;
    const int nk = SPLIT ? (int)((long long)(part + 1) * a.nk / S) - kbeg : a.nk;
    const int c0 = (tile % a.tiles_c) * TC;
    const int p0 = (tile / a.tiles_c) * TP;

    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, (short)0, a.N * a.H * a.W * a.C, kBufFlags);
    const __amdgpu_buffer_rsrc_t rw =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.wp, (short)0, a.Kpad * a.Jpad, kBufFlags);
    if (grp == 0 && wave == NW - 1) {
        // records c0 .. c0 + TC - 1 (c0 + TC <= Kpad), a kilobyte per load;
        // older than this wave's stage loads, so every stage wait covers them
        const __amdgpu_buffer_rsrc_t rc =
            __builtin_amdgcn_make_buffer_rsrc((void *)a.chan, (short)0, a.Kpad * (int)sizeof(ChanRec), kBufFlags);
#pragma unroll
        for (int q = 0; q < TC / 64; ++q)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rc, (__attribute__((address_space(3))) void *)(recs + q * 64), 16,
                                                     (c0 + q * 64 + lane) * (int)sizeof(ChanRec), 0, 0, 0);
    }

    // A 16-row x 64-byte block: lane L of the LDS-direct load that writes
    // it lands at byte 16 * L, i.e. row L / 4, physical chunk L % 4, and
    // fetches logical chunk (L % 4) ^ sw(row), so four consecutive lanes
    // read one 64-byte run of global memory.  The operand reads (lane L:
    // row L % 16, logical chunk L / 16) are then free of bank conflicts.
    const int r16 = lane >> 2, pch = lane & 3;
    int voffA[LA];
#pragma unroll
    for (int i = 0; i < LA; ++i) {
        const int row = (i * NW + wave) * 16 + r16;
        voffA[i] = (c0 + row) * a.Jpad + ((pch ^ sw64(row)) << 4);
    }
    int pbase[LB];
    uint32_t pmask[LB];
#pragma unroll
    for (int i = 0; i < LB; ++i) {
        const int row = (i * NW + wave) * 16 + r16;
        const int m = p0 + row;
        pbase[i] = 0;
        pmask[i] = 0;
        if (m < a.M && a.rowpack) {
            // row-pair mode: K-step s holds filter rows 2s and 2s + 1, each a
            // 32-byte run of the zero-point-padded image starting at the
            // window's first tap; logical chunk q: row q / 2, half q % 2
            const int t = fast_div(m, a.mWo, a.sWo);
            const int ow = m - t * a.Wo;
            const int n = fast_div(t, a.mHo, a.sHo);
            const int oh = t - n * a.Ho;
            const int q = pch ^ sw64(row);
            pbase[i] = ((n * a.H + oh * a.sh) * a.W + ow * a.sw) * a.C + (q >> 1) * a.row_bytes + (q & 1) * 16;
            pmask[i] = 0xffffffffu;
        } else if (m < a.M) {
            const int t = fast_div(m, a.mWo, a.sWo);
            const int ow = m - t * a.Wo;
            const int n = fast_div(t, a.mHo, a.sHo);
            const int oh = t - n * a.Ho;
            const int ih0 = oh * a.sh - a.pt, iw0 = ow * a.sw - a.pl;
            pbase[i] = ((n * a.H + ih0) * a.W + iw0) * a.C + ((pch ^ sw64(row)) << 4);
            uint32_t rm = 0, cm = 0;
            for (int r = 0; r < a.R; ++r)
                rm |= (uint32_t)((unsigned)(ih0 + r * a.dh) < (unsigned)a.H) << r;
            for (int s = 0; s < a.S; ++s)
                cm |= (uint32_t)((unsigned)(iw0 + s * a.dw) < (unsigned)a.W) << s;
            pmask[i] = rm | (cm << 16);
        }
    }

    // ---- loader: tap (lr, ls) and channel offset lc of the next stage ---
    int lr = 0, ls = 0, lc = 0;
    int voffB[LB];
    auto set_tap = [&]() {
        const int toff = a.rowpack ? lr * 2 * a.row_bytes : (lr * a.dh * a.W + ls * a.dw) * a.C;
        const uint32_t rin = lr < a.R ? 1u : 0u;
#pragma unroll
        for (int i = 0; i < LB; ++i) {
            const bool v = (pmask[i] >> lr) & (pmask[i] >> (16 + ls)) & rin;
            voffB[i] = v ? pbase[i] + toff : kOutOfRange;
        }
    };
    // one K-step of the loader: channel slice, then tap; steps past the end
    // of the unit's reduction are cut by the liveness test of issue()
    int wk = kbeg;   // K-step whose weights the next issue loads
    auto advance = [&]() {
        ++wk;
        lc += BK;
        if (lc == a.C) {
            lc = 0;
            if (++ls == a.S) {
                ls = 0;
                if (++lr == a.R)
                    lr = 0;
            }
            set_tap();
        }
    };
    // loader position of K-step k0 (C % 64 == 0: whole taps of C / 64 steps)
    auto start_at = [&](int k0) {
        wk = k0;
        const int cpt = a.C / BK;
        const int t = k0 / cpt;
        lc = (k0 - t * cpt) * BK;
        lr = t / a.S;
        ls = t - lr * a.S;
    };
    // LDS buffer of a group's local stage ks (global K-step ks * KS + grp)
    auto stage_buf = [&](int ks) { return lds + ((ks & (NSG - 1)) * KS + grp) * STAGE; };
    // Stages past the end are issued too (out of range: zeros, no memory
    // traffic), so every K-step waits for the same count.  Out of range is
    // signalled in the VGPR offset (>= 2^31) with a small scalar offset.
    auto issue = [&](int ks) {
        int8_t *base = stage_buf(ks);
        const int gs = ks * KS + grp;
        const bool live = gs < nk;
        const int soffA = __builtin_amdgcn_readfirstlane(live ? (a.rowpack ? gs : wk) * BK : 0);
        const int oob = __builtin_amdgcn_readfirstlane(live ? 0 : kOutOfRange);
        const int soffB = __builtin_amdgcn_readfirstlane(lc);
#pragma unroll
        for (int i = 0; i < LA; ++i)
            dma16(rw, base + (i * NW + wave) * 16 * BK, voffA[i] | oob, soffA);
#pragma unroll
        for (int i = 0; i < LB; ++i)
            dma16(rx, base + TC * BK + (i * NW + wave) * 16 * BK, voffB[i] | oob, soffB);
        if (a.rowpack) {
            ++lr;   // next row pair; lr == R (pairs) past the end: out of range
            set_tap();
            return;
        }
#pragma unroll
        for (int q = 0; q < KS; ++q)
            advance();
    };

    // ---- fragments and MFMAs ------------------------------------------
    const int lrow = lane & 15, lchk = lane >> 4;
    const int co = (lchk ^ sw64(lrow)) << 4;
    v4i acc[FC][FP];
#pragma unroll
    for (int i = 0; i < FC; ++i)
#pragma unroll
        for (int j = 0; j < FP; ++j)
            acc[i][j] = v4i{0, 0, 0, 0};
    v4i fa[2][FC], fb[2][FP];
    // fragment reads as lds_read16: the stage waits and barriers below order
    // them after their stage's LDS-direct loads, while the compiler would
    // wait for every stage in flight
    static_assert(FC + FP <= 15, "fragment reads of one step exceed the lgkmcnt range");
    auto read_frags = [&](int ks, v4i (&A)[FC], v4i (&B)[FP]) {
        const int8_t *As = stage_buf(ks) + (wc * WTC + lrow) * BK + co;
        const int8_t *Bs = stage_buf(ks) + TC * BK + (wpos * WTP + lrow) * BK + co;
#pragma unroll
        for (int i = 0; i < FC; ++i)
            A[i] = lds_read16(As + i * 16 * BK);
#pragma unroll
        for (int j = 0; j < FP; ++j)
            B[j] = lds_read16(Bs + j * 16 * BK);
    };
    // MFMAs of one step; NEWER: fragment reads issued after A and B's, which
    // may stay in flight
    auto mfma = [&](auto NEWER, v4i (&A)[FC], v4i (&B)[FP]) {
        lds_wait<decltype(NEWER)::value>();
        lds_settled(A);
        lds_settled(B);
        if constexpr (FLIP) {
#pragma unroll
            for (int j = 0; j < FP; ++j)
                B[j] ^= v4i{(int)0x80808080, (int)0x80808080, (int)0x80808080, (int)0x80808080};
        }
#pragma unroll
        for (int i = 0; i < FC; ++i)
#pragma unroll
            for (int j = 0; j < FP; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[i], B[j], acc[i][j], 0, 0, 0);
    };

    if constexpr (SHORT) {
        // every stage in flight at once; stage k is read as soon as it (and
        // the stages before it) have landed in every wave
        set_tap();
#pragma unroll
        for (int s = 0; s < NS; ++s)
            issue(s);
        auto step = [&](auto S) __attribute__((always_inline)) {
            constexpr int k = decltype(S)::value;
            if constexpr (k < NS) {
                stage_barrier<LPS *(NS - 1 - k)>();
                if constexpr (k == 0)
                    add_bconst<TC, TP, WC, WP, true>(acc, recs);   // the records landed with stage 0
                if (k < nk) {
                    read_frags(k, fa[0], fb[0]);
                    mfma(std::integral_constant<int, 0>{}, fa[0], fb[0]);
                }
            }
        };
        step(std::integral_constant<int, 0>{});
        step(std::integral_constant<int, 1>{});
        step(std::integral_constant<int, 2>{});
        step(std::integral_constant<int, 3>{});
        static_assert(NS <= 4, "short form holds at most four K-steps");
        __syncthreads();
        store_tile<TC, TP, WC, WP, LDS_BYTES, FUSE>(a, acc, lds, c0, p0, recs);
    } else {
        // ---- pipeline -----------------------------------------------------
        // Per group, NSG - 1 stages of loads in flight; the fragments of its
        // stage k + 1 are read from LDS while the MFMAs of its stage k run.
        // The barrier of step k certifies that stage k + 1 of each group has
        // landed everywhere and that every wave is done with step k - 1, so
        // the group's buffer of local stage k - 1 takes stage k + NSG - 1.
        // group grp starts at K-step grp; both groups run the same number of
        // local steps (a step past the end reads zeros), so every barrier
        // is reached by every wave
        if (SPLIT)
            start_at(kbeg);
        set_tap();
        for (int q = 0; q < grp; ++q)
            advance();
        const int nkl = (nk + KS - 1) / KS;
#pragma unroll
        for (int s = 0; s < NSG - 1; ++s)
            issue(s);
        stage_barrier<LPS *(NSG - 2)>();
        if (grp == 0 && part == 0)
            add_bconst<TC, TP, WC, WP, true>(acc, recs);   // the records landed with stage 0
        read_frags(0, fa[0], fb[0]);
        constexpr std::integral_constant<int, FC + FP> kNext{};
        int k = 0;
        for (; k + 2 <= nkl; k += 2) {
            stage_barrier<LPS *(NSG - 3)>();
            issue(k + NSG - 1);
            read_frags(k + 1, fa[1], fb[1]);
            mfma(kNext, fa[0], fb[0]);
            stage_barrier<LPS *(NSG - 3)>();
            issue(k + NSG);
            read_frags(k + 2, fa[0], fb[0]);
            mfma(kNext, fa[1], fb[1]);
        }
        if (k < nkl)
            mfma(std::integral_constant<int, 0>{}, fa[0], fb[0]);
        // with an even step count the reads of step nk (past the last one)
        // are still in flight: retire them before their registers are
        // reused (the compiler does not know they are pending); the
        // fragments stay live up to the wait, so that no instruction the
        // compiler schedules before it can be given their registers
        lds_wait<0>();
        lds_settled(fa[0]);
        lds_settled(fb[0]);
        wait_vmcnt<0>();                   // the trailing out-of-range loads also write LDS
        __syncthreads();
        if constexpr (SPLIT) {
            // Each unit stores its partial sums (int32, in the accumulator
            // layout) and counts itself in the tile's counter; the unit that
            // arrives last adds the other parts to its own and runs the
            // epilogue, then resets the counter to 0 for the next launch.
            // Integer addition is exact, so the order of the parts does not
            // matter.  The parts of a tile may run on different XCDs, whose
            // L2s are not coherent with each other: the partial sums are
            // stored and loaded with agent-scope coherence (sc1: written
            // through to, and read from, the device's coherence point, as the
            // relaxed agent-scope atomic loads and stores of this target are),
            // and the stores are complete (vmcnt 0) before the counter is
            // incremented.  No cache-wide write-back or invalidate is needed.
            constexpr int kAgentScope = 16;   // cache policy bit sc1
            constexpr int SLOT = NW * FC * FP * 64 * 16;   // bytes of one unit's partial tile
            __shared__ int arrived;
            {
                const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
                    (void *)((char *)a.part + (size_t)unit * SLOT), (short)0, SLOT, kBufFlags);
#pragma unroll
                for (int i = 0; i < FC; ++i)
#pragma unroll
                    for (int j = 0; j < FP; ++j)
                        __builtin_amdgcn_raw_buffer_store_b128(acc[i][j], rp,
                                                               (((wave * FC + i) * FP + j) * 64 + lane) * 16, 0,
                                                               kAgentScope);
            }
            wait_vmcnt<0>();
            __syncthreads();
            if (tid == 0)
                arrived = __hip_atomic_fetch_add(a.cnt + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __syncthreads();
            if (arrived != S - 1)
                return;
            if (tid == 0)
                __hip_atomic_store(a.cnt + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            // the other parts' partial tiles, QB of them loaded at once so
            // that their memory latencies overlap (QB bounded by registers)
            constexpr int QB = FC * FP >= 16 ? 1 : 16 / (FC * FP);
            for (int q0 = 0; q0 < S; q0 += QB) {
                v4i t[QB][FC][FP];
#pragma unroll
                for (int u = 0; u < QB; ++u) {
                    const int q = q0 + u;
                    if (q < S && q != part) {
                        const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
                            (void *)((char *)a.part + ((size_t)tile * S + q) * SLOT), (short)0, SLOT, kBufFlags);
#pragma unroll
                        for (int i = 0; i < FC; ++i)
#pragma unroll
                            for (int j = 0; j < FP; ++j)
                                t[u][i][j] = __builtin_amdgcn_raw_buffer_load_b128(
                                    rq, (((wave * FC + i) * FP + j) * 64 + lane) * 16, 0, kAgentScope);
                    }
                }
#pragma unroll
                for (int u = 0; u < QB; ++u) {
                    const int q = q0 + u;
                    if (q < S && q != part) {
#pragma unroll
                        for (int i = 0; i < FC; ++i)
#pragma unroll
                            for (int j = 0; j < FP; ++j)
                                acc[i][j] += t[u][i][j];
                    }
                }
            }
        }
        if constexpr (KS > 1) {
            // the second group's partial sums, through LDS, into the first's
            v4i *part = (v4i *)lds;
            if (grp == 1) {
#pragma unroll
                for (int i = 0; i < FC; ++i)
#pragma unroll
                    for (int j = 0; j < FP; ++j)
                        part[((wave * FC + i) * FP + j) * 64 + lane] = acc[i][j];
            }
            __syncthreads();
            if (grp == 1)
                return;   // the barriers below count only the first group
#pragma unroll
            for (int i = 0; i < FC; ++i)
#pragma unroll
                for (int j = 0; j < FP; ++j)
                    acc[i][j] += part[((wave * FC + i) * FP + j) * 64 + lane];
            __syncthreads();   // every partial read before the staging overwrites them
        }
        store_tile<TC, TP, WC, WP, LDS_BYTES, FUSE>(a, acc, lds, c0, p0, recs);
    }
}

// DmaTile -> tile, wave grid, ring stages, short form, K-step groups.
struct DmaCfg {
    int tc, tp, wc, wp, ns;
    bool sh;
    int ks = 1;
};
inline constexpr DmaCfg kDmaCfg[DMA_COUNT] = {
    {128, 128, 2, 2, 4, false}, {128, 128, 2, 2, 8, false}, {128, 64, 2, 2, 4, false},
    {64, 128, 2, 2, 4, false},  {64, 64, 2, 2, 4, false},   {256, 128, 4, 2, 4, false},
    {128, 256, 2, 4, 4, false}, {128, 64, 2, 2, 8, false},  {256, 128, 2, 2, 4, false},
    {128, 256, 2, 2, 4, false}, {128, 128, 1, 2, 8, false}, {128, 128, 2, 1, 8, false},
    {64, 64, 2, 2, 8, false},   {64, 128, 2, 2, 8, false},  {64, 64, 2, 2, 16, false},
    {64, 128, 2, 2, 1, true},   {64, 64, 2, 2, 1, true},    {128, 128, 2, 2, 1, true},
    {128, 64, 2, 2, 1, true},   {64, 128, 2, 2, 2, true},   {128, 128, 2, 2, 2, true},
    {64, 64, 2, 2, 2, true},    {128, 64, 2, 2, 2, true},   {64, 128, 2, 2, 4, true},
    {128, 128, 2, 2, 4, true},  {64, 64, 2, 2, 4, true},    {128, 64, 2, 2, 8, false, 2},
    {64, 64, 2, 2, 8, false, 2}, {128, 128, 2, 2, 8, false, 2},
};

// Configurations that have an instantiation with the fused residual add.
constexpr bool dma_fuse_cfg(int t)
{
    return kDmaCfg[t].tc / kDmaCfg[t].wc * (kDmaCfg[t].tp / kDmaCfg[t].wp) <= kFuseMaxWaveTile;
}

// Launch of a tile configuration's fused-add instantiation (a.res set,
// a.staged, no split reduction); hipErrorInvalidValue where there is none.
hipError_t launch_conv_dma_fused(const ConvArgs &a, int tile, hipStream_t st);

}  // namespace qnn
