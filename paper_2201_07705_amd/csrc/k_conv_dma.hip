// Implicit-GEMM convolution with an LDS-DMA pipeline (gfx950).
//
// Same GEMM as conv_bf16 (C[M][N] = A[M][K] * B[N][K]^T over the merged
// frames of several models, bf16 MFMA, fp32 accumulation, fused epilogue),
// organised for latency tolerance: each depth step of 32 is fetched by
// global_load_lds_dwordx4 straight into one of STAGES LDS buffers, so
// STAGES-1 steps are in flight while the MFMAs consume the oldest one and
// no registers hold staged data. Each stage lives in its own __shared__
// array (the compiler then tracks which buffer an outstanding LDS-DMA
// writes and waits only where a read could alias it); the waits on the
// loads are explicit vmcnt counts, and workgroup syncs are bare s_barrier
// (a fenced barrier would drain every outstanding load).
//
// An LDS-DMA instruction writes 64 consecutive 16-byte slots per wave, so
// the layout is chosen through the addresses: slot p of a stage holds row
// p/4, 16-byte chunk (p%4) ^ ((row/2)%4) of that row. The swizzle puts the
// 16-byte fragment reads of 8 consecutive rows at the same chunk onto
// distinct banks.
//
// Requirements: Cin a multiple of 32 (a step is one filter tap and 32
// channels), input pixel stride a multiple of 8, depth per split a
// multiple of 32.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "conv_epi.h"
#include "kargs.h"
#include "kernels.h"

namespace gemel {

namespace {

typedef __attribute__((address_space(3))) unsigned char lds_u8;

// Calls f(std::integral_constant<int, i>) for i = 0 .. I-1 with a
// compile-time i, so that register arrays are indexed statically.
template <int I>
struct StaticFor {
    template <typename F>
    __device__ __forceinline__ static void run(F &&f) {
        StaticFor<I - 1>::run(f);
        f(std::integral_constant<int, I - 1>{});
    }
};
template <>
struct StaticFor<0> {
    template <typename F>
    __device__ __forceinline__ static void run(F &&) {}
};

// vmcnt-only wait: expcnt and lgkmcnt left at their maxima (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Waits until at most n steps of PER vm operations each are in flight, for a
// uniform n in 0 .. MAXN-1 (s_waitcnt takes an immediate, so one branch per
// count).
template <int PER, int MAXN>
__device__ __forceinline__ void wait_steps(int n) {
    StaticFor<MAXN>::run([&](auto c) __attribute__((always_inline)) {
        constexpr int i = decltype(c)::value;
        if (n == i) wait_vm<i * PER>();
    });
}

// lgkmcnt(0) only: vmcnt and expcnt left at their maxima (gfx9 encoding).
__device__ __forceinline__ void wait_lgkm0() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));
}

}  // namespace

// MODE 1: the 2x2 stride-2 max pool fused (out_mode OUT_NHWC_POOL2);
// MODE 2: segments of different spatial sizes (ConvArgs::hetero). Separate
// instantiations, so that the plain kernels keep their code and registers.
// Waves per SIMD the kernel is compiled for: two where the LDS of two
// workgroups fits one CU and a workgroup has at most 4 waves (the register
// budget then allows both), else one.
template <int BM, int BN, int WM, int WN, int STAGES, int BK>
constexpr int dma_min_waves() {
    return WM * WN <= 4 && 2 * STAGES * (BM + BN) * BK * 2 <= 160 * 1024 ? 2 : 1;
}

template <int BM, int BN, int WM, int WN, int STAGES, int BK, int MODE>
__global__ __launch_bounds__(64 * WM *WN, (dma_min_waves<BM, BN, WM, WN, STAGES, BK>())) void conv_dma_kernel(
    const ConvArgs a) {
    constexpr int NW = WM * WN, NT = 64 * NW;
    static_assert(BK == 32 || BK == 64, "step depth");
    constexpr int CPR = BK / 8;                                 // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;                               // rows per DMA instruction
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 16, FN = TN / 16;
    constexpr int A_SLOTS = BM * CPR, B_SLOTS = BN * CPR;      // 16-byte slots per stage
    constexpr int AI = A_SLOTS / NT, BI = B_SLOTS / NT;        // DMA instructions per thread
    static_assert(AI * NT == A_SLOTS && BI * NT == B_SLOTS && AI >= 1 && BI >= 1, "tile/threads");
    constexpr int STAGE_BYTES = (A_SLOTS + B_SLOTS) * 16;
    constexpr int EPI_LD = TN + 4;                              // fp32 row pitch of a wave's staging
    static_assert(STAGES >= 2 && STAGES <= 4, "stages");
    static_assert(TN % 8 == 0 && 64 % (TN / 8) == 0 && TN <= 512,
                  "every epilogue item of a lane is the same 8-channel chunk of its wave's columns");
    constexpr int PER_STEP = AI + BI;                           // vm ops per thread per step
    __shared__ __attribute__((aligned(1024))) unsigned char st0[STAGE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char st1[STAGE_BYTES];
    __shared__ __attribute__((aligned(1024))) unsigned char st2[STAGES > 2 ? STAGE_BYTES : 16];
    __shared__ __attribute__((aligned(1024))) unsigned char st3[STAGES > 3 ? STAGE_BYTES : 16];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / WN, wn = wave - (wave / WN) * WN;
    const int tiles_n = (a.N + BN - 1) / BN;
    const int G = gridDim.x;
    const int t = (G & 7) == 0 ? (int)(blockIdx.x & 7) * (G >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
    // the tile's rows [m_lo, min(m_lo + BM, m_end)), column tile tn and
    // weights. Grouped launches tile every segment on its own (a tile never
    // straddles two segments' weights; seg[s].t_start is its first tile).
    // Segment fields are gathered with selects over a static walk of the
    // table: indexing the argument block with a computed segment number
    // makes the compiler copy the whole block to scratch memory.
    int m_lo, m_end = a.M, tn, tiles;
    const void *wseg = a.w;
    if (a.grouped) {
        int ts = 0, ms = 0;
        bool past = false;
        for (int i = 0; i < a.nseg; ++i) {
            const int ti = a.seg[i].t_start, mi = a.seg[i].m_start;
            const void *wi = a.seg[i].w;
            const bool hit = t >= ti;
            if (!hit && !past) m_end = mi;   // the next segment's first row
            past = past || !hit;
            ts = hit ? ti : ts;
            ms = hit ? mi : ms;
            wseg = hit ? wi : wseg;
            tiles = ti + ((i + 1 < a.nseg ? a.seg[i + 1].m_start : a.M) - mi + BM - 1) / BM * tiles_n;
        }
        const int local = t - ts, tml = local / tiles_n;
        tn = local - tml * tiles_n;
        m_lo = ms + tml * BM;
    } else {
        tiles = ((a.M + BM - 1) / BM) * tiles_n;
        const int tm = t / tiles_n;
        tn = t - tm * tiles_n;
        m_lo = tm * BM;
    }
    if (t >= tiles) return;
    const int k_begin = blockIdx.y * a.k_per_split;
    const int k_end = min(a.K, k_begin + a.k_per_split);
    const int HWo = a.Ho * a.Wo;
    const int H = a.H, W = a.W, in_cs = a.in_cs, N = a.N, K = a.K, Cin = a.Cin, kw = a.kw;
    const size_t frame_elems = (size_t)H * W * in_cs;
    const u16 *const zp = (const u16 *)a.zero;
    // segment of the tile's first and last row (wave-uniform, scalar loads):
    // rows of a tile inside one segment take its fields as uniform values;
    // per-row lookups only for a tile that straddles segments
    const int m_first = m_lo, m_last = min(m_end, m_first + BM) - 1;
    int s_first = 0, s_last = 0;
    for (int i = 1; i < a.nseg; ++i) {
        s_first += m_first >= a.seg[i].m_start ? 1 : 0;
        s_last += m_last >= a.seg[i].m_start ? 1 : 0;
    }
    const bool one_seg = s_first == s_last;
    const RowSeg useg = uni_seg(a, s_first);

    // ---- DMA assignment: instruction i of this thread fills slot
    // (i*NW + wave)*64 + lane: row (i*NW + wave)*RPI + lane/CPR; the slot's
    // chunk position lane%CPR holds logical chunk (lane%CPR) ^ sw(row) ----
    auto sw = [](int row) __attribute__((always_inline)) { return (row >> 1) & (CPR - 1); };
    // with the 2x2 max pool fused, rows run over the output in window
    // order: row 4g + 2dy + dx is pixel (2hp + dy, 2wp + dx) of pooled pixel g
    constexpr bool pool2 = MODE == 1;
    // with segments of different sizes, each row takes its segment's sizes
    // (and its frame within the segment from the rows before it)
    constexpr bool hetero = MODE == 2;
    const int Wp = a.Wo >> 1, HWp = HWo >> 2;
    const u16 *abase[AI];
    int ahi[AI], awi[AI], acq[AI];
    int aH[hetero ? AI : 1], aW[hetero ? AI : 1];
#pragma unroll
    for (int i = 0; i < AI; ++i) {
        const int rl = (i * NW + wave) * RPI + lane / CPR;
        acq[i] = (lane % CPR) ^ sw(rl);
        const int gm = m_lo + rl;
        abase[i] = zp;
        ahi[i] = -(1 << 28);
        awi[i] = 0;
        if constexpr (hetero) {
            aH[i] = 0;
            aW[i] = 0;
        }
        if (hetero && gm < m_end) {
            // the row's segment sizes: uniform in a tile inside one segment,
            // else gathered with scalar loads and selects like row_seg
            int sH = a.seg[s_first].H, sW = a.seg[s_first].W, sHo = a.seg[s_first].Ho, sWo = a.seg[s_first].Wo;
            if (!one_seg)
                for (int k = 1; k < a.nseg; ++k) {
                    const bool hit = gm >= a.seg[k].m_start;
                    sH = hit ? a.seg[k].H : sH;
                    sW = hit ? a.seg[k].W : sW;
                    sHo = hit ? a.seg[k].Ho : sHo;
                    sWo = hit ? a.seg[k].Wo : sWo;
                }
            const RowSeg sg = one_seg ? useg : row_seg(a, gm);
            const int local = gm - sg.m_start, hw = sHo * sWo;
            const int fl = local / hw, pix = local - fl * hw, ho = pix / sWo;
            abase[i] = (const u16 *)sg.in + (size_t)fl * sH * sW * in_cs;
            ahi[i] = ho * a.stride - a.pad;
            awi[i] = (pix - ho * sWo) * a.stride - a.pad;
            aH[i] = sH;
            aW[i] = sW;
        } else if (gm < m_end) {
            int fr, ho, wo;
            // quotients by multiply-high (the launcher's magic numbers): a
            // per-lane integer division costs dozens of instructions
            auto qdiv = [&](int n, int q) __attribute__((always_inline)) {
                return (int)((__umulhi((uint32_t)n, a.dv_m[q]) + (uint32_t)n) >> a.dv_l[q]);
            };
            if constexpr (pool2) {
                const int g = gm >> 2;
                fr = qdiv(g, 0);
                const int pp = g - fr * HWp, hp = qdiv(pp, 1);
                ho = 2 * hp + ((gm >> 1) & 1);
                wo = 2 * (pp - hp * Wp) + (gm & 1);
            } else {
                fr = qdiv(gm, 0);
                const int pix = gm - fr * HWo;
                ho = qdiv(pix, 1);
                wo = pix - ho * a.Wo;
            }
            const RowSeg sg = one_seg ? useg : row_seg(a, gm);
            abase[i] = (const u16 *)sg.in + (size_t)(fr - sg.f_start) * frame_elems;
            ahi[i] = ho * a.stride - a.pad;
            awi[i] = wo * a.stride - a.pad;
        }
    }
    // weight rows beyond N read row 0 instead (their columns are never stored)
    const u16 *bbase[BI];
#pragma unroll
    for (int i = 0; i < BI; ++i) {
        const int rl = (i * NW + wave) * RPI + lane / CPR;
        const int gn = tn * BN + rl;
        bbase[i] = (const u16 *)wseg + (size_t)(gn < N ? gn : 0) * K + ((lane % CPR) ^ sw(rl)) * 8;
    }
    // loader position (uniform): next step's tap (lr, ls) and channel base lc
    int kb = k_begin, lc, lr, ls;
    {
        const int rs = k_begin / Cin;
        lc = k_begin - rs * Cin;
        lr = rs / kw;
        ls = rs - lr * kw;
    }
    // each row's source for the current tap, the lane's chunk included: the
    // pixel, or the zero page where the tap falls outside the image (or the
    // row beyond M). Recomputed when the tap changes; a depth step only adds
    // the uniform channel offset (the zero page spans any row's channels).
    const u16 *arow[AI];
    auto set_tap = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < AI; ++i) {
            const int hi = ahi[i] + lr, wi = awi[i] + ls;
            const int Hr = hetero ? aH[hetero ? i : 0] : H, Wr = hetero ? aW[hetero ? i : 0] : W;
            const bool ok = (unsigned)hi < (unsigned)Hr && (unsigned)wi < (unsigned)Wr;
            arow[i] = (ok ? abase[i] + (size_t)(hi * Wr + wi) * in_cs : zp) + acq[i] * 8;
        }
    };
    set_tap();
    auto issue = [&](unsigned char *stage) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < AI; ++i)
            __builtin_amdgcn_global_load_lds((const void *)(arow[i] + lc), (lds_u8 *)(stage + (i * NW + wave) * 1024),
                                             16, 0, 0);
#pragma unroll
        for (int i = 0; i < BI; ++i)
            __builtin_amdgcn_global_load_lds((const void *)(bbase[i] + kb),
                                             (lds_u8 *)(stage + A_SLOTS * 16 + (i * NW + wave) * 1024), 16, 0, 0);
        kb += BK;
        lc += BK;
        if (lc == Cin) {
            lc = 0;
            if (++ls == kw) { ls = 0; ++lr; }
            set_tap();
        }
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // fragment read offsets inside a stage (swizzled slots): a fragment row
    // is wave-tile row 16*i + lane%16 (a multiple of 16 plus lane%16), so
    // its swizzle depends on the lane only
    const int g = lane >> 4;
    const int swl = sw(lane & 15);
    int aoff[FM], boff[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) aoff[i] = (wm * TM + i * 16 + (lane & 15)) * CPR * 16;
#pragma unroll
    for (int j = 0; j < FN; ++j) boff[j] = A_SLOTS * 16 + (wn * TN + j * 16 + (lane & 15)) * CPR * 16;
    // fragments of one depth step in registers: H halves of 32
    constexpr int NH = BK / 32;
    typedef bf16x8 FragA[NH][FM];
    typedef bf16x8 FragB[NH][FN];
    auto read_frags = [&](const unsigned char *stage, FragA &fa, FragB &fb) __attribute__((always_inline)) {
#pragma unroll
        for (int h = 0; h < NH; ++h) {
            const int pos = ((h * 4 + g) ^ swl) * 16;
#pragma unroll
            for (int j = 0; j < FN; ++j) fb[h][j] = *(const bf16x8 *)(stage + boff[j] + pos);
#pragma unroll
            for (int i = 0; i < FM; ++i) fa[h][i] = *(const bf16x8 *)(stage + aoff[i] + pos);
        }
    };
    auto mfmas = [&](const FragA &fa, const FragB &fb) __attribute__((always_inline)) {
#pragma unroll
        for (int h = 0; h < NH; ++h)
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[h][i], fb[h][j], acc[i][j], 0, 0, 0);
    };
    auto compute = [&](const unsigned char *stage) __attribute__((always_inline)) {
        FragA fa;
        FragB fb;
        read_frags(stage, fa, fb);
        mfmas(fa, fb);
    };

    // epilogue constants of this lane's 8 channels (every segment shares
    // one scale/shift pair), fetched ahead of the depth loop
    const int my_gn = tn * BN + wn * TN + (lane % (TN / 8)) * 8;
    f32x4 sc0 = {1.f, 1.f, 1.f, 1.f}, sc1 = sc0, sh0 = {0.f, 0.f, 0.f, 0.f}, sh1 = sh0;
    if (a.k_splits <= 1 && my_gn < N) {
        const float *scl = useg.scale + my_gn, *shl = useg.shift + my_gn;
        sc0 = *(const f32x4 *)scl;
        sc1 = *(const f32x4 *)(scl + 4);
        sh0 = *(const f32x4 *)shl;
        sh1 = *(const f32x4 *)(shl + 4);
    }

    const int nk = (k_end - k_begin) / BK;
    unsigned char *const stg[4] = {st0, st1, st2, st3};
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        if (s < nk) issue(stg[s]);

    // register double-buffering needs a second fragment set: only where it
    // fits beside the accumulators (512-thread workgroups have 256
    // registers per lane)
    constexpr bool PIPE = STAGES == 4 && (NT <= 256 || FM * FN <= 16);
    if constexpr (PIPE) {
        // Fragments double-buffered in registers: iteration it reads step
        // it+1's fragments from LDS, then issues step it's MFMAs from the
        // registers filled one iteration earlier, so the LDS reads overlap
        // the MFMAs. The DMA issued in iteration it refills the buffer of
        // step it-1, whose fragments every wave read before this
        // iteration's barrier.
        FragA fa[2];
        FragB fb[2];
        if (nk > 0) {
            // steps 0 .. min(nk, STAGES-1)-1 were issued; step 0 must land
            wait_steps<PER_STEP, STAGES - 1>(min(nk - 1, STAGES - 2));
            __builtin_amdgcn_s_barrier();
            read_frags(stg[0], fa[0], fb[0]);
        }
        int base = 0;
        // steady state: every iteration of the group waits, issues the DMA
        // STAGES-1 steps ahead and reads the next fragments (no branches, so
        // the compiler's wait placement sees one path)
        for (; base + 2 * STAGES - 1 <= nk; base += STAGES) {
#pragma unroll
            for (int s = 0; s < STAGES; ++s) {
                wait_vm<(STAGES - 3) * PER_STEP>();
                __builtin_amdgcn_s_barrier();
                issue(stg[(s + STAGES - 1) % STAGES]);
                wait_lgkm0();
                read_frags(stg[(s + 1) % STAGES], fa[(s + 1) & 1], fb[(s + 1) & 1]);
                mfmas(fa[s & 1], fb[s & 1]);
            }
        }
        // the last groups, with the bounds checks
        for (; base < nk; base += STAGES) {
#pragma unroll
            for (int s = 0; s < STAGES; ++s) {
                const int it = base + s;
                if (it < nk) {
                    if (it + 1 < nk) {
                        // step it+1 must have landed; the newer steps issued
                        // (up to it+STAGES-2, none beyond nk-1) may fly
                        wait_steps<PER_STEP, STAGES - 2>(min(nk - it - 2, STAGES - 3));
                        __builtin_amdgcn_s_barrier();
                        if (it + STAGES - 1 < nk) issue(stg[(s + STAGES - 1) % STAGES]);
                        // the fragments read one iteration ago (the operands
                        // of the MFMAs below) have long arrived: waiting for
                        // them here, before the next reads are issued, keeps
                        // the compiler from waiting for those after them
                        wait_lgkm0();
                        read_frags(stg[(s + 1) % STAGES], fa[(s + 1) & 1], fb[(s + 1) & 1]);
                    } else {
                        wait_lgkm0();   // both paths reach the MFMAs with no read pending on their operands
                    }
                    mfmas(fa[s & 1], fb[s & 1]);
                }
            }
        }
    } else {
        // main loop, unrolled by STAGES so that every buffer index is static
        for (int base = 0; base < nk; base += STAGES) {
#pragma unroll
            for (int s = 0; s < STAGES; ++s) {
                const int it = base + s;
                if (it < nk) {
                    // step it must have landed; the newer steps issued (up
                    // to it+STAGES-2, none beyond nk-1) may still fly
                    wait_steps<PER_STEP, STAGES - 1>(min(nk - it - 1, STAGES - 2));
                    __builtin_amdgcn_s_barrier();
                    if (it + STAGES - 1 < nk) issue(stg[(s + STAGES - 1) % STAGES]);
                    compute(stg[s]);
                }
            }
        }
    }

    // ---- epilogue: each wave stages PG passes of 16 rows of its tile at a
    // time in its share of the stage buffers. Only the accumulator dump is
    // unrolled per pass; the store code exists once (a kernel larger than
    // the instruction cache pays for its cold misses on every launch).
    constexpr int WPS = (NW + STAGES - 1) / STAGES;             // waves per stage buffer
    constexpr int PASS_FLOATS = 16 * EPI_LD;
    constexpr int GMAX = STAGE_BYTES / (WPS * PASS_FLOATS * 4);
    static_assert(GMAX >= 1, "a 16-row pass must fit a wave's share of a stage buffer");
    constexpr int PG = (GMAX >= 4 && FM % 4 == 0) ? 4 : (GMAX >= 2 && FM % 2 == 0) ? 2 : 1;
    constexpr int NGRP = FM / PG;
    constexpr int CHW = TN / 8;                                 // 8-channel chunks per wave row
    constexpr int ITEMS = PG * 16 * CHW / 64;                    // (row, chunk) items per lane per group
    static_assert(ITEMS * 64 == PG * 16 * CHW, "items per lane");
    wait_vm<0>();
    __builtin_amdgcn_s_barrier();
    const int sidx = wave % STAGES;
    unsigned char *const sbuf = sidx == 0 ? st0 : sidx == 1 ? st1 : sidx == 2 ? st2 : st3;
    float *const ew = (float *)(sbuf + (wave / STAGES) * PG * PASS_FLOATS * 4);
    const int out_cs = a.out_cs;
    const __amdgpu_buffer_rsrc_t pr = partial_rsrc(a.partial, (uint32_t)a.k_splits * a.M * N * 4u);
    const int ch = lane % CHW;                                  // this lane's chunk in every item
    const int gn = my_gn;
    const bool col_ok = gn < N;
    const bool pre_res = a.has_res && a.out_mode == OUT_NHWC && a.k_splits <= 1;
    const int ekind = epi_kind(a.act, a.has_res, a.res_mode, a.slope);
    const float s8[8] = {sc0[0], sc0[1], sc0[2], sc0[3], sc1[0], sc1[1], sc1[2], sc1[3]};
    const float h8[8] = {sh0[0], sh0[1], sh0[2], sh0[3], sh1[0], sh1[1], sh1[2], sh1[3]};
#pragma nounroll
    for (int grp = 0; grp < NGRP; ++grp) {
        const int row0 = m_lo + wm * TM + grp * PG * 16;
        // residuals of the group's items, loaded ahead of the staging
        u32x4 rv[ITEMS];
#pragma unroll
        for (int u = 0; u < ITEMS; ++u) {
            rv[u] = u32x4{0u, 0u, 0u, 0u};
            const int gm = row0 + (lane + u * 64) / CHW;
            if (pre_res && col_ok && gm < m_end) {
                const RowSeg sg = one_seg ? useg : row_seg(a, gm);
                rv[u] = *(const u32x4 *)((const u16 *)sg.res + (size_t)(gm - sg.m_start) * out_cs + gn);
            }
        }
        StaticFor<NGRP>::run([&](auto gc) __attribute__((always_inline)) {
            constexpr int gi = decltype(gc)::value;
            if (grp == gi) {
                StaticFor<PG>::run([&](auto pc) __attribute__((always_inline)) {
                    constexpr int pp = decltype(pc)::value;
                    constexpr int i = gi * PG + pp;
#pragma unroll
                    for (int j = 0; j < FN; ++j)
#pragma unroll
                        for (int v = 0; v < 4; ++v)
                            ew[(pp * 16 + (lane >> 4) * 4 + v) * EPI_LD + j * 16 + (lane & 15)] = acc[i][j][v];
                });
            }
        });
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // the residual loads (and the previous group's stores) complete
        // here, once: with none pending, the compiler needs no wait between
        // the stores below (vmcnt counts loads and stores together, so a
        // wait for a load would also wait for every earlier store). Without
        // a residual nothing is waited for: the epilogue kinds without one
        // never read the residual registers.
        if (pre_res) wait_vm<0>();
        if constexpr (pool2) {
            // pooled items (window, chunk): the window's 4 staged rows through
            // the epilogue, each rounded to bf16 as stored unfused, then their
            // max in window order (what the separate pool computes)
            constexpr int NPI = PG * 4 * CHW;
#pragma unroll
            for (int u = 0; u < (NPI + 63) / 64; ++u) {
                const int idx = lane + u * 64;
                const int pr = idx / CHW;
                const int gm = row0 + 4 * pr;
                if (idx >= NPI || !col_ok || gm >= m_end) continue;
                float mx[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) mx[j] = -INFINITY;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float *src = ew + (4 * pr + q) * EPI_LD + ch * 8;
                    const float4 v0 = *(const float4 *)src, v1 = *(const float4 *)(src + 4);
                    const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
                    float y[8];
                    epi8_f32(v, s8, h8, u32x4{0u, 0u, 0u, 0u}, ekind, 0, 0, a.act, a.slope, y);
#pragma unroll
                    for (int j = 0; j < 8; ++j) mx[j] = fmaxf(mx[j], bf2f(f2bf(y[j])));
                }
                const RowSeg sg = one_seg ? useg : row_seg(a, gm);
                *(u32x4 *)((u16 *)sg.out + (size_t)((gm - sg.m_start) >> 2) * out_cs + gn) = pack8_bf16(mx);
            }
        } else {
#pragma unroll
        for (int u = 0; u < ITEMS; ++u) {
            const int rl = (lane + u * 64) / CHW;
            const int gm = row0 + rl;
            if (!col_ok || gm >= m_end) continue;
            const float *src = ew + rl * EPI_LD + ch * 8;
            const float4 v0 = *(const float4 *)src, v1 = *(const float4 *)(src + 4);
            if (a.k_splits > 1) {
                const uint32_t off = (uint32_t)((((int)blockIdx.y * a.M + gm) * N + gn) * 4u);
                store_partial4(pr, off, v0);
                store_partial4(pr, off + 16, v1);
                continue;
            }
            const float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
            const RowSeg sg = one_seg ? useg : row_seg(a, gm);
            const int lr_ = gm - sg.m_start;
            if (a.out_mode == OUT_NHWC) {
                const size_t off = (size_t)lr_ * out_cs + gn;
                float y[8];
                epi8_f32(v, s8, h8, rv[u], ekind, a.has_res, a.res_mode, a.act, a.slope, y);
                store8_bf16((u16 *)sg.out + off, 0, y, a.out_pair);
            } else {
                const int f = lr_ / HWo, pix = lr_ - (lr_ / HWo) * HWo;
                const u16 *resp = (const u16 *)sg.res;
                for (int q = 0; q < 8; ++q) {
                    const int c = gn + q;
                    if (c >= a.cout) break;
                    const float r = a.has_res ? bf2f(resp[(size_t)lr_ * out_cs + c]) : 0.f;
                    ((float *)sg.out)[((size_t)f * a.cout + c) * HWo + pix] =
                        epi(v[q] * s8[q] + h8[q], r, a.has_res, a.res_mode, a.act, a.slope);
                }
            }
        }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (a.k_splits > 1 && a.counters)
        splitk_fixup<64 * WM * WN>(a, t, m_lo, min(BM, m_end - m_lo), tn * BN, BN, (int *)st2);
    if (a.pf) {
        // the next conv's weights into L2 and the memory-side cache: the
        // workgroups share them out in 1 KB wave loads into a stage buffer
        // no longer read (after every wave's epilogue)
        __builtin_amdgcn_s_barrier();
        const uint64_t stride = (uint64_t)gridDim.x * gridDim.y * NW * 1024u;
        for (uint64_t off = (((uint64_t)blockIdx.y * gridDim.x + blockIdx.x) * NW + wave) * 1024u + lane * 16u;
             off + 16u <= a.pf_bytes; off += stride)
            __builtin_amdgcn_global_load_lds((const void *)((const char *)a.pf + off),
                                             (lds_u8 *)(st0 + wave * 1024), 16, 0, 0);
        wait_vm<0>();
    }
}

bool conv_dma_supported(const ConvArgs &a) {
    // a row outside the image reads the zero page at its channel offset
    return a.Cin % 32 == 0 && a.in_cs % 8 == 0 && a.K % 32 == 0 && a.k_per_split % 32 == 0 && a.zero &&
           (a.uni_affine || a.grouped) && (long)a.in_cs * 2 + 128 <= GEMEL_ZERO_PAGE_BYTES;
}
bool conv_dma_supported(const ConvArgs &a, int tile) {
    if (!conv_dma_supported(a)) return false;
    if (tile_dma_depth(tile) == 64) return a.Cin % 64 == 0 && a.k_per_split % 64 == 0;
    return true;
}

hipError_t launch_conv_dma(const ConvArgs &a, int tile, const Sink &sk) {
    if (!conv_dma_supported(a, tile) || a.M <= 0 || a.N <= 0 || a.N % 8 || a.nseg < 1 || a.nseg > GEMEL_MAX_SEG)
        return hipErrorInvalidValue;
    if (a.K != a.kh * a.kw * a.Cin || a.out_cs < a.N || a.seg[0].m_start != 0) return hipErrorInvalidValue;
    if (a.k_splits > 1 && !a.partial) return hipErrorInvalidValue;
    // fused 2x2 pool: whole windows, no split-K, no residual
    if (a.out_mode == OUT_NHWC_POOL2 &&
        (a.k_splits > 1 || a.has_res || (a.Ho & 1) || (a.Wo & 1) || a.Ho <= 0 || a.Wo <= 0))
        return hipErrorInvalidValue;
    if (a.k_splits > 1 && (long)a.k_splits * a.M * a.N * 4 > 0x7fffffffL) return hipErrorInvalidValue;
    if ((long)a.k_per_split * a.k_splits < a.K) return hipErrorInvalidValue;
    // bf16 pairs: internal NHWC output, both halves inside the pixel
    if (a.out_pair && (a.out_mode != OUT_NHWC || a.out_pair < a.N || a.out_pair % 8 || a.out_cs < a.out_pair + a.N))
        return hipErrorInvalidValue;
    // mixed sizes: NHWC output, no fused pool; each segment whole frames of
    // its own size, the rows of the segments back to back
    if (a.hetero && a.out_mode != OUT_NHWC) return hipErrorInvalidValue;
    if (a.grouped && a.hetero) return hipErrorInvalidValue;
    for (int i = 0; i < a.nseg; ++i) {
        const ConvSeg &s = a.seg[i];
        if (!s.in || !s.scale || !s.shift) return hipErrorInvalidValue;
        if (a.grouped && (!s.w || (i && s.m_start <= a.seg[i - 1].m_start))) return hipErrorInvalidValue;
        if ((a.k_splits <= 1 || a.counters) && !s.out) return hipErrorInvalidValue;
        if (a.has_res && !s.res) return hipErrorInvalidValue;
        if (!a.hetero) {
            if (s.m_start != s.f_start * a.Ho * a.Wo) return hipErrorInvalidValue;
            continue;
        }
        const long rows = (i + 1 < a.nseg ? a.seg[i + 1].m_start : a.M) - (long)s.m_start;
        if (s.H <= 0 || s.W <= 0 || s.Ho <= 0 || s.Wo <= 0 || rows <= 0 || rows % ((long)s.Ho * s.Wo))
            return hipErrorInvalidValue;
    }
    const int bm = conv_tile_bm(tile), bn = conv_tile_bn(tile);
    if (!bm) return hipErrorInvalidValue;
    // grouped: each segment tiled on its own, from tile seg[s].t_start
    ConvArgs b = a;
    long tiles = 0;
    if (a.grouped) {
        for (int i = 0; i < a.nseg; ++i) {
            const long rows = (i + 1 < a.nseg ? a.seg[i + 1].m_start : a.M) - (long)a.seg[i].m_start;
            b.seg[i].t_start = (int32_t)tiles;
            tiles += (rows + bm - 1) / bm * ((a.N + bn - 1) / bn);
        }
    } else {
        tiles = (long)((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn);
    }
    if (tiles != conv_tiles(a, bm, bn)) return hipErrorInvalidValue;
    const long blocks = tiles >= 8 ? (tiles + 7) / 8 * 8 : tiles;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    // magic numbers of the row decomposition (exact for rows below 2^31:
    // m = floor(2^32 (2^l - d) / d) + 1 with l = ceil(log2 d))
    {
        const bool pool = a.out_mode == OUT_NHWC_POOL2;
        const long d[2] = {pool ? (long)(a.Ho / 2) * (a.Wo / 2) : (long)a.Ho * a.Wo, pool ? a.Wo / 2 : a.Wo};
        for (int q = 0; q < 2; ++q) {
            if (d[q] <= 0) {
                b.dv_m[q] = 1;
                b.dv_l[q] = 0;
                continue;
            }
            int l = 0;
            while ((1L << l) < d[q]) ++l;
            b.dv_m[q] = (uint32_t)(((uint64_t)1 << 32) * (uint64_t)((1L << l) - d[q]) / (uint64_t)d[q] + 1);
            b.dv_l[q] = l;
        }
    }
    dim3 grid((unsigned)blocks, (unsigned)a.k_splits);
    hipError_t e = hipErrorInvalidValue;
    const int mode = a.out_mode == OUT_NHWC_POOL2 ? 1 : a.hetero ? 2 : 0;
#define GEMEL_DMA_CASE(T, BM_, BN_, WM_, WN_, ST_, BK_, NT_)                                                  \
    case T:                                                                                                   \
        e = submit(sk,                                                                                        \
                   mode == 1   ? reinterpret_cast<const void *>(&conv_dma_kernel<BM_, BN_, WM_, WN_, ST_, BK_, 1>) \
                   : mode == 2 ? reinterpret_cast<const void *>(&conv_dma_kernel<BM_, BN_, WM_, WN_, ST_, BK_, 2>) \
                               : reinterpret_cast<const void *>(&conv_dma_kernel<BM_, BN_, WM_, WN_, ST_, BK_, 0>), \
                   grid, dim3(NT_), b);                                                                       \
        break;
    switch (tile) {
        GEMEL_DMA_CASE(TILE_DMA_256x256, 256, 256, 2, 4, 4, 32, 512)
        GEMEL_DMA_CASE(TILE_DMA_256x128, 256, 128, 2, 2, 4, 32, 256)
        GEMEL_DMA_CASE(TILE_DMA_128x128, 128, 128, 2, 2, 4, 32, 256)
        GEMEL_DMA_CASE(TILE_DMA_128x64, 128, 64, 2, 1, 4, 32, 128)
        GEMEL_DMA_CASE(TILE_DMA_64x64, 64, 64, 2, 2, 4, 32, 256)
        GEMEL_DMA_CASE(TILE_DMA64_64x64, 64, 64, 2, 2, 4, 64, 256)
        GEMEL_DMA_CASE(TILE_DMA64_256x256, 256, 256, 2, 4, 2, 64, 512)
        GEMEL_DMA_CASE(TILE_DMA64_256x128, 256, 128, 2, 2, 3, 64, 256)
        GEMEL_DMA_CASE(TILE_DMA64_128x128, 128, 128, 2, 2, 2, 64, 256)
        GEMEL_DMA_CASE(TILE_DMA64_128x64, 128, 64, 2, 1, 3, 64, 128)
        GEMEL_DMA_CASE(TILE_DMA_256x128W8, 256, 128, 4, 2, 4, 32, 512)
        GEMEL_DMA_CASE(TILE_DMA_128x256W8, 128, 256, 2, 4, 4, 32, 512)
        GEMEL_DMA_CASE(TILE_DMA_256x64, 256, 64, 4, 1, 4, 32, 256)
        GEMEL_DMA_CASE(TILE_DMA_64x256, 64, 256, 1, 4, 4, 32, 256)
    default: break;
    }
#undef GEMEL_DMA_CASE
    return e;
}

}  // namespace gemel
