// Merged-batch convolution kernels for gfx950.
//
// conv_bf16: implicit GEMM C[M][N] = A[M][K] * B[N][K]^T on bf16 MFMA
// (v_mfma_f32_16x16x32_bf16, fp32 accumulation).
//   M = frames of every model in the launch x Ho x Wo  (rows of all merged
//       models, concatenated; each model's rows read its own tensor)
//   N = output channels, K = kh * kw * Cin (Cin-fastest, matching KRSC
//       weights and NHWC activations, so every 8-element K chunk is one
//       16-byte load).
// A workgroup of 4 waves computes a BM x BN tile; A (im2col gathered on the
// fly) and B (the single shared weight copy) tiles of depth 64 are
// double-buffered in LDS, so one weight tile is reused by the rows of every
// model that shares the layer. The epilogue stages the fp32 tile through
// LDS and applies per-channel scale/shift (bias and batch norm), the
// residual (before or after the activation) and ReLU / leaky ReLU, then
// writes bf16 NHWC with 16-byte stores (or fp32 NCHW for model outputs).
// With k_splits > 1 each split writes fp32 partial sums instead; the last
// split of a tile to finish reduces them and applies the epilogue
// (splitk_fixup), or, without arrival counters, conv_reduce does.
//
// conv_f32: direct convolution in fp32 FMA (no reduced-precision products)
// for float32 contexts.
#include <hip/hip_runtime.h>

#include "conv_epi.h"
#include "kargs.h"
#include "kernels.h"

namespace gemel {

// Implicit-GEMM tile kernel. BM x BN output tile, WM x WN waves (each a
// (BM/WM) x (BN/WN) wave tile of 16x16 MFMA blocks), depth 64 per step.
// Global loads run DEPTH steps ahead of the MFMAs (DEPTH register sets, the
// loop unrolled by two) and land in a double-buffered LDS tile whose rows
// are padded by 16 bytes so that the 16-byte fragment reads of 16
// consecutive rows hit distinct banks. Masked-off loads read a zero page
// instead of branching. CIN64: Cin is a multiple of 64, so one depth step
// covers a single filter tap (r, s) and the gather offsets are uniform.
template <int BM, int BN, int WM, int WN, int DEPTH, bool CIN64>
__global__ __launch_bounds__(64 * WM *WN) void conv_bf16_kernel(const ConvArgs a) {
    static_assert(DEPTH == 1 || DEPTH == 2, "prefetch depth");
    constexpr int NT = 64 * WM * WN;
    constexpr int BK = CONV_BK;
    constexpr int LDA = BK + 8;
    constexpr int TM = BM / WM, TN = BN / WN;
    constexpr int FM = TM / 16, FN = TN / 16;
    constexpr int RPP = NT / 8;                 // rows per load pass
    constexpr int AP = BM / RPP, BP = BN / RPP; // 16-byte loads per thread
    static_assert(AP * RPP == BM && BP * RPP == BN && AP >= 1 && BP >= 1, "tile/threads");
    constexpr int STAGE = (BM + BN) * LDA;      // bf16 elements per stage
    constexpr int SMEM_AB = 2 * STAGE * 2;
    constexpr int LDC = BN + 4;
    constexpr int FIT = SMEM_AB / (LDC * 4);
    constexpr int WPP = (FIT / TM) < WM ? (FIT / TM) : WM;   // wave rows per epilogue pass
    static_assert(WPP >= 1, "epilogue staging does not fit");
    constexpr int EPI_ROWS = WPP * TM;
    constexpr int SMEM_C = EPI_ROWS * LDC * 4;
    constexpr int SMEM = SMEM_AB > SMEM_C ? SMEM_AB : SMEM_C;
    constexpr int CH = BN / 8;                  // 8-channel chunks per row
    static_assert(NT % CH == 0, "epilogue chunk per thread");
    __shared__ __attribute__((aligned(16))) unsigned char smem[SMEM];
    u16 *const sAB = (u16 *)smem;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave - (wave / WN) * WN;
    const int tiles_n = (a.N + BN - 1) / BN;
    const int tiles = ((a.M + BM - 1) / BM) * tiles_n;
    // XCD-aware order: consecutive tiles (same rows, all column tiles) run
    // on one XCD and share its L2.
    const int G = gridDim.x;
    const int t = (G & 7) == 0 ? (int)(blockIdx.x & 7) * (G >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
    if (t >= tiles) return;
    const int tm = t / tiles_n, tn = t - (t / tiles_n) * tiles_n;
    const int k_begin = blockIdx.y * a.k_per_split;
    const int k_end = min(a.K, k_begin + a.k_per_split);
    const int HWo = a.Ho * a.Wo;
    const size_t frame_elems = (size_t)a.H * a.W * a.in_cs;
    const u16 *const zp = (const u16 *)a.zero;
    const int H = a.H, W = a.W, in_cs = a.in_cs, N = a.N, K = a.K, Cin = a.Cin, kw = a.kw;
    // segment of the tile's first and last row (wave-uniform, scalar loads):
    // rows of a tile inside one segment (the common case: segments are
    // whole frames) take its fields as uniform values; per-row lookups only
    // for a tile that straddles segments
    const int m_first = tm * BM, m_last = min(a.M, m_first + BM) - 1;
    int s_first = 0, s_last = 0;
    for (int i = 1; i < a.nseg; ++i) {
        s_first += m_first >= a.seg[i].m_start ? 1 : 0;
        s_last += m_last >= a.seg[i].m_start ? 1 : 0;
    }
    const bool one_seg = s_first == s_last;
    const RowSeg useg = uni_seg(a, s_first);

    // ---- loader set-up: thread owns K chunk q of rows r0 + RPP j ----
    const int q = tid & 7, r0 = tid >> 3;
    const u16 *abase[AP];
    int ahi[AP], awi[AP];
#pragma unroll
    for (int j = 0; j < AP; ++j) {
        const int gm = tm * BM + r0 + RPP * j;
        abase[j] = zp;
        ahi[j] = -(1 << 28);
        awi[j] = 0;
        if (gm < a.M) {
            const int fr = gm / HWo;
            const int pix = gm - fr * HWo;
            const int ho = pix / a.Wo, wo = pix - (pix / a.Wo) * a.Wo;
            if (one_seg) {
                abase[j] = (const u16 *)useg.in + (size_t)(fr - useg.f_start) * frame_elems;
            } else {
                const RowSeg sg = row_seg(a, gm);
                abase[j] = (const u16 *)sg.in + (size_t)(fr - sg.f_start) * frame_elems;
            }
            ahi[j] = ho * a.stride - a.pad;
            awi[j] = wo * a.stride - a.pad;
        }
    }
    const int gn0 = tn * BN + r0;
    const u16 *const bbase = (const u16 *)a.w + (size_t)(gn0 < a.N ? gn0 : 0) * a.K + q * 8;

    // loader position: the next depth step to fetch
    int kb = k_begin;      // step base
    int lc, lr, ls;        // CIN64: tap (lr, ls), channel base lc; else this thread's chunk
    {
        const int k0 = CIN64 ? k_begin : k_begin + q * 8;
        const int rs = k0 / Cin;
        lc = k0 - rs * Cin;
        lr = rs / kw;
        ls = rs - lr * kw;
    }

    auto gload = [&](u32x4 (&ra)[AP], u32x4 (&rb)[BP]) __attribute__((always_inline)) {
        const int kq = kb + q * 8;
        const bool kok = CIN64 ? true : kq < k_end;
        const int c = CIN64 ? lc + q * 8 : lc;
#pragma unroll
        for (int j = 0; j < AP; ++j) {
            const int hi = ahi[j] + lr, wi = awi[j] + ls;
            const bool ok = kok && (unsigned)hi < (unsigned)H && (unsigned)wi < (unsigned)W;
            const u16 *p = ok ? abase[j] + ((size_t)(hi * W + wi) * in_cs + c) : zp;
            ra[j] = *(const u32x4 *)p;
        }
#pragma unroll
        for (int j = 0; j < BP; ++j) {
            const bool ok = kok && gn0 + RPP * j < N;
            const u16 *p = ok ? bbase + (size_t)RPP * j * K + kb : zp;
            rb[j] = *(const u32x4 *)p;
        }
        // advance the loader by one step
        kb += BK;
        if (CIN64) {
            lc += BK;
            if (lc == Cin) {
                lc = 0;
                if (++ls == kw) { ls = 0; ++lr; }
            }
        } else {
            lc += BK;
            while (lc >= Cin) {
                lc -= Cin;
                if (++ls == kw) { ls = 0; ++lr; }
            }
        }
    };
    auto sstore = [&](int stage, const u32x4 (&ra)[AP], const u32x4 (&rb)[BP]) __attribute__((always_inline)) {
        u16 *As = sAB + stage * STAGE;
        u16 *Bs = As + BM * LDA;
#pragma unroll
        for (int j = 0; j < AP; ++j) *(u32x4 *)(As + (r0 + RPP * j) * LDA + q * 8) = ra[j];
#pragma unroll
        for (int j = 0; j < BP; ++j) *(u32x4 *)(Bs + (r0 + RPP * j) * LDA + q * 8) = rb[j];
    };

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto compute = [&](int stage) __attribute__((always_inline)) {
        const u16 *As = sAB + stage * STAGE;
        const u16 *Bs = As + BM * LDA;
#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            bf16x8 bfr[FN];
#pragma unroll
            for (int j = 0; j < FN; ++j)
                bfr[j] = *(const bf16x8 *)(Bs + (wn * TN + j * 16 + (lane & 15)) * LDA + kk * 32 + (lane >> 4) * 8);
#pragma unroll
            for (int i = 0; i < FM; ++i) {
                const bf16x8 af = *(const bf16x8 *)(As + (wm * TM + i * 16 + (lane & 15)) * LDA + kk * 32 + (lane >> 4) * 8);
#pragma unroll
                for (int j = 0; j < FN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfr[j], acc[i][j], 0, 0, 0);
            }
        }
    };

    const Epi e = epi_of(a, HWo);
    // Epilogue operands fetched before the depth loop so that their latency
    // overlaps the MFMAs: this thread's 8 channels of scale/shift and, for
    // single-pass tiles, the residual chunks of its output items.
    const int my_ch = tid % CH;
    const int my_gn = tn * BN + my_ch * 8;
    float sc[8], sh[8];
    const bool pre = a.uni_affine && a.k_splits <= 1 && a.out_mode == OUT_NHWC && my_gn < a.N;
    if (pre) {
        const float4 s0 = *(const float4 *)(a.seg[0].scale + my_gn), s1 = *(const float4 *)(a.seg[0].scale + my_gn + 4);
        const float4 h0 = *(const float4 *)(a.seg[0].shift + my_gn), h1 = *(const float4 *)(a.seg[0].shift + my_gn + 4);
        sc[0] = s0.x; sc[1] = s0.y; sc[2] = s0.z; sc[3] = s0.w; sc[4] = s1.x; sc[5] = s1.y; sc[6] = s1.z; sc[7] = s1.w;
        sh[0] = h0.x; sh[1] = h0.y; sh[2] = h0.z; sh[3] = h0.w; sh[4] = h1.x; sh[5] = h1.y; sh[6] = h1.z; sh[7] = h1.w;
    }
    constexpr int ITEMS = BM * CH / NT;          // output items per thread
    constexpr bool RES_PF = WPP == WM && ITEMS <= 4 && ITEMS * NT == BM * CH;
    u32x4 rpf[RES_PF ? ITEMS : 1];
    if (RES_PF && pre && e.has_res) {
#pragma unroll
        for (int i = 0; i < (RES_PF ? ITEMS : 1); ++i) {
            const int gm = tm * BM + (tid + NT * i) / CH;
            const u16 *p = zp;
            if (gm < a.M) {
                if (one_seg) {
                    p = (const u16 *)useg.res + (size_t)(gm - useg.m_start) * e.out_cs + my_gn;
                } else {
                    const RowSeg sg = row_seg(a, gm);
                    p = (const u16 *)sg.res + (size_t)(gm - sg.m_start) * e.out_cs + my_gn;
                }
            }
            rpf[i] = *(const u32x4 *)p;
        }
    }

    const int nk = (k_end - k_begin + BK - 1) / BK;
    if (DEPTH == 2) {
        u32x4 ra0[AP], rb0[BP], ra1[AP], rb1[BP];
        gload(ra0, rb0);
        if (nk > 1) gload(ra1, rb1);
        sstore(0, ra0, rb0);
        __syncthreads();
        for (int it = 0; it < nk; it += 2) {
            if (it + 2 < nk) gload(ra0, rb0);
            compute(0);
            if (it + 1 < nk) sstore(1, ra1, rb1);
            __syncthreads();
            if (it + 1 >= nk) break;
            if (it + 3 < nk) gload(ra1, rb1);
            compute(1);
            if (it + 2 < nk) sstore(0, ra0, rb0);
            __syncthreads();
        }
    } else {
        u32x4 ra0[AP], rb0[BP];
        gload(ra0, rb0);
        sstore(0, ra0, rb0);
        __syncthreads();
        for (int it = 0; it < nk; ++it) {
            const bool more = it + 1 < nk;
            if (more) gload(ra0, rb0);
            compute(it & 1);
            if (more) sstore((it + 1) & 1, ra0, rb0);
            __syncthreads();
        }
    }

    // ---- epilogue: fp32 tile staged through LDS, WPP wave rows per pass ----
    float *Cs = (float *)smem;
    for (int pass = 0; pass < WM; pass += WPP) {
        if (wm >= pass && wm < pass + WPP) {
#pragma unroll
            for (int i = 0; i < FM; ++i)
#pragma unroll
                for (int j = 0; j < FN; ++j)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        Cs[((wm - pass) * TM + i * 16 + (lane >> 4) * 4 + v) * LDC + wn * TN + j * 16 + (lane & 15)] =
                            acc[i][j][v];
        }
        __syncthreads();
        const int row0 = pass * TM;
        const int nrows = min(EPI_ROWS, BM - row0);
        if (a.k_splits > 1) {
            const __amdgpu_buffer_rsrc_t pr = partial_rsrc(a.partial, (uint32_t)a.k_splits * a.M * a.N * 4u);
            for (int item = tid; item < nrows * CH; item += NT) {
                const int rl = item / CH, ch = item - (item / CH) * CH;
                const int gm = tm * BM + row0 + rl, gn = tn * BN + ch * 8;
                if (gm >= a.M || gn >= a.N) continue;
                const float *src = Cs + rl * LDC + ch * 8;
                const uint32_t off = (uint32_t)((((int)blockIdx.y * a.M + gm) * a.N + gn) * 4u);
                store_partial4(pr, off, *(const float4 *)src);
                store_partial4(pr, off + 16, *(const float4 *)(src + 4));
            }
        } else if (a.out_mode == OUT_NHWC) {
            for (int item = tid; item < nrows * CH; item += NT) {
                const int rl = item / CH, ch = item - (item / CH) * CH;
                const int gm = tm * BM + row0 + rl, gn = tn * BN + ch * 8;
                if (gm >= a.M || gn >= a.N) continue;
                const float4 v0 = *(const float4 *)(Cs + rl * LDC + ch * 8);
                const float4 v1 = *(const float4 *)(Cs + rl * LDC + ch * 8 + 4);
                float v[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
                if (pre) {
                    const u16 *resp;
                    u16 *outp;
                    int ms;
                    if (one_seg) {
                        resp = (const u16 *)useg.res;
                        outp = (u16 *)useg.out;
                        ms = useg.m_start;
                    } else {
                        const RowSeg sg = row_seg(a, gm);
                        resp = (const u16 *)sg.res;
                        outp = (u16 *)sg.out;
                        ms = sg.m_start;
                    }
                    const size_t off = (size_t)(gm - ms) * e.out_cs + gn;
                    u32x4 r4 = {0u, 0u, 0u, 0u};
                    if (e.has_res) {
                        if constexpr (RES_PF)
                            r4 = rpf[(item - tid) / NT];
                        else
                            r4 = *(const u32x4 *)(resp + off);
                    }
                    float y[8];
                    epi8_f32(v, sc, sh, r4, e.kind, e.has_res, e.res_mode, e.act, e.slope, y);
                    store8_bf16(outp, off, y, e.pair);
                } else if (one_seg) {
                    store8_nhwc_bf16(useg, e, gm, gn, v);
                } else {
                    store8_nhwc_bf16(row_seg(a, gm), e, gm, gn, v);
                }
            }
        } else {
            for (int item = tid; item < nrows * BN; item += NT) {
                const int col = item / nrows, rl = item - (item / nrows) * nrows;
                const int gm = tm * BM + row0 + rl, gn = tn * BN + col;
                if (gm >= a.M || gn >= a.N) continue;
                if (one_seg)
                    store1_nchw_f32<true>(useg, e, gm, gn, Cs[rl * LDC + col]);
                else
                    store1_nchw_f32<true>(row_seg(a, gm), e, gm, gn, Cs[rl * LDC + col]);
            }
        }
        __syncthreads();
    }
    if (a.k_splits > 1 && a.counters) splitk_fixup<NT>(a, t, tm * BM, BM, tn * BN, BN, (int *)smem);
}

// Split-K reduction: sum the partial tiles, then the same epilogue.
template <bool BF16>
__global__ __launch_bounds__(256) void conv_reduce_kernel(const ReduceArgs ra) {
    const int item = blockIdx.x * 256 + threadIdx.x;
    const int chunks = ra.N / 8;
    if (item >= ra.M * chunks) return;
    const int gm = item / chunks, gn = (item - gm * chunks) * 8;
    float v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int sp = 0; sp < ra.splits; ++sp) {
        const float *p = ra.partial + ((size_t)sp * ra.M + gm) * ra.N + gn;
        const float4 p0 = *(const float4 *)p, p1 = *(const float4 *)(p + 4);
        v[0] += p0.x; v[1] += p0.y; v[2] += p0.z; v[3] += p0.w;
        v[4] += p1.x; v[5] += p1.y; v[6] += p1.z; v[7] += p1.w;
    }
    const Epi e = epi_of(ra, ra.HWo);
    const RowSeg sg = row_seg(ra, gm);
    if (ra.out_mode == OUT_NHWC) {
        if (BF16)
            store8_nhwc_bf16(sg, e, gm, gn, v);
        else
            store8_nhwc_f32(sg, e, gm, gn, v);
    } else {
        for (int j = 0; j < 8; ++j) store1_nchw_f32<BF16>(sg, e, gm, gn + j, v[j]);
    }
}

// Direct fp32 convolution: one thread per output element (row gm, col gn).
__global__ __launch_bounds__(256) void conv_f32_kernel(const ConvArgs a) {
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)a.M * a.N) return;
    const int gm = (int)(idx / a.N), gn = (int)(idx - (long)gm * a.N);
    const int HWo = a.Ho * a.Wo;
    const RowSeg sg = row_seg(a, gm);
    const int fr = gm / HWo, pix = gm - fr * HWo;
    const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
    const float *in = (const float *)sg.in + (size_t)(fr - sg.f_start) * a.H * a.W * a.in_cs;
    const float *w = (const float *)a.w + (size_t)gn * a.K;
    float acc = 0.f;
    for (int r = 0; r < a.kh; ++r) {
        const int hi = ho * a.stride - a.pad + r;
        if (hi < 0 || hi >= a.H) continue;
        for (int q = 0; q < a.kw; ++q) {
            const int wi = wo * a.stride - a.pad + q;
            if (wi < 0 || wi >= a.W) continue;
            const float *ip = in + (size_t)(hi * a.W + wi) * a.in_cs;
            const float *wp = w + (r * a.kw + q) * a.Cin;
            for (int cc = 0; cc < a.Cin; ++cc) acc = fmaf(ip[cc], wp[cc], acc);
        }
    }
    const Epi e = epi_of(a, HWo);
    if (a.out_mode == OUT_NHWC) {
        const size_t off = (size_t)(gm - sg.m_start) * a.out_cs + gn;
        const float r = a.has_res ? ((const float *)sg.res)[off] : 0.f;
        const float z = acc * sg.scale[gn] + sg.shift[gn];
        ((float *)sg.out)[off] = epi(z, r, a.has_res, a.res_mode, a.act, a.slope);
    } else {
        store1_nchw_f32<false>(sg, e, gm, gn, acc);
    }
}

struct TileShape {
    int bm, bn, threads;
};
static const TileShape kTiles[TILE_COUNT] = {
    {128, 128, 256}, {128, 64, 256}, {64, 64, 256}, {256, 256, 512}, {256, 128, 512},
    {256, 64, 256},  {64, 64, 256},  {128, 64, 256}, {64, 128, 256},
    {256, 256, 512}, {256, 128, 256}, {128, 128, 256}, {128, 64, 128}, {256, 32, 256},
    {256, 256, 512}, {256, 128, 256}, {128, 128, 256}, {128, 64, 128},
    {64, 64, 256}, {64, 64, 256},
    {256, 128, 512}, {128, 256, 512}, {256, 64, 256}, {64, 256, 256}};

int conv_tile_bm(int tile) { return tile >= 0 && tile < TILE_COUNT ? kTiles[tile].bm : 0; }
int conv_tile_bn(int tile) { return tile >= 0 && tile < TILE_COUNT ? kTiles[tile].bn : 0; }
int conv_tile_threads(int tile) { return tile >= 0 && tile < TILE_COUNT ? kTiles[tile].threads : 0; }

static bool conv_args_ok(const ConvArgs &a) {
    if (a.M <= 0 || a.N <= 0 || a.K <= 0 || a.nseg < 1 || a.nseg > GEMEL_MAX_SEG) return false;
    if (a.grouped) return false;   // the LDS-DMA kernel's form
    if (a.N % 8 || a.K % 8 || a.Cin % 8 || a.in_cs < a.Cin || a.in_cs % 8) return false;
    if (a.K != a.kh * a.kw * a.Cin || a.out_cs < a.N || a.out_cs % 8) return false;
    if (a.Ho <= 0 || a.Wo <= 0 || a.H <= 0 || a.W <= 0) return false;
    if (a.seg[0].m_start != 0) return false;
    for (int i = 0; i < a.nseg; ++i) {
        if (!a.seg[i].in || !a.seg[i].scale || !a.seg[i].shift) return false;
        if ((a.k_splits <= 1 || a.counters) && !a.seg[i].out) return false;
        if (a.has_res && !a.seg[i].res) return false;
        if (i && a.seg[i].m_start < a.seg[i - 1].m_start) return false;
        if (a.seg[i].m_start != a.seg[i].f_start * a.Ho * a.Wo) return false;
    }
    if (a.k_splits > 1 && (!a.partial || a.k_per_split % CONV_BK)) return false;
    if (a.k_splits > 1 && (long)a.k_splits * a.M * a.N * 4 > 0x7fffffffL) return false;
    if (a.k_per_split <= 0 || (long)a.k_per_split * a.k_splits < a.K) return false;
    if (a.out_mode == OUT_NCHW_F32 && a.cout > a.N) return false;
    // bf16 pairs: internal NHWC output, both halves inside the pixel
    if (a.out_pair && (a.out_mode != OUT_NHWC || a.out_pair < a.N || a.out_pair % 8 || a.out_cs < a.out_pair + a.N))
        return false;
    // the fused 2x2 pool and segments of mixed sizes exist only in the
    // LDS-DMA kernel
    if ((a.out_mode != OUT_NHWC && a.out_mode != OUT_NCHW_F32) || a.hetero) return false;
    return true;
}

template <bool C64>
static hipError_t launch_tile(int tile, dim3 grid, const Sink &sk, const ConvArgs &a) {
    hipError_t e = hipErrorInvalidValue;
    switch (tile) {
    case TILE_128x128: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<128, 128, 2, 2, 1, C64>), grid, dim3(256), a); break;
    case TILE_128x64: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<128, 64, 2, 2, 1, C64>), grid, dim3(256), a); break;
    case TILE_64x64: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<64, 64, 2, 2, 1, C64>), grid, dim3(256), a); break;
    case TILE_256x256: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<256, 256, 2, 4, 1, C64>), grid, dim3(512), a); break;
    case TILE_256x128: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<256, 128, 4, 2, 1, C64>), grid, dim3(512), a); break;
    case TILE_256x64: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<256, 64, 4, 1, 1, C64>), grid, dim3(256), a); break;
    case TILE_64x64_D2: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<64, 64, 2, 2, 2, C64>), grid, dim3(256), a); break;
    case TILE_128x64_D2: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<128, 64, 2, 2, 2, C64>), grid, dim3(256), a); break;
    case TILE_64x128: e = submit(sk, reinterpret_cast<const void *>(&conv_bf16_kernel<64, 128, 2, 2, 1, C64>), grid, dim3(256), a); break;
    }
    return e;
}

hipError_t launch_conv_bf16(const ConvArgs &a, int tile, const Sink &sk) {
    if (tile_is_dma(tile)) return launch_conv_dma(a, tile, sk);
    if (tile == TILE_STEM) return launch_conv_stem(a, sk);
    if (!conv_args_ok(a) || !a.zero) return hipErrorInvalidValue;
    const int bm = conv_tile_bm(tile), bn = conv_tile_bn(tile);
    if (!bm) return hipErrorInvalidValue;
    const long tiles = (long)((a.M + bm - 1) / bm) * ((a.N + bn - 1) / bn);
    const long blocks = tiles >= 8 ? (tiles + 7) / 8 * 8 : tiles;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    dim3 grid((unsigned)blocks, (unsigned)a.k_splits);
    const bool c64 = a.Cin % 64 == 0 && a.k_per_split % CONV_BK == 0 && a.in_cs % 8 == 0;
    return c64 ? launch_tile<true>(tile, grid, sk, a) : launch_tile<false>(tile, grid, sk, a);
}

hipError_t launch_conv_f32(const ConvArgs &a, const Sink &sk) {
    if (!conv_args_ok(a) || a.k_splits != 1 || a.out_pair) return hipErrorInvalidValue;
    const long n = (long)a.M * a.N;
    dim3 grid((unsigned)((n + 255) / 256)), block(256);
    return submit(sk, reinterpret_cast<const void *>(&conv_f32_kernel), grid, block, a);
}

hipError_t launch_conv_reduce(const ReduceArgs &a, bool bf16, const Sink &sk) {
    if (a.M <= 0 || a.N <= 0 || a.N % 8 || a.splits < 1 || !a.partial || a.nseg < 1 || a.nseg > GEMEL_MAX_SEG)
        return hipErrorInvalidValue;
    if (a.out_mode != OUT_NHWC && a.out_mode != OUT_NCHW_F32) return hipErrorInvalidValue;
    if (a.out_pair && (!bf16 || a.out_mode != OUT_NHWC || a.out_pair < a.N || a.out_pair % 8 ||
                       a.out_cs < a.out_pair + a.N))
        return hipErrorInvalidValue;
    for (int i = 0; i < a.nseg; ++i)
        if (!a.seg[i].out || !a.seg[i].scale || !a.seg[i].shift || (a.has_res && !a.seg[i].res))
            return hipErrorInvalidValue;
    const long n = (long)a.M * (a.N / 8);
    dim3 grid((unsigned)((n + 255) / 256)), block(256);
    return bf16 ? submit(sk, reinterpret_cast<const void *>(&conv_reduce_kernel<true>), grid, block, a)
                : submit(sk, reinterpret_cast<const void *>(&conv_reduce_kernel<false>), grid, block, a);
}

}  // namespace gemel
