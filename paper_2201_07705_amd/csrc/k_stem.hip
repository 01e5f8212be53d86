// Implicit-GEMM convolution for inputs with 8 physical channels (the RGB
// stems of the CNNs: 3 logical channels padded to 8), bf16 MFMA with fp32
// accumulation and the fused epilogue of the other conv kernels.
//
// With 8 channels per pixel, the 8 depth values a lane supplies to a
// 16x16x32 MFMA operand (one 16-byte chunk) are exactly one filter tap of
// one pixel, so both operands are loaded straight from global memory into
// registers: no LDS staging and no im2col. A depth step of 32 covers 4 taps
// (the last step of a filter is padded with zero taps). The weight
// fragment is the MFMA's first operand and the pixel fragment its second,
// so a lane's result is 4 consecutive output channels of one pixel, stored
// as one 8-byte write (NHWC) or 4 coalesced fp32 writes (NCHW output).
//
// Tile: 4 waves x 64 pixels (four 16-pixel fragments each) by 32 output
// channels; the depth loop loads step k+1 while the MFMAs of step k run.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kargs.h"
#include "kernels.h"

namespace gemel {

namespace {

typedef unsigned short u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float s_bf2f(u16 h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ u16 s_f2bf(float f) { return __builtin_bit_cast(u16, (__bf16)f); }
__device__ __forceinline__ float s_act(float y, int act, float slope) {
    if (act == 1) return fmaxf(y, 0.f);
    if (act == 2) return y > 0.f ? y : y * slope;
    return y;
}
__device__ __forceinline__ float s_epi(float z, float r, int has_res, int res_mode, int act, float slope) {
    if (!has_res) return s_act(z, act, slope);
    if (res_mode == 0) return s_act(z + r, act, slope);
    return s_act(z, act, slope) + r;
}

template <int I>
struct SFor {
    template <typename F>
    __device__ __forceinline__ static void run(F &&f) {
        SFor<I - 1>::run(f);
        f(std::integral_constant<int, I - 1>{});
    }
};
template <>
struct SFor<0> {
    template <typename F>
    __device__ __forceinline__ static void run(F &&) {}
};

constexpr int STEM_PX = 256;   // pixels per workgroup (4 waves x 64)

}  // namespace

template <int NF>
__global__ __launch_bounds__(256) void conv_stem_kernel(const ConvArgs a) {
    constexpr int BN = NF * 16;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int tiles_n = (a.N + BN - 1) / BN;
    const int tiles = ((a.M + STEM_PX - 1) / STEM_PX) * tiles_n;
    const int G = gridDim.x;
    const int t = (G & 7) == 0 ? (int)(blockIdx.x & 7) * (G >> 3) + (int)(blockIdx.x >> 3) : (int)blockIdx.x;
    if (t >= tiles) return;
    const int tm = t / tiles_n, tn = t - (t / tiles_n) * tiles_n;
    const int HWo = a.Ho * a.Wo, H = a.H, W = a.W, K = a.K, N = a.N, kw = a.kw;
    const int taps = a.kh * a.kw;
    const int steps = (taps + 3) / 4;
    const int l16 = lane & 15, kq = lane >> 4;   // fragment row/column, tap within a step
    const u16 *const zp = (const u16 *)a.zero;

    // this lane's pixel in each of the wave's 4 pixel fragments
    const u16 *pbase[4];
    int phi[4], pwi[4];
    SFor<4>::run([&](auto I) {
        const int m = tm * STEM_PX + wave * 64 + I * 16 + l16;
        pbase[I] = zp;
        phi[I] = -(1 << 28);
        pwi[I] = 0;
        if (m < a.M) {
            int s = 0;
            for (int i = 1; i < a.nseg; ++i) s += (m >= a.seg[i].m_start) ? 1 : 0;
            const int fr = m / HWo, pix = m - (m / HWo) * HWo;
            const int ho = pix / a.Wo, wo = pix - (pix / a.Wo) * a.Wo;
            pbase[I] = (const u16 *)a.seg[s].in + (size_t)(fr - a.seg[s].f_start) * H * W * 8;
            phi[I] = ho * a.stride - a.pad;
            pwi[I] = wo * a.stride - a.pad;
        }
    });
    // this lane's weight row in each of the NF channel fragments
    const u16 *wrow[NF];
    SFor<NF>::run([&](auto J) {
        const int n = tn * BN + J * 16 + l16;
        wrow[J] = n < N ? (const u16 *)a.w + (size_t)n * K : nullptr;
    });

    auto load = [&](int step, bf16x8 (&wf)[NF], bf16x8 (&pf)[4]) __attribute__((always_inline)) {
        const int tap = step * 4 + kq;
        const bool tok = tap < taps;
        const int r = tok ? tap / kw : 0, s = tok ? tap - (tap / kw) * kw : 0;
        SFor<NF>::run([&](auto J) {
            const u16 *p = (tok && wrow[J]) ? wrow[J] + tap * 8 : zp;
            wf[J] = *(const bf16x8 *)p;
        });
        SFor<4>::run([&](auto I) {
            const int hi = phi[I] + r, wi = pwi[I] + s;
            const bool ok = tok && (unsigned)hi < (unsigned)H && (unsigned)wi < (unsigned)W;
            const u16 *p = ok ? pbase[I] + (size_t)(hi * W + wi) * 8 : zp;
            pf[I] = *(const bf16x8 *)p;
        });
    };

    f32x4 acc[4][NF];
    SFor<4>::run([&](auto I) { SFor<NF>::run([&](auto J) { acc[I][J] = f32x4{0.f, 0.f, 0.f, 0.f}; }); });
    bf16x8 w0[NF], p0[4], w1[NF], p1[4];
    load(0, w0, p0);
    auto mma = [&](const bf16x8 (&wf)[NF], const bf16x8 (&pf)[4]) __attribute__((always_inline)) {
        SFor<4>::run([&](auto I) {
            SFor<NF>::run([&](auto J) {
                acc[I][J] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[J], pf[I], acc[I][J], 0, 0, 0);
            });
        });
    };
    for (int st = 0; st < steps; st += 2) {
        if (st + 1 < steps) load(st + 1, w1, p1);
        mma(w0, p0);
        if (st + 1 < steps) {
            if (st + 2 < steps) load(st + 2, w0, p0);
            mma(w1, p1);
        }
    }

    // epilogue: lane holds channels c0..c0+3 of pixel m for each (I, J)
    SFor<4>::run([&](auto I) {
        const int m = tm * STEM_PX + wave * 64 + I * 16 + l16;
        if (m >= a.M) return;
        int sidx = 0;
        for (int i = 1; i < a.nseg; ++i) sidx += (m >= a.seg[i].m_start) ? 1 : 0;
        const ConvSeg &sg = a.seg[sidx];
        const int ml = m - sg.m_start;
        SFor<NF>::run([&](auto J) {
            const int c0 = tn * BN + J * 16 + kq * 4;
            if (c0 >= N) return;
            const f32x4 sc = *(const f32x4 *)(sg.scale + c0);
            const f32x4 sh = *(const f32x4 *)(sg.shift + c0);
            float rv[4] = {0.f, 0.f, 0.f, 0.f};
            if (a.has_res) {
                const u32x2 rr = *(const u32x2 *)((const u16 *)sg.res + (size_t)ml * a.out_cs + c0);
                rv[0] = s_bf2f((u16)(rr.x & 0xffff));
                rv[1] = s_bf2f((u16)(rr.x >> 16));
                rv[2] = s_bf2f((u16)(rr.y & 0xffff));
                rv[3] = s_bf2f((u16)(rr.y >> 16));
            }
            float y[4];
            SFor<4>::run([&](auto V) {
                constexpr int v = V;
                y[v] = s_epi(acc[I][J][v] * sc[v] + sh[v], rv[v], a.has_res, a.res_mode, a.act, a.slope);
            });
            if (a.out_mode == OUT_NHWC) {
                u32x2 o;
                o.x = (uint32_t)s_f2bf(y[0]) | ((uint32_t)s_f2bf(y[1]) << 16);
                o.y = (uint32_t)s_f2bf(y[2]) | ((uint32_t)s_f2bf(y[3]) << 16);
                *(u32x2 *)((u16 *)sg.out + (size_t)ml * a.out_cs + c0) = o;
            } else {
                const int fl = ml / HWo, pix = ml - (ml / HWo) * HWo;
                float *o = (float *)sg.out + (size_t)fl * a.cout * HWo + pix;
                SFor<4>::run([&](auto V) {
                    constexpr int v = V;
                    if (c0 + v < a.cout) o[(size_t)(c0 + v) * HWo] = y[v];
                });
            }
        });
    });
}

bool conv_stem_supported(const ConvArgs &a) {
    return a.Cin == 8 && a.in_cs == 8 && a.k_splits <= 1 && a.kh * a.kw <= 64 && a.zero &&
           (a.out_mode == OUT_NHWC || a.out_mode == OUT_NCHW_F32);
}

hipError_t launch_conv_stem(const ConvArgs &a, const Sink &sk) {
    if (!conv_stem_supported(a) || a.M <= 0 || a.N <= 0 || a.N % 8 || a.nseg < 1 || a.nseg > GEMEL_MAX_SEG)
        return hipErrorInvalidValue;
    if (a.K != a.kh * a.kw * 8 || a.out_cs < a.N || a.out_cs % 4 || a.seg[0].m_start != 0) return hipErrorInvalidValue;
    if (a.out_mode == OUT_NCHW_F32 && a.cout > a.N) return hipErrorInvalidValue;
    for (int i = 0; i < a.nseg; ++i) {
        const ConvSeg &s = a.seg[i];
        if (!s.in || !s.out || !s.scale || !s.shift || (a.has_res && !s.res)) return hipErrorInvalidValue;
        if (s.m_start != s.f_start * a.Ho * a.Wo || (i && s.m_start < a.seg[i - 1].m_start)) return hipErrorInvalidValue;
    }
    // 32 output channels per tile: the pixel loads of a wider tile would be
    // re-used across more MFMAs, but its registers spill
    constexpr int NF = 2;
    const long tiles = (long)((a.M + STEM_PX - 1) / STEM_PX) * ((a.N + NF * 16 - 1) / (NF * 16));
    const long blocks = tiles >= 8 ? (tiles + 7) / 8 * 8 : tiles;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(256);
    return submit(sk, reinterpret_cast<const void *>(&conv_stem_kernel<NF>), grid, block, a);
}

}  // namespace gemel
