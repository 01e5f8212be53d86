// Implicit-GEMM convolution for inputs with 8 physical channels (the RGB
// stems of the CNNs: 3 logical channels padded to 8), bf16 MFMA with fp32
// accumulation and the fused epilogue of the other conv kernels.
//
// With 8 channels per pixel, the 8 depth values a lane supplies to a
// 16x16x32 MFMA operand (one 16-byte chunk) are exactly one filter tap of
// one pixel, so both operands are loaded straight from global memory into
// registers (no im2col). With 64-channel tiles the weight fragments are
// staged in LDS once per workgroup instead (all four waves use the same
// ones; fetched by every wave they are two thirds of the loads, 5% of the
// time measured on the VGG and ResNet stems; with 32-channel tiles the
// staging costs more than it saves). A depth step of 32 covers 4 taps
// (the last step of a filter is padded with zero taps). The weight
// fragment is the MFMA's first operand and the pixel fragment its second,
// so a lane's result is 4 output channels of one pixel. The weight rows of
// each pair of channel fragments are interleaved so that those are channels
// 8q..8q+3 in one fragment and 8q+4..8q+7 in the other: a lane writes 8
// consecutive channels as one 16-byte store (NHWC) or 8 coalesced fp32
// writes (NCHW output). Epilogue scale/shift (one pair of arrays shared by
// every segment) are fetched together once the depth loop ends.
//
// Tile: 4 waves x PF 16-pixel fragments by NF 16-channel fragments: 64
// channels (PF 2) or 32 (PF 4) per workgroup, so that a pixel's output
// channels are written whole by one workgroup. The depth loop loads step
// k+1 while the MFMAs of step k run; with three steps (3x3 filters) every
// load is issued before the first MFMA.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kargs.h"
#include "kernels.h"

namespace gemel {

namespace {

typedef unsigned short u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float s_bf2f(u16 h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ u16 s_f2bf(float f) { return __builtin_bit_cast(u16, (__bf16)f); }
// Epilogue with selects on the launch-wide flags (branches would let the
// compiler duplicate the unrolled store code per flag combination).
__device__ __forceinline__ float s_act(float y, int act, float slope) {
    const float relu = fmaxf(y, 0.f);
    const float leaky = y > 0.f ? y : y * slope;
    return act == 1 ? relu : act == 2 ? leaky : y;
}
__device__ __forceinline__ float s_epi(float z, float r, int has_res, int res_mode, int act, float slope) {
    const bool pre = has_res && res_mode == 0, post = has_res && res_mode != 0;
    const float u = s_act(pre ? z + r : z, act, slope);
    return post ? u + r : u;
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

}  // namespace

template <int PF, int NF, int S>
__global__ __launch_bounds__(256) void conv_stem_kernel(const ConvArgs a) {
    constexpr int BN = NF * 16, STEM_PX = 4 * PF * 16;
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

    // segment of the tile's first and last pixel (wave-uniform, scalar
    // loads). A tile inside one segment (the common case: segments are whole
    // frames) takes that segment's fields as uniform values; only a tile
    // that straddles segments looks them up per pixel.
    const int m_first = tm * STEM_PX, m_last = min(a.M, m_first + STEM_PX) - 1;
    int s_first = 0, s_last = 0;
    for (int i = 1; i < a.nseg; ++i) {
        s_first += m_first >= a.seg[i].m_start ? 1 : 0;
        s_last += m_last >= a.seg[i].m_start ? 1 : 0;
    }
    const bool one_seg = s_first == s_last;
    // fields of the segment holding pixel m, gathered with uniform loads and
    // selects (a per-lane index into the argument block's segment table
    // would make each field a per-lane global load)
    struct SegF {
        const void *in, *res;
        void *out;
        int m_start, f_start;
    };
    auto seg_at = [&](int m) __attribute__((always_inline)) {
        SegF r{a.seg[0].in, a.seg[0].res, a.seg[0].out, a.seg[0].m_start, a.seg[0].f_start};
        for (int i = 1; i < a.nseg; ++i) {
            const bool hit = m >= a.seg[i].m_start;
            r.in = hit ? a.seg[i].in : r.in;
            r.res = hit ? a.seg[i].res : r.res;
            r.out = hit ? a.seg[i].out : r.out;
            r.m_start = hit ? a.seg[i].m_start : r.m_start;
            r.f_start = hit ? a.seg[i].f_start : r.f_start;
        }
        return r;
    };

    // this lane's pixel in each of the wave's PF pixel fragments. The
    // coordinates of the wave's first pixel come from uniform (scalar)
    // divisions; a lane's then follow by carrying its offset through the
    // columns, rows and frames (at most once per fragment for outputs at
    // least 16 wide), which costs far fewer vector instructions than a
    // division per lane and fragment
    const u16 *pbase[PF];
    int phi[PF], pwi[PF];
    const u16 *const in_u = (const u16 *)a.seg[s_first].in;
    const int f_u = a.seg[s_first].f_start;
    const int mw = tm * STEM_PX + wave * PF * 16;
    const int fw = mw / HWo, pw = mw - fw * HWo, how = pw / a.Wo;
    int fr = fw, ho = how, wo = pw - how * a.Wo + l16;
    SFor<PF>::run([&](auto I) __attribute__((always_inline)) {
        if (I > 0) wo += 16;
        while (wo >= a.Wo) {
            wo -= a.Wo;
            if (++ho == a.Ho) {
                ho = 0;
                ++fr;
            }
        }
        const int m = mw + I * 16 + l16;
        pbase[I] = zp;
        phi[I] = -(1 << 28);
        pwi[I] = 0;
        if (m < a.M) {
            if (one_seg) {
                pbase[I] = in_u + (size_t)(fr - f_u) * H * W * 8;
            } else {
                const SegF g = seg_at(m);
                pbase[I] = (const u16 *)g.in + (size_t)(fr - g.f_start) * H * W * 8;
            }
            phi[I] = ho * a.stride - a.pad;
            pwi[I] = wo * a.stride - a.pad;
        }
    });
    // this lane's weight row in each of the NF channel fragments: MFMA row r
    // of fragment J holds channel 32*(J/2) + 8*(r/4) + 4*(J%2) + r%4
    static_assert(NF % 2 == 0, "channel fragments come in pairs");
    // epilogue constants of this lane's channels c = 32*j + 8*kq .. +7 of
    // fragment pair j (every segment shares them; loaded from an in-range
    // channel), in named registers per pair
    struct Aff {
        f32x4 s0, s1, h0, h1;
    };
    auto load_aff = [&](int c) __attribute__((always_inline)) {
        const int cc = c < N ? c : 0;
        const float *sp = a.seg[0].scale + cc, *hp = a.seg[0].shift + cc;
        return Aff{*(const f32x4 *)sp, *(const f32x4 *)(sp + 4), *(const f32x4 *)hp, *(const f32x4 *)(hp + 4)};
    };

    // weight fragments of the channel tile: with 64-channel tiles staged in
    // LDS once per workgroup (fragment J of step st for lane l at
    // wl[(st * NF + J) * 64 + l]), else read by each wave from global memory
    constexpr bool WLDS = NF == 4;
    constexpr int MAX_STEPS = S > 0 ? S : (STEM_MAX_TAPS + 3) / 4;
    __shared__ bf16x8 wl[WLDS ? MAX_STEPS * NF * 64 : 1];
    const u16 *wrow[NF];
    SFor<NF>::run([&](auto J) __attribute__((always_inline)) {
        const int n = tn * BN + (J / 2) * 32 + (l16 >> 2) * 8 + (J % 2) * 4 + (l16 & 3);
        wrow[J] = n < N ? (const u16 *)a.w + (size_t)n * K : nullptr;
    });
    auto stage_weights = [&]() __attribute__((always_inline)) {
        if constexpr (!WLDS) return;
        for (int e = threadIdx.x; e < steps * NF * 64; e += 256) {
            const int l = e & 63, sj = e >> 6, st = sj / NF, J = sj - (sj / NF) * NF;
            // MFMA row r of fragment J holds channel 32*(J/2) + 8*(r/4) + 4*(J%2) + r%4
            const int n = tn * BN + (J / 2) * 32 + ((l & 15) >> 2) * 8 + (J % 2) * 4 + (l & 3);
            const int tap = st * 4 + (l >> 4);
            wl[e] = *(const bf16x8 *)((n < N && tap < taps) ? (const u16 *)a.w + (size_t)n * K + tap * 8 : zp);
        }
        __syncthreads();
    };
    auto read_w = [&](int step, bf16x8 (&wf)[NF]) __attribute__((always_inline)) {
        if constexpr (WLDS) {
            SFor<NF>::run([&](auto J) __attribute__((always_inline)) { wf[J] = wl[(step * NF + J) * 64 + lane]; });
        } else {
            const int tap = step * 4 + kq;
            SFor<NF>::run([&](auto J) __attribute__((always_inline)) {
                wf[J] = *(const bf16x8 *)((tap < taps && wrow[J]) ? wrow[J] + tap * 8 : zp);
            });
        }
    };
    auto load = [&](int step, bf16x8 (&pf)[PF]) __attribute__((always_inline)) {
        // filter row and column of this lane's tap: the step's first tap
        // (uniform) carried by kq < 4 columns
        const int tap = step * 4 + kq;
        const bool tok = tap < taps;
        const int r0 = (step * 4) / kw;
        int r = r0, s = step * 4 - r0 * kw + kq;
        while (s >= kw) {
            s -= kw;
            ++r;
        }
        SFor<PF>::run([&](auto I) __attribute__((always_inline)) {
            const int hi = phi[I] + r, wi = pwi[I] + s;
            const bool ok = tok && (unsigned)hi < (unsigned)H && (unsigned)wi < (unsigned)W;
            const u16 *p = ok ? pbase[I] + (size_t)(hi * W + wi) * 8 : zp;
            pf[I] = *(const bf16x8 *)p;
        });
    };

    f32x4 acc[PF][NF];
    SFor<PF>::run([&](auto I) __attribute__((always_inline)) { SFor<NF>::run([&](auto J) __attribute__((always_inline)) { acc[I][J] = f32x4{0.f, 0.f, 0.f, 0.f}; }); });
    bf16x8 w0[NF], p0[PF], w1[NF], p1[PF];
    auto mma = [&](const bf16x8 (&wf)[NF], const bf16x8 (&pf)[PF]) __attribute__((always_inline)) {
        SFor<PF>::run([&](auto I) __attribute__((always_inline)) {
            SFor<NF>::run([&](auto J) __attribute__((always_inline)) {
                acc[I][J] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[J], pf[I], acc[I][J], 0, 0, 0);
            });
        });
    };
    // the first pixel loads are issued before the weights are staged, so
    // that both wait out one memory latency together
    if constexpr (S > 0) {
        // S depth steps known at compile time (3x3 and 7x7 filters):
        // straight-line code with the pixel loads issued D steps ahead of
        // their MFMAs (3x3: all at once). A loop would carry the
        // accumulators, and the register allocator copies those between
        // register files on every iteration (64 instructions per two
        // steps, measured as half of the 7x7 stem's vector instructions).
        constexpr int D = S < 4 ? S : 4;
        bf16x8 pf[S][PF];
        SFor<D>::run([&](auto st) __attribute__((always_inline)) { load(st, pf[st]); });
        stage_weights();
        SFor<S>::run([&](auto st) __attribute__((always_inline)) {
            constexpr int si = decltype(st)::value;
            if constexpr (si + D < S) load(si + D, pf[si + D]);
            bf16x8 wf[NF];
            read_w(si, wf);
            mma(wf, pf[si]);
        });
    } else {
        load(0, p0);
        stage_weights();
        read_w(0, w0);
        for (int st = 0; st < steps; st += 2) {
            if (st + 1 < steps) {
                load(st + 1, p1);
                read_w(st + 1, w1);
            }
            mma(w0, p0);
            if (st + 1 < steps) {
                if (st + 2 < steps) {
                    load(st + 2, p0);
                    read_w(st + 2, w0);
                }
                mma(w1, p1);
            }
        }
    }

    // all epilogue constants at once, after the depth loop (held across it
    // they would be spilled; the empty asm keeps the compiler from hoisting
    // the loads above the loop)
    asm volatile("" ::: "memory");
    const Aff aff0 = load_aff(tn * BN + kq * 8);
    const Aff aff1 = NF > 2 ? load_aff(tn * BN + 32 + kq * 8) : aff0;
    void *const out_u = a.seg[s_first].out;
    const void *const res_u = a.seg[s_first].res;
    const int ms_u = a.seg[s_first].m_start;

    // epilogue kind: 0 none, 1 ReLU, 2 ReLU after the residual add, 3 leaky
    // ReLU with 0 <= slope <= 1 (max(y, slope * y)), 4 anything else
    const int skind = (!a.has_res && a.act == 0)                                  ? 0
                      : (!a.has_res && a.act == 1)                                ? 1
                      : (a.has_res && a.res_mode == 0 && a.act == 1)              ? 2
                      : (!a.has_res && a.act == 2 && a.slope >= 0.f && a.slope <= 1.f) ? 3
                                                                                  : 4;
    // epilogue: for each pixel fragment I and fragment pair j the lane holds
    // channels c0..c0+7 of pixel m (acc[I][2j] then acc[I][2j+1])
    SFor<PF>::run([&](auto I) __attribute__((always_inline)) {
        const int m = tm * STEM_PX + wave * PF * 16 + I * 16 + l16;
        if (m >= a.M) return;
        void *outp;
        const void *resp;
        int ml;
        if (one_seg) {
            outp = out_u;
            resp = res_u;
            ml = m - ms_u;
        } else {
            const SegF g = seg_at(m);
            outp = g.out;
            resp = g.res;
            ml = m - g.m_start;
        }
        SFor<NF / 2>::run([&](auto JP) __attribute__((always_inline)) {
            constexpr int j0 = 2 * JP, j1 = 2 * JP + 1;
            const int c0 = tn * BN + JP * 32 + kq * 8;
            if (c0 >= N) return;
            f32x4 sc0, sc1, sh0, sh1;
            if constexpr (decltype(JP)::value == 0) {
                sc0 = aff0.s0; sc1 = aff0.s1; sh0 = aff0.h0; sh1 = aff0.h1;
            } else {
                sc0 = aff1.s0; sc1 = aff1.s1; sh0 = aff1.h0; sh1 = aff1.h1;
            }
            float rv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            if (a.has_res) {
                const u32x4 rr = *(const u32x4 *)((const u16 *)resp + (size_t)ml * a.out_cs + c0);
                SFor<4>::run([&](auto Q) __attribute__((always_inline)) {
                    constexpr int q = Q;
                    rv[2 * q] = s_bf2f((u16)(rr[q] & 0xffff));
                    rv[2 * q + 1] = s_bf2f((u16)(rr[q] >> 16));
                });
            }
            float z[8], y[8];
            SFor<4>::run([&](auto V) __attribute__((always_inline)) {
                constexpr int v = V;
                z[v] = acc[I][j0][v] * sc0[v] + sh0[v];
                z[4 + v] = acc[I][j1][v] * sc1[v] + sh1[v];
            });
            // short sequences for the common epilogues (uniform switch)
            switch (skind) {
            case 0:
                for (int v = 0; v < 8; ++v) y[v] = z[v];
                break;
            case 1:
                for (int v = 0; v < 8; ++v) y[v] = fmaxf(z[v], 0.f);
                break;
            case 2:
                for (int v = 0; v < 8; ++v) y[v] = fmaxf(z[v] + rv[v], 0.f);
                break;
            case 3:
                for (int v = 0; v < 8; ++v) y[v] = fmaxf(z[v], z[v] * a.slope);
                break;
            default:
                for (int v = 0; v < 8; ++v) y[v] = s_epi(z[v], rv[v], a.has_res, a.res_mode, a.act, a.slope);
                break;
            }
            if (a.out_mode == OUT_NHWC) {
                u32x4 o;
                SFor<4>::run([&](auto Q) __attribute__((always_inline)) {
                    constexpr int q = Q;
                    o[q] = (uint32_t)s_f2bf(y[2 * q]) | ((uint32_t)s_f2bf(y[2 * q + 1]) << 16);
                });
                *(u32x4 *)((u16 *)outp + (size_t)ml * a.out_cs + c0) = o;
            } else {
                const int fl = ml / HWo, pix = ml - (ml / HWo) * HWo;
                float *o = (float *)outp + (size_t)fl * a.cout * HWo + pix;
                SFor<8>::run([&](auto V) __attribute__((always_inline)) {
                    constexpr int v = V;
                    if (c0 + v < a.cout) o[(size_t)(c0 + v) * HWo] = y[v];
                });
            }
        });
    });
}

bool conv_stem_supported(const ConvArgs &a) {
    return a.Cin == 8 && a.in_cs == 8 && a.k_splits <= 1 && a.kh * a.kw <= STEM_MAX_TAPS && a.zero && a.uni_affine &&
           !a.hetero && !a.grouped && !a.out_pair && (a.out_mode == OUT_NHWC || a.out_mode == OUT_NCHW_F32);
}

hipError_t launch_conv_stem(const ConvArgs &a, const Sink &sk) {
    if (!conv_stem_supported(a) || a.M <= 0 || a.N <= 0 || a.N % 8 || a.nseg < 1 || a.nseg > GEMEL_MAX_SEG)
        return hipErrorInvalidValue;
    if (a.K != a.kh * a.kw * 8 || a.out_cs < a.N || a.out_cs % 8 || a.seg[0].m_start != 0) return hipErrorInvalidValue;
    if (a.out_mode == OUT_NCHW_F32 && a.cout > a.N) return hipErrorInvalidValue;
    for (int i = 0; i < a.nseg; ++i) {
        const ConvSeg &s = a.seg[i];
        if (!s.in || !s.out || !s.scale || !s.shift || (a.has_res && !s.res)) return hipErrorInvalidValue;
        if (s.m_start != s.f_start * a.Ho * a.Wo || (i && s.m_start < a.seg[i - 1].m_start)) return hipErrorInvalidValue;
    }
    // up to 32 channels: 4 pixel fragments x 2 channel fragments per wave;
    // more: 2 x 4 (a wider tile holds its pixels' whole output rows; 4 x 4
    // would spill registers)
    const bool narrow = a.N <= 32;
    const int px = narrow ? 256 : 128, bn = narrow ? 32 : 64;
    const long tiles = (long)((a.M + px - 1) / px) * ((a.N + bn - 1) / bn);
    const long blocks = tiles >= 8 ? (tiles + 7) / 8 * 8 : tiles;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(256);
    // straight-line forms for 3 and 13 depth steps (3x3 and 7x7 filters)
    const int steps = (a.kh * a.kw + 3) / 4;
    const void *k = narrow ? (steps == 3    ? reinterpret_cast<const void *>(&conv_stem_kernel<4, 2, 3>)
                              : steps == 13 ? reinterpret_cast<const void *>(&conv_stem_kernel<4, 2, 13>)
                                            : reinterpret_cast<const void *>(&conv_stem_kernel<4, 2, 0>))
                           : (steps == 3    ? reinterpret_cast<const void *>(&conv_stem_kernel<2, 4, 3>)
                              : steps == 13 ? reinterpret_cast<const void *>(&conv_stem_kernel<2, 4, 13>)
                                            : reinterpret_cast<const void *>(&conv_stem_kernel<2, 4, 0>));
    return submit(sk, k, grid, block, a);
}

}  // namespace gemel
