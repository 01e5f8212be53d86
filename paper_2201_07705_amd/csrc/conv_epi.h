// Device helpers shared by the implicit-GEMM conv kernels: the fused
// epilogue (per-channel scale/shift, residual before or after the
// activation, ReLU / leaky ReLU, bf16 NHWC or fp32 NCHW stores), the
// segment fields of a GEMM row (the last segment whose m_start <= row), and
// the fused split-K reduction.
#pragma once
#include <hip/hip_runtime.h>

#include "kargs.h"
#include "splitk.h"

namespace gemel {

typedef unsigned short u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf2f(u16 h) {
    return __uint_as_float((uint32_t)h << 16);
}
__device__ __forceinline__ u16 f2bf(float f) {
    return __builtin_bit_cast(u16, (__bf16)f);
}
// Activation (0 none, 1 ReLU, 2 leaky ReLU) and the residual epilogue,
// written with selects rather than branches: the flags are the same for a
// whole launch, and branches on them let the compiler duplicate every
// unrolled store loop once per flag combination (code that outgrows the
// instruction cache). The arithmetic of each case is unchanged.
__device__ __forceinline__ float act_fn(float y, int act, float slope) {
    const float relu = fmaxf(y, 0.f);
    const float leaky = y > 0.f ? y : y * slope;
    return act == 1 ? relu : act == 2 ? leaky : y;
}
__device__ __forceinline__ float epi(float z, float r, int has_res,
                                     int res_mode, int act, float slope) {
    const bool pre = has_res && res_mode == 0, post = has_res && res_mode != 0;
    const float u = act_fn(pre ? z + r : z, act, slope);
    return post ? u + r : u;
}

// Epilogue kinds with their own short instruction sequence; everything
// else takes the general form (epi). The flags are launch-wide, so the
// switch in epi8_bf16 is a uniform branch.
enum { EK_NONE = 0, EK_RELU = 1, EK_RELU_RES = 2, EK_LEAKY = 3, EK_GENERAL = 4 };
__device__ __forceinline__ int epi_kind(int act, int has_res, int res_mode, float slope) {
    if (!has_res && act == 0) return EK_NONE;
    if (!has_res && act == 1) return EK_RELU;
    if (has_res && res_mode == 0 && act == 1) return EK_RELU_RES;
    // for 0 <= slope <= 1, max(y, slope * y) is y for y > 0 and slope * y
    // otherwise (the leaky ReLU), one select fewer
    if (!has_res && act == 2 && slope >= 0.f && slope <= 1.f) return EK_LEAKY;
    return EK_GENERAL;
}
// y = the activation / residual of `kind` applied to z = v * scale + shift,
// in fp32. r4 holds the residual's 8 bf16 values (ignored unless the kind
// has a residual).
__device__ __forceinline__ void epi8_f32(const float *v, const float *sc, const float *sh, const u32x4 &r4,
                                         int kind, int has_res, int res_mode, int act, float slope, float *y) {
    // the residual is unpacked only where a kind reads it, so that kinds
    // without one never wait for its load
    auto res = [&](int j) __attribute__((always_inline)) {
        const uint32_t w = r4[j >> 1];
        return __uint_as_float((j & 1) ? (w & 0xffff0000u) : (w << 16));
    };
    switch (kind) {
    case EK_NONE:
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = v[j] * sc[j] + sh[j];
        break;
    case EK_RELU:
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = fmaxf(v[j] * sc[j] + sh[j], 0.f);
        break;
    case EK_RELU_RES:
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = fmaxf((v[j] * sc[j] + sh[j]) + res(j), 0.f);
        break;
    case EK_LEAKY:
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float z = v[j] * sc[j] + sh[j];
            y[j] = fmaxf(z, z * slope);
        }
        break;
    default:
#pragma unroll
        for (int j = 0; j < 8; ++j) y[j] = epi(v[j] * sc[j] + sh[j], res(j), has_res, res_mode, act, slope);
        break;
    }
}
// 8 fp32 values rounded to bf16 and packed in channel order.
__device__ __forceinline__ u32x4 pack8_bf16(const float *y) {
    u32x4 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = (uint32_t)f2bf(y[2 * q]) | ((uint32_t)f2bf(y[2 * q + 1]) << 16);
    return o;
}
// Stores 8 values y at out[off, off + 8) as bf16. With pair > 0 the
// remainders y - bf16(y) (exact in fp32), rounded to bf16, are stored at
// out[off + pair, off + pair + 8): the tensor then holds each value as a
// pair of bf16 whose sum carries about 16 significant bits.
__device__ __forceinline__ void store8_bf16(u16 *out, size_t off, const float *y, int pair) {
    const u32x4 hi = pack8_bf16(y);
    *(u32x4 *)(out + off) = hi;
    if (pair) {
        float lo[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t w = hi[j >> 1];
            lo[j] = y[j] - __uint_as_float((j & 1) ? (w & 0xffff0000u) : (w << 16));
        }
        *(u32x4 *)(out + off + pair) = pack8_bf16(lo);
    }
}

// epi8_f32, rounded to bf16 and packed in channel order.
__device__ __forceinline__ u32x4 epi8_bf16(const float *v, const float *sc, const float *sh, const u32x4 &r4,
                                           int kind, int has_res, int res_mode, int act, float slope) {
    float y[8];
    epi8_f32(v, sc, sh, r4, kind, has_res, res_mode, act, slope, y);
    return pack8_bf16(y);
}

// Fields of one segment. The segment table lives in the kernel argument
// block: indexing it with a per-lane segment number turns every field
// access into a per-lane global load on the critical path, so per-row
// fields are gathered by row_seg with uniform (scalar) loads and selects.
struct RowSeg {
    const void *in;
    const void *res;
    void *out;
    const float *scale;
    const float *shift;
    int m_start, f_start;
};
template <typename Args>
__device__ __forceinline__ RowSeg uni_seg(const Args &a, int s) {
    const ConvSeg &g = a.seg[s];
    return RowSeg{g.in, g.res, g.out, g.scale, g.shift, g.m_start, g.f_start};
}
template <typename Args>
__device__ __forceinline__ RowSeg row_seg(const Args &a, int gm) {
    RowSeg r = uni_seg(a, 0);
    for (int i = 1; i < a.nseg; ++i) {
        const RowSeg c = uni_seg(a, i);
        const bool hit = gm >= c.m_start;
        r.in = hit ? c.in : r.in;
        r.res = hit ? c.res : r.res;
        r.out = hit ? c.out : r.out;
        r.scale = hit ? c.scale : r.scale;
        r.shift = hit ? c.shift : r.shift;
        r.m_start = hit ? c.m_start : r.m_start;
        r.f_start = hit ? c.f_start : r.f_start;
    }
    return r;
}

// Scalars of the fused epilogue.
struct Epi {
    int out_cs, cout, act, res_mode, has_res, HWo, kind, pair;
    float slope;
};
template <typename Args>
__device__ __forceinline__ Epi epi_of(const Args &a, int HWo) {
    Epi e;
    e.pair = a.out_pair;
    e.out_cs = a.out_cs; e.cout = a.cout; e.act = a.act; e.res_mode = a.res_mode;
    e.has_res = a.has_res; e.HWo = HWo; e.slope = a.slope;
    e.kind = epi_kind(a.act, a.has_res, a.res_mode, a.slope);
    return e;
}

// Epilogue of 8 consecutive channels [gn, gn+8) of row gm into NHWC bf16.
__device__ __forceinline__ void store8_nhwc_bf16(const RowSeg &sg, const Epi &e,
                                                 int gm, int gn, const float *v) {
    const size_t off = (size_t)(gm - sg.m_start) * e.out_cs + gn;
    const float4 sc0 = *(const float4 *)(sg.scale + gn);
    const float4 sc1 = *(const float4 *)(sg.scale + gn + 4);
    const float4 sh0 = *(const float4 *)(sg.shift + gn);
    const float4 sh1 = *(const float4 *)(sg.shift + gn + 4);
    const float sc[8] = {sc0.x, sc0.y, sc0.z, sc0.w, sc1.x, sc1.y, sc1.z, sc1.w};
    const float sh[8] = {sh0.x, sh0.y, sh0.z, sh0.w, sh1.x, sh1.y, sh1.z, sh1.w};
    u32x4 r4 = {0u, 0u, 0u, 0u};
    if (e.has_res) r4 = *(const u32x4 *)((const u16 *)sg.res + off);
    float y[8];
    epi8_f32(v, sc, sh, r4, e.kind, e.has_res, e.res_mode, e.act, e.slope, y);
    store8_bf16((u16 *)sg.out, off, y, e.pair);
}

// Epilogue of 8 consecutive channels of row gm into NHWC fp32.
__device__ __forceinline__ void store8_nhwc_f32(const RowSeg &sg, const Epi &e,
                                                int gm, int gn, const float *v) {
    const size_t off = (size_t)(gm - sg.m_start) * e.out_cs + gn;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float r = e.has_res ? ((const float *)sg.res)[off + j] : 0.f;
        const float z = v[j] * sg.scale[gn + j] + sg.shift[gn + j];
        ((float *)sg.out)[off + j] = epi(z, r, e.has_res, e.res_mode, e.act, e.slope);
    }
}

// Epilogue of one element into a caller-owned fp32 NCHW output.
template <bool BF16>
__device__ __forceinline__ void store1_nchw_f32(const RowSeg &sg, const Epi &e,
                                                int gm, int gn, float v) {
    if (gn >= e.cout) return;
    const int lr = gm - sg.m_start;
    const int f = lr / e.HWo, pix = lr - f * e.HWo;
    float r = 0.f;
    if (e.has_res) {
        const size_t roff = (size_t)lr * e.out_cs + gn;
        r = BF16 ? bf2f(((const u16 *)sg.res)[roff]) : ((const float *)sg.res)[roff];
    }
    const float z = v * sg.scale[gn] + sg.shift[gn];
    ((float *)sg.out)[((size_t)f * e.cout + gn) * e.HWo + pix] =
        epi(z, r, e.has_res, e.res_mode, e.act, e.slope);
}

// Fused split-K reduction of output tile `tile` (rows [m0, m0 + bm),
// columns [n0, n0 + bn)): the last split to arrive sums the partials in
// split order and applies the epilogue with the arithmetic of the separate
// reduction kernel, so both give the same bits. The launcher guarantees
// that the partial sums span less than 2^31 bytes.
template <int NT>
__device__ __forceinline__ void splitk_fixup(const ConvArgs &a, int tile, int m0, int bm, int n0, int bn,
                                             int *flag) {
    if (!splitk_arrive(a.counters + tile, a.k_splits, flag)) return;
    const Epi e = epi_of(a, a.Ho * a.Wo);
    const __amdgpu_buffer_rsrc_t pr = partial_rsrc(a.partial, (uint32_t)a.k_splits * a.M * a.N * 4u);
    const int chunks = bn / 8, items = bm * chunks;
    const uint32_t split_bytes = (uint32_t)a.M * a.N * 4u;
    // two items per thread and four splits per batch: the 16 loads of a
    // batch are issued together, then summed in split order
    for (int i0 = threadIdx.x; i0 < items; i0 += 2 * NT) {
        int gm[2], gn[2];
        bool ok[2];
        uint32_t off[2];
        float v[2][8];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int item = i0 + u * NT;
            const int rl = item / chunks;
            gm[u] = m0 + rl;
            gn[u] = n0 + (item - rl * chunks) * 8;
            ok[u] = item < items && gm[u] < a.M && gn[u] < a.N;
            off[u] = ok[u] ? (uint32_t)((gm[u] * a.N + gn[u]) * 4u) : 0u;
#pragma unroll
            for (int j = 0; j < 8; ++j) v[u][j] = 0.f;
        }
        for (int sp0 = 0; sp0 < a.k_splits; sp0 += 4) {
            float4 p[2][4][2];
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (ok[u] && sp0 + q < a.k_splits) {
                        const uint32_t o = off[u] + (uint32_t)(sp0 + q) * split_bytes;
                        p[u][q][0] = load_partial4(pr, o);
                        p[u][q][1] = load_partial4(pr, o + 16);
                    }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (ok[u] && sp0 + q < a.k_splits) {
                        v[u][0] += p[u][q][0].x; v[u][1] += p[u][q][0].y;
                        v[u][2] += p[u][q][0].z; v[u][3] += p[u][q][0].w;
                        v[u][4] += p[u][q][1].x; v[u][5] += p[u][q][1].y;
                        v[u][6] += p[u][q][1].z; v[u][7] += p[u][q][1].w;
                    }
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            if (!ok[u]) continue;
            const RowSeg sg = row_seg(a, gm[u]);
            if (a.out_mode == OUT_NHWC) {
                store8_nhwc_bf16(sg, e, gm[u], gn[u], v[u]);
            } else {
                for (int j = 0; j < 8; ++j) store1_nchw_f32<true>(sg, e, gm[u], gn[u] + j, v[u][j]);
            }
        }
    }
}

}  // namespace gemel
