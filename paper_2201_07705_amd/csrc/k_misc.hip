// Memory-bound layout, pooling and routing kernels (NHWC, physical channel
// counts multiple of 8). Every thread moves 8 channels (16 bytes of bf16)
// so that loads and stores are full-width and coalesced along C; one launch
// covers all models of a node, blockIdx.y selecting the model's segment.
#include <hip/hip_runtime.h>

#include "kargs.h"
#include "kernels.h"

namespace gemel {

typedef unsigned short u16;

__device__ __forceinline__ float m_bf2f(u16 h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ u16 m_f2bf(float f) { return __builtin_bit_cast(u16, (__bf16)f); }

__device__ __forceinline__ void load8(const u16 *p, float *v) {
    const uint4 x = *(const uint4 *)p;
    const u16 *h = (const u16 *)&x;
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = m_bf2f(h[j]);
}
__device__ __forceinline__ void load8(const float *p, float *v) {
    const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void store8(u16 *p, const float *v) {
    uint4 x;
    u16 *h = (u16 *)&x;
#pragma unroll
    for (int j = 0; j < 8; ++j) h[j] = m_f2bf(v[j]);
    *(uint4 *)p = x;
}
__device__ __forceinline__ void store8(float *p, const float *v) {
    *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]);
    *(float4 *)(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
// exact copies (no conversion) of 8 elements
__device__ __forceinline__ void copy8(u16 *d, const u16 *s) { *(uint4 *)d = *(const uint4 *)s; }
__device__ __forceinline__ void copy8(float *d, const float *s) {
    *(float4 *)d = *(const float4 *)s;
    *(float4 *)(d + 4) = *(const float4 *)(s + 4);
}

// Caller frames NCHW f32 -> NHWC, channels zero-padded to Co.
template <typename T>
__global__ __launch_bounds__(256) void pack_kernel(const EwArgs a) {
    const EwSeg &sg = a.seg[blockIdx.y];
    const long hw = (long)a.H * a.W;
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= sg.frames * hw) return;
    const long f = idx / hw, p = idx - f * hw;
    const float *src = (const float *)sg.in0 + f * a.c_logical * hw + p;
    T *dst = (T *)sg.out + idx * a.Co;
    for (int c0 = 0; c0 < a.Co; c0 += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (c0 + j < a.c_logical) ? src[(c0 + j) * hw] : 0.f;
        store8(dst + c0, v);
    }
}

// Max pool, window k, stride, pad; out-of-range taps are skipped (= -inf).
template <typename T>
__global__ __launch_bounds__(256) void maxpool_kernel(const EwArgs a) {
    const EwSeg &sg = a.seg[blockIdx.y];
    const int ch = a.C / 8;
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)sg.frames * a.Ho * a.Wo * ch) return;
    const int cc = (int)(idx % ch);
    long t = idx / ch;
    const int wo = (int)(t % a.Wo);
    t /= a.Wo;
    const int ho = (int)(t % a.Ho);
    const long f = t / a.Ho;
    const T *in = (const T *)sg.in0 + f * a.H * a.W * a.C + cc * 8;
    float m[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) m[j] = -INFINITY;
    for (int i = 0; i < a.k; ++i) {
        const int hi = ho * a.stride - a.pad + i;
        if (hi < 0 || hi >= a.H) continue;
        for (int q = 0; q < a.k; ++q) {
            const int wi = wo * a.stride - a.pad + q;
            if (wi < 0 || wi >= a.W) continue;
            float v[8];
            load8(in + ((long)hi * a.W + wi) * a.C, v);
#pragma unroll
            for (int j = 0; j < 8; ++j) m[j] = fmaxf(m[j], v[j]);
        }
    }
    store8((T *)sg.out + idx * 8, m);
}

// Global average pool: [f][H][W][C] -> [f][C], fp32 sums. A workgroup
// covers one frame and 64 8-channel chunks; its 4 waves take every 4th
// pixel (independent loads in flight), and the 4 partial sums meet in LDS.
// Grid: x = frames * ceil(chunks / 64), y = segment.
template <typename T>
__global__ __launch_bounds__(256) void avgpool_kernel(const EwArgs a) {
    __shared__ float part[4][64][9];
    const EwSeg &sg = a.seg[blockIdx.y];
    const int ch = a.C / 8, cblocks = (ch + 63) / 64;
    const long f = blockIdx.x / cblocks;
    if (f >= sg.frames) return;
    const int lane = threadIdx.x & 63, pg = threadIdx.x >> 6;
    const int cc = (int)(blockIdx.x - f * cblocks) * 64 + lane;
    const long hw = (long)a.H * a.W;
    float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (cc < ch) {
        const T *in = (const T *)sg.in0 + f * hw * a.C + cc * 8;
        for (long p = pg; p < hw; p += 4) {
            float v[8];
            load8(in + p * a.C, v);
#pragma unroll
            for (int j = 0; j < 8; ++j) s[j] += v[j];
        }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) part[pg][lane][j] = s[j];
    __syncthreads();
    if (pg == 0 && cc < ch) {
        const float inv = 1.0f / (float)hw;
#pragma unroll
        for (int j = 0; j < 8; ++j) s[j] = (part[0][lane][j] + part[1][lane][j] + part[2][lane][j] + part[3][lane][j]) * inv;
        store8((T *)sg.out + f * a.C + cc * 8, s);
    }
}

// Nearest-neighbour 2x upsample.
template <typename T>
__global__ __launch_bounds__(256) void upsample2x_kernel(const EwArgs a) {
    const EwSeg &sg = a.seg[blockIdx.y];
    const int ch = a.C / 8;
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)sg.frames * a.Ho * a.Wo * ch) return;
    const int cc = (int)(idx % ch);
    long t = idx / ch;
    const int wo = (int)(t % a.Wo);
    t /= a.Wo;
    const int ho = (int)(t % a.Ho);
    const long f = t / a.Ho;
    const T *in = (const T *)sg.in0 + ((f * a.H + ho / 2) * a.W + wo / 2) * a.C + cc * 8;
    copy8((T *)sg.out + idx * 8, in);
}

// Channel concat [in0 (C), in1 (C1)] -> out (C + C1), same H x W.
template <typename T>
__global__ __launch_bounds__(256) void concat_kernel(const EwArgs a) {
    const EwSeg &sg = a.seg[blockIdx.y];
    const int ch = a.Co / 8;
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)sg.frames * a.H * a.W * ch) return;
    const int cc = (int)(idx % ch);
    const long p = idx / ch;
    const int c = cc * 8;
    const T *src = c < a.C ? (const T *)sg.in0 + p * a.C + c : (const T *)sg.in1 + p * a.C1 + (c - a.C);
    copy8((T *)sg.out + idx * 8, src);
}

// Internal NHWC (C physical) -> caller NCHW f32 with c_logical channels.
// One thread per (frame, 8-channel chunk, pixel), pixels fastest: a 16-byte
// load of the pixel's 8 channels, then 8 plane writes that consecutive
// threads make to consecutive addresses.
template <typename T>
__global__ __launch_bounds__(256) void export_kernel(const EwArgs a) {
    const EwSeg &sg = a.seg[blockIdx.y];
    const long hw = (long)a.H * a.W;
    const int ch = (a.c_logical + 7) / 8;
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)sg.frames * ch * hw) return;
    const long p = idx % hw;
    const long t = idx / hw;
    const int cc = (int)(t % ch);
    const long f = t / ch;
    float v[8];
    load8((const T *)sg.in0 + (f * hw + p) * a.C + cc * 8, v);
    float *o = (float *)sg.out + (f * a.c_logical + cc * 8) * hw + p;
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (cc * 8 + j < a.c_logical) o[j * hw] = v[j];
}

// A launcher with nothing to launch (no frames): the sink's timing events,
// if any, are recorded on its stream where the kernel would have run, so
// that they bound an empty interval instead of staying unrecorded.
static hipError_t submit_nothing(const Sink &sk) {
    if (sk.graph) return hipSuccess;
    if (sk.ev_start) {
        const hipError_t e = hipEventRecord(sk.ev_start, sk.stream);
        if (e != hipSuccess) return e;
    }
    return sk.ev_stop ? hipEventRecord(sk.ev_stop, sk.stream) : hipSuccess;
}

static bool ew_ok(const EwArgs &a, bool need_in1) {
    if (a.nseg < 1 || a.nseg > GEMEL_MAX_SEG || a.max_frames < 0) return false;
    for (int i = 0; i < a.nseg; ++i) {
        if (a.seg[i].frames < 0 || a.seg[i].frames > a.max_frames) return false;
        if (!a.seg[i].in0 || !a.seg[i].out || (need_in1 && !a.seg[i].in1)) return false;
    }
    return true;
}

static hipError_t ew_launch(const void *kern, long items_per_frame, const EwArgs &a, const Sink &sk) {
    const long items = items_per_frame * a.max_frames;
    if (items <= 0) return submit_nothing(sk);
    const long blocks = (items + 255) / 256;
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    return submit(sk, kern, dim3((unsigned)blocks, (unsigned)a.nseg), dim3(256), a);
}

hipError_t launch_pack(const EwArgs &a, bool bf16, const Sink &sk) {
    if (!ew_ok(a, false) || a.Co % 8 || a.c_logical > a.Co || a.c_logical <= 0) return hipErrorInvalidValue;
    const long per = (long)a.H * a.W;
    return bf16 ? ew_launch(reinterpret_cast<const void *>(&pack_kernel<u16>), per, a, sk) : ew_launch(reinterpret_cast<const void *>(&pack_kernel<float>), per, a, sk);
}

hipError_t launch_maxpool(const EwArgs &a, bool bf16, const Sink &sk) {
    if (!ew_ok(a, false) || a.C % 8 || a.k <= 0 || a.stride <= 0 || a.pad >= a.k) return hipErrorInvalidValue;
    if (a.Ho != (a.H + 2 * a.pad - a.k) / a.stride + 1 || a.Wo != (a.W + 2 * a.pad - a.k) / a.stride + 1)
        return hipErrorInvalidValue;
    const long per = (long)a.Ho * a.Wo * (a.C / 8);
    return bf16 ? ew_launch(reinterpret_cast<const void *>(&maxpool_kernel<u16>), per, a, sk) : ew_launch(reinterpret_cast<const void *>(&maxpool_kernel<float>), per, a, sk);
}

hipError_t launch_avgpool(const EwArgs &a, bool bf16, const Sink &sk) {
    if (!ew_ok(a, false) || a.C % 8 || a.H <= 0 || a.W <= 0) return hipErrorInvalidValue;
    const long blocks = (long)a.max_frames * ((a.C / 8 + 63) / 64);
    if (blocks <= 0) return submit_nothing(sk);
    if (blocks > 0x7fffffffL) return hipErrorInvalidValue;
    const void *k = bf16 ? reinterpret_cast<const void *>(&avgpool_kernel<u16>)
                         : reinterpret_cast<const void *>(&avgpool_kernel<float>);
    return submit(sk, k, dim3((unsigned)blocks, (unsigned)a.nseg), dim3(256), a);
}

hipError_t launch_upsample2x(const EwArgs &a, bool bf16, const Sink &sk) {
    if (!ew_ok(a, false) || a.C % 8 || a.Ho != 2 * a.H || a.Wo != 2 * a.W) return hipErrorInvalidValue;
    const long per = (long)a.Ho * a.Wo * (a.C / 8);
    return bf16 ? ew_launch(reinterpret_cast<const void *>(&upsample2x_kernel<u16>), per, a, sk) : ew_launch(reinterpret_cast<const void *>(&upsample2x_kernel<float>), per, a, sk);
}

hipError_t launch_concat(const EwArgs &a, bool bf16, const Sink &sk) {
    if (!ew_ok(a, true) || a.C % 8 || a.C1 % 8 || a.Co != a.C + a.C1) return hipErrorInvalidValue;
    const long per = (long)a.H * a.W * (a.Co / 8);
    return bf16 ? ew_launch(reinterpret_cast<const void *>(&concat_kernel<u16>), per, a, sk) : ew_launch(reinterpret_cast<const void *>(&concat_kernel<float>), per, a, sk);
}

hipError_t launch_export(const EwArgs &a, bool bf16, const Sink &sk) {
    if (!ew_ok(a, false) || a.c_logical > a.C || a.c_logical <= 0) return hipErrorInvalidValue;
    const long per = (long)((a.c_logical + 7) / 8) * a.H * a.W;
    return bf16 ? ew_launch(reinterpret_cast<const void *>(&export_kernel<u16>), per, a, sk) : ew_launch(reinterpret_cast<const void *>(&export_kernel<float>), per, a, sk);
}

}  // namespace gemel
