// Fully connected layers for small frame counts (M <= 64 frames).
//
// An FC layer at a few frames is a weight-streaming problem: every weight
// byte is read once and used M times, far below the MFMA ridge point, so
// the kernel is organised for HBM bandwidth. Each wave owns 16 output
// neurons and a slice of K; every lane streams 64 contiguous bytes of one
// weight row per step (4 lanes cover 256 contiguous bytes of a row) and the
// same K positions of up to 16 frames, and v_mfma_f32_16x16x32_bf16 does the
// multiply-adds (weights as the 16-row A operand, frames as the 16-column B
// operand; the K order inside a step is the same for A and B, so any order
// is correct). K is split over blockIdx.y so that enough waves are in flight
// to saturate HBM; partial sums go to a [splits][M][N] fp32 buffer and the
// last split of each column of 64 neurons to finish reduces them and
// applies bias, activation and the store (or, without arrival counters,
// fc_reduce does). With one split the epilogue is applied directly.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kargs.h"
#include "kernels.h"
#include "splitk.h"

namespace gemel {

typedef unsigned short u16;
typedef __attribute__((address_space(3))) unsigned char fc_lds_u8;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float fc_bf2f(u16 h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ u16 fc_f2bf(float f) { return __builtin_bit_cast(u16, (__bf16)f); }
__device__ __forceinline__ float fc_act(float y, int act, float slope) {
    const float relu = fmaxf(y, 0.f);
    const float leaky = y > 0.f ? y : y * slope;
    return act == 1 ? relu : act == 2 ? leaky : y;
}

// Segment holding launch frame f: the last one with f_start <= f.
__device__ __forceinline__ int fc_seg(const FcArgs &a, int f) {
    int s = 0;
    for (int i = 1; i < a.nseg; ++i) s += (f >= a.seg[i].f_start) ? 1 : 0;
    return s;
}

// Input row of launch frame f. A select walk over the segments with
// constant indices: indexing the kernel-argument array with a computed
// index would copy it to scratch memory.
__device__ __forceinline__ const u16 *fc_in_row(const FcArgs &a, int f) {
    const u16 *p = (const u16 *)a.seg[0].in + (size_t)f * a.K;
#pragma unroll
    for (int i = 1; i < GEMEL_MAX_SEG; ++i)
        if (i < a.nseg && f >= a.seg[i].f_start) p = (const u16 *)a.seg[i].in + (size_t)(f - a.seg[i].f_start) * a.K;
    return p;
}

__device__ __forceinline__ void fc_store(const FcArgs &a, int f, int n, float acc, bool bf16) {
    const FcSeg &sg = a.seg[fc_seg(a, f)];
    const int lf = f - sg.f_start;
    const float y = fc_act(acc * sg.scale[n] + sg.shift[n], a.act, a.slope);
    if (a.out_mode == OUT_NHWC) {
        if (bf16)
            ((u16 *)sg.out)[(size_t)lf * a.out_cs + n] = fc_f2bf(y);
        else
            ((float *)sg.out)[(size_t)lf * a.out_cs + n] = y;
    } else if (n < a.cout) {
        ((float *)sg.out)[(size_t)lf * a.cout + n] = y;
    }
}

// Elements of the LDS input slice: (depth per split) x (frames padded to
// 16 per block), frame-minor, in runs of 64 16-byte slots. The planner
// keeps MB * 16 * k_per_split within it with room for the last run.
constexpr int FC_X_ELEMS = 32768;

// vmcnt(0) only: expcnt and lgkmcnt left at their maxima (gfx9 encoding).
__device__ __forceinline__ void fc_wait_vm0() { __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8)); }

template <int MB>  // frame blocks of 16
__global__ __launch_bounds__(256) void fc_bf16_kernel(const FcArgs a) {
    constexpr int COLS = 64;   // neurons of a workgroup, 16 per wave
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = blockIdx.x * COLS + wave * 16;
    const int k_begin = blockIdx.y * a.k_per_split;
    const int k_end = min(a.K, k_begin + a.k_per_split);
    const int g = lane >> 4;
    // frames [f0, f1) of this grid slice and their weights: every frame of
    // the launch, or (grouped) segment blockIdx.z alone. A select walk with
    // constant indices: indexing the kernel-argument array with a computed
    // index would copy it to scratch memory.
    const void *wsrc = a.w;
    int f0 = 0, f1 = a.M;
    if (a.grouped) {
        const int z = blockIdx.z;
#pragma unroll
        for (int i = 0; i < GEMEL_MAX_SEG; ++i) {
            if (i == z) {
                wsrc = a.seg[i].w;
                f0 = a.seg[i].f_start;
            }
            if (i == z + 1 && i < a.nseg) f1 = a.seg[i].f_start;
        }
    }
    const int mz = f1 - f0;
    const int row = n0 + (lane & 15);
    const bool row_ok = row < a.N;
    const u16 *wrow = (const u16 *)wsrc + (size_t)(row_ok ? row : 0) * a.K;
    // depth steps of 256: 8 weight chunks of 16 bytes per lane
    // (lane g of a row covers 32 contiguous bytes of every 128), the next
    // step's weights loaded while the current step's MFMAs run. The first
    // step is requested before the input slice is staged, so that its
    // latency overlaps the staging.
    constexpr int KS = 256, WJ = KS / 32;
    auto wload = [&](int k, uint4 (&wv)[WJ]) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < WJ; ++j) {
            const int kk = k + j * 32 + g * 8;
            wv[j] = (row_ok && kk < k_end) ? *(const uint4 *)(wrow + kk) : make_uint4(0, 0, 0, 0);
        }
    };
    uint4 w0[WJ], w1[WJ];
    if (n0 < a.N) wload(k_begin, w0);
    // the workgroup's slice of the inputs, [k_begin, k_end) x frames, staged
    // in LDS once: every wave reads it, and from LDS its reads need no wait
    // on a global round trip inside the depth loop. With MP frames staged
    // (M rounded up to a power of two up to 16, else 16 per frame block),
    // chunk c (8 elements) of frame f sits in 16-byte slot c * MP + f, so
    // the frames of a fragment are contiguous (no bank conflicts; lanes of
    // frames beyond MP read a staged frame again, for output columns that
    // are never stored). The slots are filled by direct global-to-LDS loads
    // (each wave instruction writes 64 consecutive slots), all in flight at
    // once; staged frames beyond M repeat frame M - 1.
    const int MP = mz > 16 ? 16 * MB : mz > 8 ? 16 : mz > 4 ? 8 : mz > 2 ? 4 : mz;
    __shared__ __attribute__((aligned(16))) u16 xs[FC_X_ELEMS];
    const int kn = k_end - k_begin;
    {
        const int slots = (kn / 8) * MP;
        for (int s0 = wave * 64; s0 < slots; s0 += 256) {
            const int sl = min(s0 + lane, slots - 1);
            const int c = sl / MP, f = f0 + min(sl - c * MP, mz - 1);
            __builtin_amdgcn_global_load_lds((const void *)(fc_in_row(a, f) + k_begin + c * 8),
                                             (fc_lds_u8 *)(xs + s0 * 8), 16, 0, 0);
        }
        fc_wait_vm0();
    }
    __syncthreads();
    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

    auto step = [&](int k, const uint4 (&wv)[WJ]) __attribute__((always_inline)) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            uint4 xv[WJ];
            const int fr = mb * 16 + (lane & 15);
            const u16 *xr = xs + (fr < MP ? fr : (fr & (MP - 1))) * 8;
#pragma unroll
            for (int j = 0; j < WJ; ++j) {
                const int kk = k + j * 32 + g * 8;
                xv[j] = kk < k_end ? *(const uint4 *)(xr + ((kk - k_begin) >> 3) * MP * 8) : make_uint4(0, 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < WJ; ++j)
                acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    __builtin_bit_cast(bf16x8, wv[j]), __builtin_bit_cast(bf16x8, xv[j]), acc[mb], 0, 0, 0);
        }
    };
    if (n0 < a.N) {
        for (int k = k_begin; k < k_end; k += 2 * KS) {
            if (k + KS < k_end) wload(k + KS, w1);
            step(k, w0);
            if (k + KS < k_end) {
                if (k + 2 * KS < k_end) wload(k + 2 * KS, w0);
                step(k + KS, w1);
            }
        }
    }
    // D[neuron = n0 + 4 g + v][frame = mb*16 + lane%16]
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
        const int f = f0 + mb * 16 + (lane & 15);
        if (f >= f1) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int n = n0 + g * 4 + v;
            if (n >= a.N) continue;
            if (a.k_splits > 1)
                store_partial1(a.partial + ((size_t)blockIdx.y * a.M + f) * a.N + n, acc[mb][v]);
            else
                fc_store(a, f, n, acc[mb][v], true);
        }
    }
    // fused split-K reduction: the last split of this column of neurons
    // sums the partials in split order, as fc_reduce does
    if (a.k_splits > 1 && a.counters) {
        __shared__ int flag;
        if (!splitk_arrive(a.counters + (a.grouped ? blockIdx.z * gridDim.x : 0) + blockIdx.x, a.k_splits, &flag))
            return;
        // four items per thread, eight splits per batch of loads
        for (int i0 = threadIdx.x; i0 < mz * COLS; i0 += 4 * 256) {
            float sum[4] = {0.f, 0.f, 0.f, 0.f};
            bool ok[4];
            const float *base[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int item = i0 + u * 256;
                const int f = f0 + item / COLS, n = blockIdx.x * COLS + (item % COLS);
                ok[u] = item < mz * COLS && n < a.N;
                base[u] = a.partial + (ok[u] ? (size_t)f * a.N + n : 0);
            }
            const size_t split_elems = (size_t)a.M * a.N;
            for (int sp0 = 0; sp0 < a.k_splits; sp0 += 8) {
                float p[4][8];
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (ok[u] && sp0 + q < a.k_splits) p[u][q] = load_partial1(base[u] + (sp0 + q) * split_elems);
#pragma unroll
                for (int u = 0; u < 4; ++u)
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (ok[u] && sp0 + q < a.k_splits) sum[u] += p[u][q];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int item = i0 + u * 256;
                if (ok[u]) fc_store(a, f0 + item / COLS, blockIdx.x * COLS + (item % COLS), sum[u], true);
            }
        }
    }
}

// float32 FC: one thread per (frame, neuron), fp32 FMA over K.
__global__ __launch_bounds__(256) void fc_f32_kernel(const FcArgs a) {
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)a.M * a.N) return;
    const int f = (int)(idx / a.N), n = (int)(idx - (long)f * a.N);
    const FcSeg &sg = a.seg[fc_seg(a, f)];
    const float *x = (const float *)sg.in + (size_t)(f - sg.f_start) * a.K;
    const float *w = (const float *)a.w + (size_t)n * a.K;
    float acc = 0.f;
    for (int k = 0; k < a.K; ++k) acc = fmaf(x[k], w[k], acc);
    fc_store(a, f, n, acc, false);
}

template <bool BF16>
__global__ __launch_bounds__(256) void fc_reduce_kernel(const FcArgs a) {
    const long idx = (long)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (long)a.M * a.N) return;
    const int f = (int)(idx / a.N), n = (int)(idx - (long)f * a.N);
    float acc = 0.f;
    for (int s = 0; s < a.k_splits; ++s) acc += a.partial[((size_t)s * a.M + f) * a.N + n];
    fc_store(a, f, n, acc, BF16);
}

static bool fc_args_ok(const FcArgs &a) {
    if (a.M <= 0 || a.N <= 0 || a.K <= 0 || a.nseg < 1 || a.nseg > GEMEL_MAX_SEG) return false;
    if (a.N % 8 || a.K % 8 || a.k_splits < 1 || a.k_per_split <= 0) return false;
    if ((long)a.k_splits * a.k_per_split < a.K) return false;
    if (a.out_mode == OUT_NHWC && a.out_cs < a.N) return false;
    if (a.out_mode == OUT_NCHW_F32 && a.cout > a.N) return false;
    if (a.seg[0].f_start != 0) return false;
    for (int i = 0; i < a.nseg; ++i)
        if (!a.seg[i].in || !a.seg[i].out || !a.seg[i].scale || !a.seg[i].shift) return false;
    if (a.k_splits > 1 && !a.partial) return false;
    if (a.grouped)
        for (int i = 0; i < a.nseg; ++i)
            if (!a.seg[i].w || (i > 0 && a.seg[i].f_start <= a.seg[i - 1].f_start)) return false;
    return true;
}

// Frames of the largest grid slice: the whole launch, or (grouped) the
// largest segment.
static int fc_slice_frames(const FcArgs &a) {
    if (!a.grouped) return a.M;
    int m = 0;
    for (int i = 0; i < a.nseg; ++i) m = std::max(m, (i + 1 < a.nseg ? a.seg[i + 1].f_start : a.M) - a.seg[i].f_start);
    return m;
}

hipError_t launch_fc_bf16(const FcArgs &a, const Sink &sk) {
    if (!fc_args_ok(a) || (a.k_splits > 1 && a.k_per_split % 128)) return hipErrorInvalidValue;
    const int ms = fc_slice_frames(a);
    if (ms < 1 || ms > 64) return hipErrorInvalidValue;
    {
        // LDS slots of the input slice, rounded up to whole 64-slot runs
        const int mp = ms > 16 ? (ms + 15) / 16 * 16 : ms > 8 ? 16 : ms > 4 ? 8 : ms > 2 ? 4 : ms;
        const long slots = (long)std::min(a.K, a.k_per_split) / 8 * mp;
        if ((slots + 63) / 64 * 64 * 8 > FC_X_ELEMS) return hipErrorInvalidValue;
    }
    dim3 grid((unsigned)((a.N + 63) / 64), (unsigned)a.k_splits, (unsigned)(a.grouped ? a.nseg : 1)), block(256);
    const int mb = (ms + 15) / 16;
    const void *t[4] = {reinterpret_cast<const void *>(&fc_bf16_kernel<1>),
                        reinterpret_cast<const void *>(&fc_bf16_kernel<2>),
                        reinterpret_cast<const void *>(&fc_bf16_kernel<3>),
                        reinterpret_cast<const void *>(&fc_bf16_kernel<4>)};
    const void *fn = t[mb - 1];
    return submit(sk, fn, grid, block, a);
}

hipError_t launch_fc_f32(const FcArgs &a, const Sink &sk) {
    if (!fc_args_ok(a) || a.k_splits != 1 || a.grouped) return hipErrorInvalidValue;
    const long n = (long)a.M * a.N;
    return submit(sk, reinterpret_cast<const void *>(&fc_f32_kernel), dim3((unsigned)((n + 255) / 256)), dim3(256), a);
}

hipError_t launch_fc_reduce(const FcArgs &a, bool bf16, const Sink &sk) {
    if (!fc_args_ok(a) || a.k_splits < 2) return hipErrorInvalidValue;
    const long n = (long)a.M * a.N;
    dim3 grid((unsigned)((n + 255) / 256)), block(256);
    return bf16 ? submit(sk, reinterpret_cast<const void *>(&fc_reduce_kernel<true>), grid, block, a)
                : submit(sk, reinterpret_cast<const void *>(&fc_reduce_kernel<false>), grid, block, a);
}

}  // namespace gemel
