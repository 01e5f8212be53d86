// Host-side launchers of the HIP kernels. Each launcher checks on the host
// that the argument block matches what its kernel and grid assume and
// returns hipErrorInvalidValue instead of launching otherwise.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "kargs.h"

namespace gemel {

// Where a launcher puts its kernel: enqueued on a stream, or, when graph is
// set, added to that HIP graph as a kernel node that runs after the ndeps
// nodes in deps (the new node is returned in *node). On a stream, ev_start
// and ev_stop (if set) take the start and end time of the kernel's own
// execution (hipExtLaunchKernel), not of its place in the stream.
struct Sink {
    hipStream_t stream = nullptr;
    hipGraph_t graph = nullptr;
    const hipGraphNode_t *deps = nullptr;
    size_t ndeps = 0;
    hipGraphNode_t *node = nullptr;
    hipEvent_t ev_start = nullptr;
    hipEvent_t ev_stop = nullptr;
};

// Launch kernel fn (one by-value argument block of type A, no dynamic LDS)
// into the sink. Node parameters are copied when the node is added.
template <typename A>
inline hipError_t submit(const Sink &sk, const void *fn, dim3 grid, dim3 block, const A &args) {
    void *params[] = {const_cast<A *>(&args)};
    if (!sk.graph && (sk.ev_start || sk.ev_stop))
        return hipExtLaunchKernel(fn, grid, block, params, 0, sk.stream, sk.ev_start, sk.ev_stop, 0);
    if (!sk.graph) return hipLaunchKernel(fn, grid, block, params, 0, sk.stream);
    hipKernelNodeParams p{};
    p.func = const_cast<void *>(fn);
    p.gridDim = grid;
    p.blockDim = block;
    p.sharedMemBytes = 0;
    p.kernelParams = params;
    p.extra = nullptr;
    return hipGraphAddKernelNode(sk.node, sk.graph, sk.deps, sk.ndeps, &p);
}

// Tile configurations of the bf16 implicit-GEMM convolution.
enum ConvTile {
    TILE_128x128 = 0,  // 4 waves, 64x64 per wave
    TILE_128x64 = 1,   // 4 waves, 64x32 per wave
    TILE_64x64 = 2,    // 4 waves, 32x32 per wave
    TILE_256x256 = 3,  // 8 waves, 128x64 per wave
    TILE_256x128 = 4,  // 8 waves, 64x64 per wave
    TILE_256x64 = 5,   // 4 waves, 64x64 per wave
    TILE_64x64_D2 = 6, // as 64x64, loads two depth steps ahead
    TILE_128x64_D2 = 7,// as 128x64, loads two depth steps ahead
    TILE_64x128 = 8,   // 4 waves, 32x64 per wave
    // LDS-DMA pipeline (k_conv_dma.hip), Cin a multiple of 32
    TILE_DMA_256x256 = 9,  // 8 waves, 128x64 per wave, 4 stages of depth 32
    TILE_DMA_256x128 = 10, // 4 waves, 128x64 per wave
    TILE_DMA_128x128 = 11, // 4 waves, 64x64 per wave
    TILE_DMA_128x64 = 12,  // 2 waves, 64x64 per wave
    // 8-channel inputs (k_stem.hip): 128 pixels x 64 channels (256 x 32
    // when N <= 32), no LDS
    TILE_STEM = 13,
    // LDS-DMA pipeline with depth steps of 64 (each row load a whole
    // 128-byte line), Cin a multiple of 64
    TILE_DMA64_256x256 = 14, // 8 waves, 2 stages
    TILE_DMA64_256x128 = 15, // 4 waves, 3 stages
    TILE_DMA64_128x128 = 16, // 4 waves, 2 stages
    TILE_DMA64_128x64 = 17,  // 2 waves, 3 stages
    // small tiles for latency-bound layers: 4 waves of 32x32, 4 stages
    TILE_DMA_64x64 = 18,     // depth 32 (4 workgroups per CU)
    TILE_DMA64_64x64 = 19,   // depth 64 (2 workgroups per CU)
    // LDS-DMA, depth 32, 4 stages, every wave a 64x64 tile (register
    // double-buffered fragments at two waves per SIMD)
    TILE_DMA_256x128W8 = 20, // 8 waves (4 x 2)
    TILE_DMA_128x256W8 = 21, // 8 waves (2 x 4)
    TILE_DMA_256x64 = 22,    // 4 waves (4 x 1), 2 workgroups per CU
    TILE_DMA_64x256 = 23,    // 4 waves (1 x 4), 2 workgroups per CU
    TILE_COUNT = 24
};
int conv_tile_threads(int tile);
int conv_tile_bm(int tile);
int conv_tile_bn(int tile);
// Output tiles of a conv launch for a bm x bn tile shape: a grouped launch
// tiles every segment on its own (a tile never straddles two segments).
inline long conv_tiles(const ConvArgs &a, int bm, int bn) {
    const long tn = (a.N + bn - 1) / bn;
    if (!a.grouped) return (long)((a.M + bm - 1) / bm) * tn;
    long t = 0;
    for (int i = 0; i < a.nseg; ++i) {
        const long rows = (i + 1 < a.nseg ? a.seg[i + 1].m_start : a.M) - (long)a.seg[i].m_start;
        t += (rows + bm - 1) / bm * tn;
    }
    return t;
}
constexpr int CONV_BK = 64;

hipError_t launch_conv_bf16(const ConvArgs &a, int tile, const Sink &sk);
bool conv_dma_supported(const ConvArgs &a);             // any DMA tile of depth 32
bool conv_dma_supported(const ConvArgs &a, int tile);   // this DMA tile
hipError_t launch_conv_dma(const ConvArgs &a, int tile, const Sink &sk);
inline bool tile_is_dma(int tile) {
    return (tile >= TILE_DMA_256x256 && tile <= TILE_DMA_128x64) ||
           (tile >= TILE_DMA64_256x256 && tile <= TILE_DMA_64x256);
}
inline int tile_dma_depth(int tile) {
    return (tile >= TILE_DMA64_256x256 && tile <= TILE_DMA64_128x64) || tile == TILE_DMA64_64x64 ? 64 : 32;
}
// Stem kernel: Cin == in_cs == 8, at most STEM_MAX_TAPS filter taps (7x7
// and smaller), no split-K.
constexpr int STEM_MAX_TAPS = 52;
bool conv_stem_supported(const ConvArgs &a);
hipError_t launch_conv_stem(const ConvArgs &a, const Sink &sk);
hipError_t launch_conv_f32(const ConvArgs &a, const Sink &sk);
// Split-K reduction + fused epilogue (bf16 or f32 internal activations).
hipError_t launch_conv_reduce(const ReduceArgs &a, bool bf16, const Sink &sk);

// Static device scratch of the allocation-free round: its address on the
// current device `device` (looked up once per device), and a fill kernel
// (stream sinks only) used to clear what must start at zero.
#define GEMEL_STATIC_SCRATCH_BYTES (64ull << 20)
hipError_t static_scratch(int device, void **ptr);
hipError_t launch_fill_u32(uint32_t *p, size_t n, uint32_t v, const Sink &sk);

hipError_t launch_fc_bf16(const FcArgs &a, const Sink &sk);
hipError_t launch_fc_f32(const FcArgs &a, const Sink &sk);
hipError_t launch_fc_reduce(const FcArgs &a, bool bf16, const Sink &sk);

// Input pack: caller NCHW f32 -> NHWC physical channels (bf16 or f32).
hipError_t launch_pack(const EwArgs &a, bool bf16, const Sink &sk);
hipError_t launch_maxpool(const EwArgs &a, bool bf16, const Sink &sk);
hipError_t launch_avgpool(const EwArgs &a, bool bf16, const Sink &sk);
hipError_t launch_upsample2x(const EwArgs &a, bool bf16, const Sink &sk);
hipError_t launch_concat(const EwArgs &a, bool bf16, const Sink &sk);
// Internal NHWC tensor -> caller NCHW f32 output.
hipError_t launch_export(const EwArgs &a, bool bf16, const Sink &sk);

}  // namespace gemel
