// Host-side launchers of the HIP kernels. Each launcher checks on the host
// that the argument block matches what its kernel and grid assume and
// returns hipErrorInvalidValue instead of launching otherwise.
#pragma once
#include <hip/hip_runtime.h>

#include "kargs.h"

namespace gemel {

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
    TILE_COUNT = 13
};
int conv_tile_threads(int tile);
int conv_tile_bm(int tile);
int conv_tile_bn(int tile);
constexpr int CONV_BK = 64;

hipError_t launch_conv_bf16(const ConvArgs &a, int tile, hipStream_t st);
bool conv_dma_supported(const ConvArgs &a);
hipError_t launch_conv_dma(const ConvArgs &a, int tile, hipStream_t st);
inline bool tile_is_dma(int tile) { return tile >= TILE_DMA_256x256 && tile < TILE_COUNT; }
hipError_t launch_conv_f32(const ConvArgs &a, hipStream_t st);
// Split-K reduction + fused epilogue (bf16 or f32 internal activations).
hipError_t launch_conv_reduce(const ReduceArgs &a, bool bf16, hipStream_t st);

hipError_t launch_fc_bf16(const FcArgs &a, hipStream_t st);
hipError_t launch_fc_f32(const FcArgs &a, hipStream_t st);
hipError_t launch_fc_reduce(const FcArgs &a, bool bf16, hipStream_t st);

// Input pack: caller NCHW f32 -> NHWC physical channels (bf16 or f32).
hipError_t launch_pack(const EwArgs &a, bool bf16, hipStream_t st);
hipError_t launch_maxpool(const EwArgs &a, bool bf16, hipStream_t st);
hipError_t launch_avgpool(const EwArgs &a, bool bf16, hipStream_t st);
hipError_t launch_upsample2x(const EwArgs &a, bool bf16, hipStream_t st);
hipError_t launch_concat(const EwArgs &a, bool bf16, hipStream_t st);
// Internal NHWC tensor -> caller NCHW f32 output.
hipError_t launch_export(const EwArgs &a, bool bf16, hipStream_t st);

}  // namespace gemel
