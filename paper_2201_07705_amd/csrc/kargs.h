// Kernel argument blocks shared by the host planner and the HIP kernels.
//
// Activations are NHWC with a channel count padded to a multiple of 8
// ("physical" channels; padded channels hold zeros). A merged launch covers
// the concatenated frames of several models: GEMM row m belongs to segment
// s when seg[s].m_start <= m < seg[s+1].m_start, and each segment carries
// its own input, residual, output and scale/shift pointers, so the models'
// tensors can live anywhere while the weight tile is shared by all rows.
#pragma once
#include <stdint.h>

#define GEMEL_MAX_SEG 16
// Bytes of zeros behind ConvArgs::zero (masked-off loads read there, at up
// to a pixel's channel offset).
#define GEMEL_ZERO_PAGE_BYTES 16384

// OUT_NHWC_POOL2: the conv's 2x2 stride-2 max pool fused into its
// epilogue. GEMM rows then run over the output in window order: row
// 4*g + 2*dy + dx of a frame is output pixel (2*hp + dy, 2*wp + dx) of
// pooled pixel g = hp * Wo/2 + wp, and the output tensor is the pooled one
// (Ho/2 x Wo/2 pixels per frame, out_cs channels).
enum { OUT_NHWC = 0, OUT_NCHW_F32 = 1, OUT_PARTIAL_F32 = 2, OUT_NHWC_POOL2 = 3 };

struct ConvSeg {
    const void *in;       // NHWC [frames][H][W][in_cs], frame 0 of the segment
    const void *res;      // NHWC [frames][Ho][Wo][out_cs] or null
    void *out;            // NHWC [frames][Ho][Wo][out_cs] or NCHW f32 final
    const float *scale;   // [N] per output channel
    const float *shift;   // [N]
    int32_t m_start;      // first GEMM row (rows of the earlier segments)
    int32_t f_start;      // first frame of the segment in the launch
    int32_t H, W, Ho, Wo; // the segment's input and output sizes (ConvArgs::hetero)
    const void *w;        // ConvArgs::grouped: this segment's weights [N][K]
    int32_t t_start;      // ConvArgs::grouped: first output tile of the
                          // segment (set by the launcher for its tile shape)
};

struct ConvArgs {
    const void *w;        // [N][K], k = (r * kw + s) * Cin + c
    const void *zero;     // GEMEL_ZERO_PAGE_BYTES zero bytes (target of masked-off loads)
    int32_t M, N, K;      // rows = frames*Ho*Wo, cols = out channels, depth
    int32_t H, W, Cin;    // input spatial size, physical input channels
    int32_t in_cs;        // input pixel stride in elements (>= Cin)
    int32_t Ho, Wo;
    int32_t kh, kw, stride, pad;
    int32_t out_cs;       // output pixel stride (NHWC) in elements
    int32_t cout;         // logical output channels (NCHW f32 stores)
    int32_t act;
    float slope;
    int32_t res_mode;     // 0: act(z + r), 1: act(z) + r
    int32_t has_res;
    int32_t out_mode;     // OUT_NHWC or OUT_NCHW_F32
    int32_t out_pair;     // 0, or (OUT_NHWC) the channel offset at which
                          // the low halves of bf16 (hi, lo) pairs are
                          // stored: hi = bf16(y), lo = bf16(y - hi)
    int32_t nseg;
    int32_t uni_affine;   // every segment uses the same scale/shift arrays
    int32_t hetero;       // 1: segments of different spatial sizes (one weight
                          // copy used at several positions or input sizes):
                          // each row's sizes are its segment's H, W, Ho, Wo,
                          // the launch-wide ones are unused (LDS-DMA kernel,
                          // NHWC output, no fused pool)
    int32_t grouped;      // 1: the segments are separate GEMMs of one shape
                          // (the same layer of several models, each with its
                          // own weights seg[s].w and scale/shift): output
                          // tiles never straddle segments (LDS-DMA kernel)
    int32_t k_splits;     // >1: write fp32 partials to `partial`
    int32_t k_per_split;  // depth handled by one split (multiple of BK)
    float *partial;       // [k_splits][M][N] when k_splits > 1
    int32_t *counters;    // split-K: one arrival counter per output tile,
                          // zero between launches; the last split of a tile
                          // reduces the partials. Null: a separate reduce
                          // launch does.
    uint32_t dv_m[2];     // LDS-DMA kernel (set by its launcher): row n of a
    int32_t dv_l[2];      // frame splits as n / d = (umulhi(n, m) + n) >> l
                          // for d = pixels per frame [0] and per row [1] of
                          // the output (of the pooled output with a fused
                          // pool)
    const void *pf;       // or null: bytes [0, pf_bytes) read (into the
    uint32_t pf_bytes;    // caches) once the tiles are done, the weights of
    int32_t pf_pad;       // the conv that follows on the stream
    ConvSeg seg[GEMEL_MAX_SEG];
};

// Split-K reduction + epilogue over partial sums [splits][M][N].
struct ReduceArgs {
    const float *partial;
    int32_t M, N, splits;
    int32_t HWo;          // rows per frame
    int32_t out_cs, cout;
    int32_t act;
    float slope;
    int32_t res_mode, has_res, out_mode, nseg;
    int32_t out_pair;     // as ConvArgs::out_pair
    ConvSeg seg[GEMEL_MAX_SEG];
};

struct FcSeg {
    const void *in;       // [frames][K] (the producer tensor, NHWC-flat)
    void *out;            // [frames][out_cs] internal, or [frames][cout] f32
    const float *scale, *shift;
    const void *w;        // grouped launch: this segment's weights [N][K]
    int32_t f_start;      // first frame of the segment in the launch
};

struct FcArgs {
    const void *w;        // [N][K]
    int32_t M, N, K;      // frames, out features (physical), in features
    int32_t out_cs, cout;
    int32_t act;
    float slope;
    int32_t out_mode;     // OUT_NHWC (internal) or OUT_NCHW_F32 (final)
    int32_t nseg;
    int32_t k_splits, k_per_split;
    float *partial;       // [k_splits][M][N]
    int32_t *counters;    // split-K: one arrival counter per workgroup
                          // column (64 neurons) and grid slice, as in
                          // ConvArgs
    int32_t grouped;      // bf16 kernel: every segment has its own weights
                          // (seg[i].w; the same N, K and epilogue), one
                          // grid slice (blockIdx.z) per segment
    FcSeg seg[GEMEL_MAX_SEG];
};

struct EwSeg {
    const void *in0;
    const void *in1;
    void *out;
    int32_t frames;
};

// Element-wise / pooling / layout kernels, one segment per model.
struct EwArgs {
    int32_t H, W, C;      // input spatial size and physical channels (in0)
    int32_t C1;           // concat: physical channels of in1
    int32_t Ho, Wo, Co;   // output size and physical channels
    int32_t k, stride, pad;
    int32_t c_logical;    // pack: logical input channels; export: cout
    int32_t nseg;
    int32_t max_frames;
    EwSeg seg[GEMEL_MAX_SEG];
};
