// Internal state of a gemel context: registry of models and parameter
// blobs, device placement of the weights, and cached execution plans.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <map>
#include <memory>
#include <string>
#include <vector>

#include "gemel.h"
#include "kargs.h"
#include "kernels.h"

namespace gemel {

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// One stored copy of a conv/FC layer's parameters in kernel layout:
// weights [rows][k] (rows = physical output channels, k = kh*kw*cin_p for a
// conv, producer NHWC-flat size for an FC) and fp32 scale/shift [rows]
// holding bias and batch norm folded together.
struct Blob {
    int64_t rows = 0, k = 0;
    size_t elem = 2;                 // bytes per weight element
    std::vector<uint8_t> w;          // host master copy
    std::vector<float> scale, shift;
    size_t w_bytes() const { return w.size(); }
    size_t aff_bytes() const { return 2 * scale.size() * sizeof(float); }
    size_t bytes() const { return w_bytes() + aff_bytes(); }
    // placement (valid while the context's weights are materialised)
    void *w_dev = nullptr;           // resident weights, null if streamed
    float *aff_dev = nullptr;        // scale[rows] then shift[rows], resident
    uint8_t *w_pinned = nullptr;     // pinned host copy of a streamed blob
    int users = 0;                   // registered layers using this copy
    // weight cache (GEMEL_OPT_SWAP_CACHE): number in placement order, offset
    // in the cache (-1: not cached), event recorded after its last load
    int index = -1;
    int64_t cache_off = -1;
    hipEvent_t ev_loaded = nullptr;
    int loaded_round = -1;           // round of the last load
    int used_round = -1;             // last round that needed it
};

struct Layer {
    int op = 0, src0 = -1, src1 = -1, cin = 0, cout = 0, kh = 1, kw = 1;
    int stride = 1, pad = 0, act = 0, res = -1, res_mode = 0, is_output = 0;
    float slope = 0.f;
    bool has_bias = false, has_bn = false;
    int in_c = 0, in_h = 0, in_w = 0, in_cp = 0;  // src0 tensor
    int src1_cp = 0;                              // concat: src1 channels
    int out_c = 0, out_h = 0, out_w = 0, out_cp = 0;
    std::shared_ptr<Blob> own;   // this layer's own parameters
    std::shared_ptr<Blob> eff;   // parameters in use (own or a group source's)
    int group = -1;              // index of the merge group containing it
    int out_index = -1;          // position among the model's outputs
    int consumers = 0;           // layers that read this layer's output
    // storage of the tensors (assign_layouts, with the weight placement):
    // physical channels per pixel of the src0 / src1 / output tensors, and
    // whether the output holds bf16 (hi, lo) pairs: hi in channels
    // [0, out_cp), lo in [out_cp, 2 * out_cp)
    int in_phys = 0, src1_phys = 0, out_phys = 0;
    bool out_paired = false;
    std::shared_ptr<Blob> exec;  // parameters as the kernels read them: eff,
                                 // or eff gathered to a paired input's channels
};

struct Model {
    int id = 0;
    int in_c = 0, in_h = 0, in_w = 0, in_cp = 0;
    std::vector<Layer> layers;
    std::vector<int> outputs;    // layer indices of the outputs
};

// A caller pointer patched into an argument block at every call.
struct Patch {
    enum Kind { FRAMES = 0, OUTPUT = 1 } kind;
    int slot;        // model slot within the plan
    int out_idx;     // output number (OUTPUT)
    int seg;         // segment index inside the argument block
};

enum LaunchType {
    L_PACK, L_CONV_BF16, L_CONV_F32, L_CONV_REDUCE, L_FC_BF16, L_FC_F32, L_FC_REDUCE,
    L_MAXPOOL, L_AVGPOOL, L_UPSAMPLE, L_CONCAT, L_EXPORT
};

struct Launch {
    LaunchType type;
    int tile = 0;
    bool bf16 = true;
    // kernel family (GEMEL_K_*) and algorithmic work of this launch
    int kind = 0;
    bool merged = false;  // runs a merged layer over several models' frames
    double flops = 0, bytes = 0;
    ConvArgs conv{};
    ReduceArgs red{};
    FcArgs fc{};
    EwArgs ew{};
    std::vector<Patch> patches;
    // weight streaming: >= 0 when the weights come from a staging slot
    int chunk = -1;
    // weight cache: the blob(s) whose current cache address the launch
    // reads (one per segment for a grouped launch, else one)
    std::vector<Blob *> wblobs;
    int ctr_n = 0;  // arrival counters of a fused split-K launch
    // concurrency: stream index, plan events waited for before the launch,
    // plan event recorded after it (-1 = none)
    int stream = 0;
    std::vector<int> waits;
    int record = -1;
    // plan step (layer node or export) the launch belongs to, and the
    // launches it must follow: the last launch of each producer step (the
    // input packs for a step reading a model input), or the previous launch
    // of its own step
    int step = -1;
    std::vector<int> deps;
};

// A chunk of a streamed blob: weight rows [row0, row0 + nrows).
struct Chunk {
    Blob *blob;
    int64_t row0, nrows;
    size_t bytes() const { return (size_t)(nrows * blob->k) * blob->elem; }
};

// A run of one stream's launches with cross-stream waits only before its
// first launch and an event record only after its last: one chain-shaped
// HIP graph, launched on its stream.
struct Segment {
    int stream = 0;
    std::vector<int> launches;
    std::vector<int> waits;   // plan events waited for before the segment
    int record = -1;          // plan event recorded after it
    hipGraphExec_t exec = nullptr;
};

struct Plan {
    std::vector<int> model_ids, n_frames;  // active models (key)
    std::vector<int> out_base;             // first output index per slot
    std::vector<Launch> launches;          // input packs first, then steps
    int n_pack = 0;                        // launches before the fork
    int n_streams = 1;                     // streams the launches use
    std::vector<hipEvent_t> events;        // cross-stream dependencies
    hipEvent_t ev_fork = nullptr;          // origin -> worker streams
    std::vector<hipEvent_t> ev_join;       // worker streams -> origin
    std::vector<Chunk> chunks;             // streamed chunks, consumption order
    // Streamed chunks packed in consumption order into one pinned host image,
    // cut into copy segments of at most one staging slot each (a chunk never
    // straddles two): one copy per segment per round. Built at the plan's
    // first round.
    struct CopySeg {
        size_t off, bytes;                 // in the image
    };
    void *image = nullptr;
    std::vector<CopySeg> copy_segs;
    std::vector<int> chunk_seg;            // segment of each chunk
    std::vector<size_t> chunk_off;         // its offset in the segment (and slot)
    std::vector<hipEvent_t> ev_chunk;      // recorded after each chunk's consumer
    void *arena = nullptr;
    size_t arena_bytes = 0;
    // split-K partial sums: one region per split-K step; steps that may run
    // concurrently get disjoint regions
    float *partial = nullptr;
    size_t partial_bytes = 0;
    // arrival counters of the fused split-K reductions, a disjoint range per
    // launch (never shared: a counter must read zero when its launch starts)
    int32_t *counters = nullptr;
    size_t counters_n = 0;                 // ints in `counters`
    // arena, partial sums and counters carved from the static scratch
    // (gemel_infer_noalloc): never freed; counters cleared every round
    bool static_mem = false;
    size_t streamed_bytes = 0;
    // HIP graphs of the round for one set of caller pointers: one chain per
    // segment; one graph whose edges are the launches' data dependencies; one
    // graph with those edges plus each plan stream's order
    std::vector<Segment> segs;
    hipGraphExec_t graph[2] = {nullptr, nullptr};
    // execution mode of a multi-stream graphable plan, chosen by timing
    // each candidate over its first rounds (autotune)
    int tune_round = 0;
    double tune_ms[4][4] = {};   // timed rounds of each candidate mode
    int best_mode = -1;
    hipEvent_t tune_ev[2] = {nullptr, nullptr};
    std::vector<const void *> graph_frames;
    std::vector<void *> graph_outputs;
    hipStream_t graph_stream = nullptr;
};

// Per-launch timing with HIP events (GEMEL_OPT_PROFILE).
struct Profile {
    struct Rec {
        hipEvent_t a, b;
        int kind;
        int subset;   // GEMEL_K_CONV_MERGED for merged convs, else -1
    };
    std::vector<hipEvent_t> pool;    // free events
    std::vector<Rec> pending;        // recorded, not yet read
    double ms[GEMEL_K_COUNT] = {}, flops[GEMEL_K_COUNT] = {}, bytes[GEMEL_K_COUNT] = {};
    int64_t launches[GEMEL_K_COUNT] = {};
    int rounds = 0;
    bool used = false;
};

struct Options {
    int streams = 3;
    int profile = 0;
    int conv_tile = -1;
    int conv_splits = 0;
    int use_graph = 1;
    int graph_dag = 0;
    int autotune = 1;
    int fork_us = 12;
    int splitk_fused = 1;
    int tune = 1;             // measured conv configuration at plan time
    int tune_candidates = 4;  // configurations timed per conv shape
    int fuse_pool = 1;        // 2x2 max pools fused into their conv
    int mixed_sizes = 1;      // merged members of different sizes in one launch
    int64_t slot_bytes = 32ll << 20;
    int slots = 3;
    int64_t fail_copy_at = 0;
    int64_t fail_alloc_at = 0;
    int split_merged = 0;
    int paired_acts = 0;      // unmerged conv chains keep bf16 (hi, lo) pairs
    int group_unmerged = 1;   // same-shape unmerged convs of several models: one launch
    int swap_cache = 0;       // weights cached across rounds (with a budget)
    int prefetch = 1;         // conv launches read the next conv's weights into the caches (2: in any round)
};

}  // namespace gemel

struct gemel_ctx {
    int device = 0;
    int dtype = GEMEL_BF16;
    uint64_t budget = 0;
    std::vector<std::unique_ptr<gemel::Model>> models;
    std::vector<std::vector<gemel_member>> groups;
    gemel::Options opt;
    std::string err;
    // device state
    bool dev_ready = false;
    bool weights_ready = false;      // placement matches registry + groups
    hipStream_t side = nullptr;      // weight-copy stream
    std::vector<hipStream_t> workers;  // extra streams for concurrent steps
    std::vector<hipEvent_t> ev_copied, ev_free;
    // per staging slot: for each stream, the event of the last consumer on
    // it of the segment that last used the slot (the next copy into the
    // slot waits for all of them)
    std::vector<std::vector<std::pair<hipStream_t, hipEvent_t>>> slot_users;
    void *wpool = nullptr;           // resident weights + all scale/shift
    void *zero_page = nullptr;       // GEMEL_ZERO_PAGE_BYTES zero bytes inside wpool
    size_t wpool_bytes = 0;
    void *staging = nullptr;         // slots x slot_bytes
    int staging_slots = 0;
    int64_t staging_slot_bytes = 0;
    std::vector<std::shared_ptr<gemel::Blob>> placed;  // blobs of the pool
    size_t resident_bytes = 0, peak_bytes = 0;
    int64_t copies_issued = 0;
    int64_t allocs_issued = 0;
    int64_t graph_replays = 0;
    int last_mode = 0;   // execution mode of the last round (GEMEL_Q_ROUND_MODE)
    int tuning_left = 0; // rounds the last plan's round-mode tuner still runs
    // ordering between rounds: ev_round_done is recorded on a round's stream
    // after its last work; a round on another stream first waits for it
    hipEvent_t ev_round_done = nullptr;
    hipStream_t round_stream = nullptr;
    bool round_seen = false;
    hipEvent_t ev_side_join = nullptr;   // side stream -> caller after a failed round
    // weight cache across rounds (GEMEL_OPT_SWAP_CACHE with a budget): the
    // cache's device bytes, the models of the next round (their shared
    // blobs stay cached), and the last round's load statistics
    bool cache_mode = false;
    char *cache_base = nullptr;
    size_t cache_cap = 0;
    int cache_round = 0;
    // end of the last two cache rounds (slot r % 2 holds round
    // cache_done_round[r % 2]): a copy waits only for the rounds that last
    // used the bytes it overwrites, so the next round's loads can overlap
    // the current round's compute
    hipEvent_t ev_cache_done[2] = {nullptr, nullptr};
    int cache_done_round[2] = {-1, -1};
    // cache bytes freed by evictions and the last round that used them
    struct Freed {
        int64_t off, size;
        int round;
    };
    std::vector<Freed> cache_freed;
    std::vector<int> next_models;
    int64_t round_loaded = 0, round_evicted = 0;
    std::map<std::vector<int>, std::unique_ptr<gemel::Plan>> plans;
    gemel::Plan *last_plan = nullptr;
    gemel::Profile prof;
    // plan-time conv tuning: chosen (tile, splits) per conv shape, and the
    // stream, events and scratch the timing runs use
    std::map<std::vector<int64_t>, std::pair<int, int>> tune_cache;
    hipStream_t tune_stream = nullptr;
    hipEvent_t tune_ev[2] = {nullptr, nullptr};
    void *tune_partial = nullptr;
    size_t tune_partial_bytes = 0;
    void *tune_ctr = nullptr;
    size_t tune_ctr_bytes = 0;
    void *tune_w = nullptr;   // stand-in weights while the weight cache is on
    size_t tune_w_bytes = 0;
};

namespace gemel {
gemel_status fail(gemel_ctx *ctx, gemel_status code, const std::string &msg);
gemel_status materialise(gemel_ctx *ctx);
void release_device(gemel_ctx *ctx);
void drop_plans(gemel_ctx *ctx);
gemel_status run(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                 const void *const *frames, const int32_t *n_frames, void *const *outputs,
                 hipStream_t stream);
gemel_status run_noalloc(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                         const void *const *frames, const int32_t *n_frames, void *const *outputs,
                         hipStream_t stream);
size_t unmerged_bytes(const gemel_ctx *ctx);
// hipMalloc, counted for GEMEL_OPT_FAIL_ALLOC_AT
hipError_t alloc_device(gemel_ctx *ctx, void **p, size_t bytes);
void profile_reset(gemel_ctx *ctx);
gemel_status profile_read(gemel_ctx *ctx, gemel_kernel_stat *stats, int32_t *rounds);
size_t merged_bytes(const gemel_ctx *ctx);
}  // namespace gemel
