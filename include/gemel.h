/*
 * gemel.h - C ABI of libgemel: batched inference of a workload of vision
 * CNNs whose merged layers keep one weight copy in GPU memory.
 *
 * Model merging (GEMEL, arXiv 2201.07705, Section 4): layers that are
 * architecturally identical across models (same type and same type-specific
 * properties; Section 4.1) may be shared so that a single copy of the
 * layer's definition and weights serves every model that includes it.
 * Layer outputs are never shared, because models may watch different
 * videos. Merging therefore changes where weights live, not what each model
 * computes: a model's outputs after merging equal that model evaluated
 * alone with the shared layers holding the group source's weights.
 *
 * Execution scheme of this library: every merged conv/FC layer runs ONCE
 * over the concatenated frame batches of all active models that share it
 * (one weight read, one launch); unmerged layers run per model. With a
 * weight budget, the weights that do not fit stay in pinned host memory and
 * are copied in on a side stream for every inference round (the paper's
 * edge boxes swap models over PCIe, Section 3.2; Section 5.4 and Appendix
 * A.4 load only layers not already resident and never evict shared ones).
 *
 * General conventions
 *  - Every call returns a gemel_status: 0 on success, a negative code on
 *    failure. No C++ exception and no abort crosses the ABI.
 *  - Host-side validation (pointers, shapes, merge rules) happens before any
 *    HIP call, so invalid arguments never touch the device; on any error the
 *    context is left exactly as it was before the call.
 *  - A context is bound to one device and is not thread-safe: calls on one
 *    context must be serialised by the caller. Separate contexts are
 *    independent.
 *  - gemel_last_error(ctx) returns a NUL-terminated description of the last
 *    failure on ctx (or, with ctx == NULL, of the last gemel_create failure
 *    on this thread). The string is owned by the library.
 */
#ifndef GEMEL_H
#define GEMEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gemel_ctx gemel_ctx;
typedef int32_t gemel_status;

enum {
    GEMEL_OK = 0,
    GEMEL_EINVAL = -1,        /* bad pointer, enum, id or count            */
    GEMEL_ENOMEM = -2,        /* host or device allocation failed          */
    GEMEL_ESHAPE = -3,        /* inconsistent layer or tensor shapes       */
    GEMEL_ENOTMERGEABLE = -4, /* group members not architecturally equal   */
    GEMEL_EBUDGET = -5,       /* weight budget too small to run at all     */
    GEMEL_EDEVICE = -6,       /* HIP runtime / device failure              */
    GEMEL_ESTATE = -7         /* call not valid in the context's state     */
};

/* Arithmetic/storage type of a context. */
enum { GEMEL_F32 = 0, GEMEL_BF16 = 1 };

/* Layer types. */
enum {
    GEMEL_OP_CONV = 0,       /* 2-D convolution (+ optional BN, act, residual) */
    GEMEL_OP_FC = 1,         /* fully connected on the NCHW-flattened input    */
    GEMEL_OP_MAXPOOL = 2,    /* kh x kw window, stride, pad (pad = -inf)       */
    GEMEL_OP_AVGPOOL = 3,    /* global average pool over H x W                 */
    GEMEL_OP_UPSAMPLE2X = 4, /* nearest-neighbour 2x                           */
    GEMEL_OP_CONCAT = 5      /* channels [src0, src1]; both multiples of 8     */
};

enum { GEMEL_ACT_NONE = 0, GEMEL_ACT_RELU = 1, GEMEL_ACT_LEAKY = 2 };

/* Where a residual is added relative to the activation. */
enum {
    GEMEL_RES_ADD_THEN_ACT = 0, /* y = act(z + r)   (ResNet blocks)  */
    GEMEL_RES_ACT_THEN_ADD = 1  /* y = act(z) + r   (Darknet blocks) */
};

/*
 * One layer of a model, in topological order (every producer index is
 * smaller than the layer's own index).
 *
 *  op           GEMEL_OP_*
 *  src0, src1   producer layer index; -1 = the model input. src1 is used by
 *               CONCAT only (must be -1 otherwise).
 *  cin, cout    CONV: input/output channels. FC: flattened input features
 *               (C*H*W of the producer) and output features. Pools,
 *               upsample, concat: cin = producer channels, cout = output
 *               channels.
 *  kh, kw, stride, pad   CONV and MAXPOOL window (kh == kw).
 *  act, act_slope        activation applied by CONV/FC (slope for LEAKY).
 *  res_src, res_mode     CONV only: layer whose output (same shape as this
 *               layer's) is added, -1 = none; GEMEL_RES_*.
 *  is_output    nonzero: the layer's output is returned by gemel_infer.
 *  weight       CONV: float32 [cout][cin][kh][kw] (PyTorch OIHW). FC:
 *               float32 [cout][cin], cin in the producer's NCHW flatten
 *               order. NULL for other ops.
 *  bias         float32 [cout] or NULL.
 *  bn_*         batch norm applied to the conv output: float32 [cout] each,
 *               y = gamma * (z - mean) / sqrt(var + eps) + beta. All four
 *               NULL = no batch norm. CONV only.
 *
 * The library copies every array during gemel_register_model; the caller
 * may free them when the call returns.
 */
typedef struct gemel_layer_desc {
    int32_t op;
    int32_t src0, src1;
    int32_t cin, cout;
    int32_t kh, kw, stride, pad;
    int32_t act;
    float act_slope;
    int32_t res_src, res_mode;
    int32_t is_output;
    const float *weight;
    const float *bias;
    const float *bn_gamma, *bn_beta, *bn_mean, *bn_var;
    float bn_eps;
} gemel_layer_desc;

/* One appearance of a layer: (model id, layer index inside that model). */
typedef struct gemel_member {
    int32_t model_id;
    int32_t layer;
} gemel_member;

/*
 * A group (Section 5.3): all appearances of one layer that share a single
 * copy. members[0] is the weight source; every other member uses its
 * weights, bias and batch norm. The paper seeds a merged group from one
 * member's weights; taking the first member makes the choice deterministic.
 */
typedef struct gemel_group {
    int32_t n_members;
    const gemel_member *members;
} gemel_group;

/*
 * Create a context on HIP device `device`: the GPU memory into which
 * registered models are loaded. When a workload's models do not fit it,
 * they are time-shared by swapping weights in from host memory over PCIe
 * (Section 3.2); the paper evaluates each workload under fixed caps on
 * that memory (Appendix A.3), which hbm_weight_budget stands for.
 *  dtype              GEMEL_F32 (float32 everywhere) or GEMEL_BF16 (bf16
 *                     weights and activations, float32 accumulation and
 *                     epilogue, float32 outputs).
 *  hbm_weight_budget  bytes of device memory that weights may occupy
 *                     (resident copies plus the swap staging buffers);
 *                     0 = unlimited. Weights beyond the budget stay in
 *                     pinned host memory and are streamed in every round.
 * No device memory is touched until the first gemel_infer.
 * Errors: EINVAL (null out, bad dtype, negative device), ENOMEM.
 */
gemel_status gemel_create(gemel_ctx **out, int32_t device, int32_t dtype,
                          uint64_t hbm_weight_budget);

/*
 * Register a model (a DNN supplied with a query, Section 5.1) and copy its
 * weights into the library's host master copy, converted to the kernel
 * layout (bf16 round-to-nearest-even for GEMEL_BF16; conv KRSC; FC columns
 * permuted to the internal NHWC flatten order; batch norm and bias folded
 * into a float32 per-channel scale/shift, never into the weights).
 *  in_c, in_h, in_w   frame shape; frames are float32 NCHW.
 *  *out_model_id      receives the model id (0, 1, 2, ... in call order).
 * Errors: EINVAL (null pointers, bad enums, bad producer index), ESHAPE
 * (channels or sizes inconsistent with the producers), ESTATE.
 */
gemel_status gemel_register_model(gemel_ctx *ctx,
                                  const gemel_layer_desc *layers,
                                  int32_t n_layers, int32_t in_c,
                                  int32_t in_h, int32_t in_w,
                                  int32_t *out_model_id);

/*
 * Install a sharing map: after the call every group's members use one copy
 * of members[0]'s parameters. Replaces the previous map entirely (calling
 * it again with the same groups is a no-op; n_groups == 0 unmerges all).
 * Members must be architecturally identical to members[0] (Section 4.1:
 * same type and type-specific properties: op, cin, cout, kh, kw, stride,
 * pad, bias and batch-norm presence; weights may differ), appear in at most
 * one group, and name registered models and valid layers.
 * Errors: EINVAL, ENOTMERGEABLE (no state change on any error).
 */
gemel_status gemel_merge(gemel_ctx *ctx, const gemel_group *groups,
                         int32_t n_groups);

/*
 * Candidate groups of a workload (Section 5.3, the merging heuristic's first
 * step): every appearance of a parametric layer (CONV, FC) in the models
 * `model_ids`, grouped by architectural identity (exactly the properties
 * gemel_merge checks, so any returned group is accepted by it), each group
 * with the memory its appearances consume in total, and the groups listed
 * in descending order of that memory, so that the groups whose merging
 * would save the most come first. Only groups with at least two
 * appearances are listed (a layer that appears once has nothing to share).
 * The memory of one appearance is its parameter count (weights, plus cout
 * for a bias, plus 4 * cout for batch norm) times the context's element
 * size (2 bytes for GEMEL_BF16, 4 for GEMEL_F32).
 *  model_ids, n_models   distinct registered model ids.
 *  groups, groups_cap    caller array receiving the groups in order; each
 *                        group's members point into `members`.
 *  members, members_cap  caller array receiving all members back to back,
 *                        group after group; within a group in order of the
 *                        model's position in model_ids, then layer index
 *                        (so members[0], the weight source gemel_merge
 *                        uses, is the first appearance).
 *  group_bytes           NULL, or groups_cap int64 receiving each group's
 *                        total memory.
 *  *n_groups, *n_members receive the counts. With groups and members both
 *                        NULL the call only reports the counts.
 * The context is not changed (the current sharing map plays no part).
 * Errors: EINVAL (null counts, bad or repeated model id, arrays smaller
 * than the counts, which are still reported), ENOMEM.
 */
gemel_status gemel_enumerate_groups(gemel_ctx *ctx, const int32_t *model_ids,
                                    int32_t n_models, gemel_group *groups,
                                    int32_t groups_cap, gemel_member *members,
                                    int32_t members_cap, int64_t *group_bytes,
                                    int32_t *n_groups, int32_t *n_members);

/*
 * Run one inference round over `n_models` registered models (the edge
 * box's inference step, Section 3.2: each query's DNN processes its frames;
 * with merging, Section 4, a shared layer is computed from its one stored
 * copy, here once over the concatenated frames of all models that share it,
 * and outputs are those of each model evaluated alone; with a weight budget,
 * only layers that are not resident are loaded, Section 5.4 and Appendix
 * A.4).
 *  model_ids   distinct model ids; their order does not change any output.
 *  frames      per model: device pointer to float32 NCHW
 *              [n_frames[i]][in_c][in_h][in_w].
 *  n_frames    per model frame count (>= 0; 0 skips the model).
 *  outputs     flattened: for each model in model_ids order, one device
 *              pointer per is_output layer in layer order, caller-allocated
 *              float32. Conv outputs are NCHW [n][cout][H][W]; FC outputs
 *              [n][cout] (gemel_output_shape gives the dims).
 *  hip_stream  hipStream_t to enqueue on (NULL = the null stream).
 * Stream-ordered: the call enqueues work and returns; all buffers must stay
 * valid until the stream passes this point. Rounds of one context are
 * ordered among themselves: a round on another stream than the previous
 * round first waits (on the device) for the previous round to finish.
 * Argument errors are returned synchronously without enqueuing anything.
 * A failure part way through enqueuing (EDEVICE) leaves the work already
 * enqueued joined back to hip_stream, so a synchronisation of that stream
 * covers it; an asynchronous device fault surfaces as EDEVICE on this or a
 * later call.
 * Stream capture: a round may be enqueued while hip_stream is being
 * captured into a graph once an earlier round outside capture has placed
 * the weights and built the plan for the same model set and frame counts;
 * the captured round then runs on hip_stream alone (no worker streams,
 * events, allocations or synchronisation), and the caller orders the
 * graph's replays against other rounds. Otherwise, and for rounds that
 * stream weights or are profiled, the call returns ESTATE while capturing.
 * Errors: EINVAL, ESHAPE, ENOMEM, EBUDGET, EDEVICE, ESTATE.
 */
gemel_status gemel_infer(gemel_ctx *ctx, const int32_t *model_ids,
                         int32_t n_models, const void *const *frames,
                         const int32_t *n_frames, void *const *outputs,
                         void *hip_stream);

/*
 * gemel_infer for callers that cannot allocate device memory: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc. Same arguments, outputs and stream ordering as gemel_infer;
 * it calls no hipMalloc, hipFree or other allocating routine. Instead:
 *  - the weights must already be placed on the device (by an earlier
 *    gemel_infer round; since then no merge, registration, budget or
 *    storage option change), else ESTATE;
 *  - the round's activations, split-K partial sums and split-K arrival
 *    counters lie in one static device array of GEMEL_STATIC_SCRATCH_BYTES
 *    (64 MiB) per GPU, held until the process ends; a model set and frame
 *    count whose activations and partial sums exceed it is refused with
 *    EBUDGET (nothing enqueued);
 *  - every launch runs in plan order on hip_stream alone (no worker
 *    stream, event, graph or plan-time tuning), after a fill kernel that
 *    clears the counters (no memset node);
 *  - rounds that would stream weights (a weight budget below the model
 *    set's weights) and profiled rounds are refused with ESTATE.
 * Every call on one GPU shares that GPU's array, from any context: calls
 * whose rounds overlap on the device race, so the caller orders them (one
 * stream, or events). The array keeps the last round's contents.
 * Errors: EINVAL, ESHAPE, ESTATE, EBUDGET, EDEVICE.
 */
gemel_status gemel_infer_noalloc(gemel_ctx *ctx, const int32_t *model_ids,
                                 int32_t n_models, const void *const *frames,
                                 const int32_t *n_frames,
                                 void *const *outputs, void *hip_stream);

/*
 * Models of the round that will follow the next gemel_infer call, for the
 * weight cache (GEMEL_OPT_SWAP_CACHE): their shared layers are not evicted
 * while that call loads its own (Appendix A.4: the scheduler keeps the
 * shared layers needed by the models next in line). n_models == 0 clears
 * the hint. Errors: EINVAL.
 */
gemel_status gemel_set_next_round(gemel_ctx *ctx, const int32_t *model_ids,
                                  int32_t n_models);

/*
 * Sharing-aware load order of a round-robin cycle over `model_ids`
 * (Section 5.4: models that share the most layers are placed next to one
 * another, so each swap loads fewer bytes): start with the model whose
 * stored parameter copies take the most bytes, then repeatedly place the
 * remaining model sharing the most bytes of copies with one end of the
 * order so far at that end (ties: more bytes, lower id, the back end).
 * Bytes are kernel-layout weights rounded up to 256 per copy, under the
 * current sharing map. `order` receives n_models ids. Errors: EINVAL.
 */
gemel_status gemel_load_order(gemel_ctx *ctx, const int32_t *model_ids,
                              int32_t n_models, int32_t *order);

/*
 * Per-model batch sizes of a round-robin schedule under a per-frame
 * deadline (Section 3.2: the time-sharing scheduler's offline profiling
 * picks one global list of per-model batch sizes that maximises the
 * minimum per-model throughput within the SLA, loading the next model
 * while the current one runs; Section 5.4: merging changes those swap
 * delays; Section 6.1: 100 ms). A host computation: no context, no device.
 *
 * cost_ms: [n_models][max_batch] row-major, entry (m, b - 1) the time of
 *   model m on a batch of b frames; each row nondecreasing (as
 *   gemel_profile_batches writes it). swap_ms: [n_models] load time of
 *   model m when its turn comes, or NULL for none.
 * One cycle visits the models once in index order. pipelined != 0: the
 *   next model's load overlaps the current model's inference, a visit takes
 *   max(cost of model i's batch, swap_ms[i + 1 mod n]); pipelined == 0:
 *   swap_ms[i] + cost. T = the sum over the visits (ms).
 * A frame waits at most one cycle for its model's next batch, so the
 *   choice must satisfy T + cost(m, b_m) <= sla_ms for every m. Model m
 *   then processes min(b_m / T, fps) frames/s (fps: its frames arriving per
 *   second). Among batch lists in 1..max_batch, the one returned maximises
 *   the minimum of these over the models; ties go to the shorter cycle,
 *   then to the smaller batches (it is componentwise the smallest list
 *   reaching the optimum).
 * Outputs: batch[n_models]; min_fps and cycle_ms (either may be NULL).
 * Errors: EINVAL (sizes, null cost/batch, non-finite or negative entries,
 * a decreasing row, sla_ms or fps not positive); EBUDGET when batches of
 * one frame already miss the deadline. Outputs are untouched on error.
 */
gemel_status gemel_sla_batches(int32_t n_models, int32_t max_batch,
                               const double *cost_ms, const double *swap_ms,
                               int32_t pipelined, double sla_ms, double fps,
                               int32_t *batch, double *min_fps,
                               double *cycle_ms);

/*
 * Measures the cost table gemel_sla_batches takes (Section 3.2's offline
 * profiling): for each listed model and each batch b in 1..max_batch, a
 * round of that model alone on b frames (zeroed buffers the call
 * allocates), after untimed rounds that build and tune its plan, then
 * `reps` rounds timed one by one with HIP events on hip_stream (null: the
 * default stream; not captured); entry (i, b - 1) of cost_ms ([n_models][max_batch]) is the
 * largest median over batches 1..b, so rows are nondecreasing. The call
 * is synchronous, runs rounds like gemel_infer (same options, budget and
 * weight cache), frees its buffers and drops every plan it built (the
 * next gemel_infer builds its plan again). max_batch in 1..4096, reps in
 * 1..1000. Errors: EINVAL, ESTATE (stream captured), ENOMEM, EDEVICE and
 * those of gemel_infer.
 */
gemel_status gemel_profile_batches(gemel_ctx *ctx, const int32_t *model_ids,
                                   int32_t n_models, int32_t max_batch,
                                   int32_t reps, void *hip_stream,
                                   double *cost_ms);

/* Number of output layers of a model. Errors: EINVAL. */
gemel_status gemel_model_outputs(gemel_ctx *ctx, int32_t model_id,
                                 int32_t *n_outputs);

/*
 * Shape of output `output_idx` of a model for `n_frames` frames: dims =
 * {n, C, H, W} for conv-type outputs, {n, C, 1, 1} for FC outputs.
 * Errors: EINVAL.
 */
gemel_status gemel_output_shape(gemel_ctx *ctx, int32_t model_id,
                                int32_t output_idx, int32_t n_frames,
                                int64_t dims[4]);

/* Keys of gemel_query. Byte counts are device bytes of stored parameters
 * (weights in kernel layout plus float32 scale/shift). */
enum {
    GEMEL_Q_UNMERGED_BYTES = 0, /* all registered layers, nothing shared  */
    GEMEL_Q_MERGED_BYTES = 1,   /* one copy per merged group              */
    GEMEL_Q_RESIDENT_BYTES = 2, /* weights kept resident in device memory */
    GEMEL_Q_PEAK_BYTES = 3,     /* high-water mark: resident + staging    */
    GEMEL_Q_STREAMED_BYTES = 4, /* host->device weight bytes per round    */
    GEMEL_Q_ACTIVATION_BYTES = 5, /* activation arena of the last plan    */
    GEMEL_Q_LAUNCHES = 6,       /* kernel launches per round, last plan   */
    GEMEL_Q_N_MODELS = 7,       /* registered models                      */
    GEMEL_Q_GRAPH_REPLAYS = 8,  /* rounds served by a replayed HIP graph  */
    GEMEL_Q_STREAMS = 9,        /* GEMEL_OPT_STREAMS now in force         */
    GEMEL_Q_ROUND_MODE = 10,    /* how the last round ran: 0 enqueued
                                   directly, 1 per-stream chain graphs,
                                   2 one graph with data edges, 3 one graph
                                   with data edges and stream order, 4 on
                                   the caller's stream alone (a round
                                   enqueued while that stream was being
                                   captured)                             */
    GEMEL_Q_ROUND_TUNING = 11,  /* rounds the last plan's round-mode tuner
                                   (GEMEL_OPT_AUTOTUNE) still runs before
                                   its choice is fixed; 0 = settled      */
    GEMEL_Q_ROUND_LOADED_BYTES = 12,  /* weight cache: bytes the last round
                                   loaded into the cache                 */
    GEMEL_Q_ROUND_EVICTED_BYTES = 13, /* weight cache: bytes it evicted   */
    GEMEL_Q_CACHED_BYTES = 14,  /* weight cache: bytes cached after it    */
    GEMEL_Q_CACHE_CAPACITY = 15,/* weight cache: its capacity (the weight
                                   budget minus the resident scale/shift
                                   vectors), 0 without the cache         */
    GEMEL_Q_PREFETCHES = 16     /* conv launches of the last plan that
                                   prefetch the next conv's weights
                                   (GEMEL_OPT_PREFETCH)                  */
};

/* Read a counter. Errors: EINVAL (unknown key, null val). */
gemel_status gemel_query(gemel_ctx *ctx, int32_t key, int64_t *val);

/* Tunables and test hooks of gemel_set_option. */
enum {
    GEMEL_OPT_USE_GRAPH = 0,     /* 1 (default): a round without streamed
                                    weights is replayed as a HIP graph
                                    (built once per frames/outputs pointer
                                    set and stream, edges as set by
                                    GEMEL_OPT_GRAPH_DAG); 0: rounds are
                                    enqueued directly                      */
    GEMEL_OPT_SWAP_SLOT_BYTES = 1, /* staging slot size (default 32 MiB)   */
    GEMEL_OPT_SWAP_SLOTS = 2,    /* number of staging slots (default 3)    */
    GEMEL_OPT_FAIL_COPY_AT = 3,  /* test hook: the n-th (1-based) swap copy
                                    issued from now fails; 0 = off         */
    GEMEL_OPT_SPLIT_MERGED = 4,  /* 1: run merged layers per model (one
                                    launch per member, same single weight
                                    copy); 0 (default): one launch         */
    GEMEL_OPT_WEIGHT_BUDGET = 5, /* replace the hbm_weight_budget given to
                                    gemel_create (bytes, 0 = unlimited)    */
    GEMEL_OPT_PROFILE = 6,       /* 1: time every kernel launch with HIP
                                    events bound to the kernel's own start
                                    and end (hipExtLaunchKernel; disables
                                    graph replay); 0 (default): off. Setting
                                    it clears the collected statistics.    */
    GEMEL_OPT_CONV_TILE = 7,     /* -1 (default): pick each conv's tile
                                    shape and split-K by the cost model;
                                    0..19: force one tile shape (128x128,
                                    128x64, 64x64, 256x256, 256x128,
                                    256x64, 64x64 and 128x64 with deeper
                                    prefetch, 64x128; then the LDS-DMA
                                    pipeline's 256x256, 256x128, 128x128,
                                    128x64, used where Cin % 32 == 0; 13:
                                    the 8-channel stem kernel, used where
                                    the input has 8 physical channels and
                                    without split-K; 14..17: the LDS-DMA
                                    pipeline with depth steps of 64,
                                    256x256, 256x128, 128x128, 128x64, used
                                    where Cin % 64 == 0; 18, 19: LDS-DMA
                                    64x64 of depth 32 and 64; 20..23:
                                    LDS-DMA of depth 32 with a 64x64 tile
                                    per wave, 256x128 and 128x256 of 8
                                    waves, 256x64 and 64x256 of 4) with
                                    split-K still chosen. A forced tile a
                                    conv cannot use falls back to 64x64    */
    GEMEL_OPT_CONV_SPLITS = 8,   /* 0 (default): split-K chosen per conv;
                                    n >= 1: force n depth splits (capped
                                    so that every split has work)          */
    GEMEL_OPT_STREAMS = 9,       /* 1..8 (default 3): at most this many
                                    streams carry a round (forked from and
                                    joined to the caller's stream; 1 with
                                    the null stream). A branch of the
                                    layer graph gets a stream of its own
                                    when the work only it leads to is worth
                                    the fork; cross-stream dependencies are
                                    event waits                            */
    GEMEL_OPT_GRAPH_DAG = 10,    /* graph rounds over several streams with
                                    autotune off: 0 (default): the launches
                                    of each stream are cut where a cross-
                                    stream wait or event record falls, and
                                    each piece is a chain-shaped graph
                                    launched on its stream (with the
                                    round's fork, joins and events between
                                    pieces); 1: one graph whose nodes
                                    follow only the launches whose results
                                    they read (activation bytes are reused
                                    only along such dependencies)          */
    GEMEL_OPT_FORK_US = 11,      /* a branch gets a stream of its own when
                                    the work only it leads to is estimated
                                    at this many microseconds or more
                                    (default 12), or spans 3 or more
                                    launch steps                           */
    GEMEL_OPT_AUTOTUNE = 12,     /* 1 (default): the first 20 rounds of a
                                    graphable plan over several streams try
                                    the two graph forms of GEMEL_OPT_GRAPH_DAG,
                                    one graph with data edges plus each
                                    stream's order, and direct enqueue: one
                                    untimed round of each, then 4 timed
                                    rounds of each, interleaved, timing
                                    each round with
                                    HIP events on the caller's stream (the
                                    timed rounds synchronise with it), and
                                    later rounds use the one with the
                                    smallest median. Skipped
                                    while the caller's stream is being
                                    captured. 0: the mode set by
                                    GEMEL_OPT_GRAPH_DAG                    */
    GEMEL_OPT_SPLITK_FUSED = 13, /* how split-K layers reduce their fp32
                                    partial sums: 1 (default) inside the
                                    GEMM launch (the last split of each
                                    output tile to finish sums the tile and
                                    applies the epilogue) for FC layers and
                                    for convs of 256 output tiles or more,
                                    else in a separate reduction launch;
                                    2: inside the GEMM launch always; 0: in
                                    a separate launch always. Every form
                                    sums in split order: same bits         */
    GEMEL_OPT_TUNE = 14,         /* 1 (default): when a plan is built, each
                                    bf16 conv shape whose tile and split-K
                                    are not forced (and whose weights are
                                    resident and whose output is internal)
                                    times the cost model's best estimated
                                    configurations (up to 4, those within
                                    2x of the best estimate) on the device
                                    and keeps the fastest; choices are kept
                                    for the context's life. Not while the
                                    caller's stream is being captured. 0:
                                    the cost model alone; 2..16: as 1, up
                                    to that many candidates. Different
                                    choices change fp32 summation order,
                                    so bits may differ between contexts    */
    GEMEL_OPT_FUSE_POOL = 15,    /* 1 (default): a bf16 conv whose only
                                    consumer is a 2x2 stride-2 max pool
                                    (even output size, no residual, not an
                                    output, input channels a multiple of
                                    32) writes the pooled tensor from its
                                    epilogue, and the pool launch and the
                                    full-size tensor disappear. Results are
                                    bit-identical to the separate pool. 0:
                                    off                                    */
    GEMEL_OPT_MIXED_SIZES = 16,  /* 1 (default): members of a merged group
                                    whose inputs differ in spatial size
                                    (one weight copy at several positions
                                    or input sizes) run as one launch whose
                                    segments keep their own sizes, where
                                    the conv takes the LDS-DMA kernel (bf16,
                                    input channels a multiple of 32,
                                    internal output, no fused pool). 0: one
                                    launch per size                        */
    GEMEL_OPT_PAIRED_ACTS = 17,  /* bf16 contexts: 1 = a tensor written by
                                    an unmerged conv (not an output, not a
                                    residual, input wider than 8 channels)
                                    and read only by unmerged convs, either
                                    directly or through upsample / concat,
                                    is stored as pairs of bf16 (hi =
                                    bf16(y), lo = bf16(y - hi)), and each
                                    conv reading it multiplies both halves
                                    by its weights (stored twice along the
                                    input channels), so those activations
                                    keep about 16 significant bits instead
                                    of 8 (deep per-model chains, e.g.
                                    detection heads, then drift less from
                                    the float32 result). Costs twice the
                                    bytes of those tensors and twice the
                                    MFMA work of their consumers. 0
                                    (default): bf16 activations            */
    GEMEL_OPT_FAIL_ALLOC_AT = 18,/* test hook: the n-th (1-based) device or
                                    pinned-host allocation the library makes
                                    from now fails as if out of memory (the
                                    call reports ENOMEM, or, for the scratch
                                    of plan-time tuning, skips that tuning);
                                    0 = off                                */
    GEMEL_OPT_GROUP_UNMERGED = 19,/* 1 (default): an unmerged bf16 conv that
                                    appears with the same shape and epilogue
                                    in several active models (their k-th such
                                    layer each, e.g. per-model heads of one
                                    architecture) runs as ONE grouped launch
                                    whose segments keep their own weights and
                                    scale/shift (output tiles never straddle
                                    two segments), where the LDS-DMA kernel
                                    can take it and the weights are resident.
                                    Results are those of separate launches
                                    of the same tile configuration. 0: one
                                    launch per model                       */
    GEMEL_OPT_SWAP_CACHE = 20,   /* with a weight budget: 1 = time-shared
                                    rounds over subsets of the models keep
                                    a weight cache across rounds (Section
                                    5.4: loading a model brings in only its
                                    layers not already in GPU memory;
                                    Appendix A.4: layers shared by the
                                    models of the current or next round are
                                    never evicted). The scale/shift vectors
                                    stay resident and the rest of the
                                    budget is the cache; every weight blob
                                    waits in pinned host memory. A round
                                    loads the blobs its models need that
                                    are not cached, in first-use order
                                    (models by id, then layers), each
                                    first-fit at the lowest 256-byte-aligned
                                    offset with room, after evicting, while
                                    none has room, cached blobs that are
                                    not pinned: unshared before shared,
                                    larger before smaller, then the blob
                                    first used earlier (models by id, then
                                    layers). Pinned: the round's blobs and the
                                    shared blobs of the models named by
                                    gemel_set_next_round. Copies run on a
                                    side stream after the previous round's
                                    work and each launch waits only for its
                                    own weights' copy. A round whose pinned
                                    blobs exceed the cache returns EBUDGET
                                    and changes nothing. Rounds are not
                                    graphed or captured. 0 (default): the
                                    budget keeps the largest blobs (merged
                                    ones first) resident and streams the
                                    rest through staging slots every round */
    GEMEL_OPT_PREFETCH = 21      /* 1 (default): in a round that moves more
                                    bytes than the GPU's 256 MiB memory-side
                                    cache holds, an LDS-DMA conv launch,
                                    after its own tiles, reads the resident
                                    weights (up to 16 MiB) of the next conv
                                    launch of its stream into the L2 and
                                    memory-side caches, so that launch's
                                    depth loop starts on cache hits instead
                                    of HBM reads (ungrouped, resident
                                    weights only). Results are unchanged.
                                    2: in every round; 0: no prefetch      */
};

/* Set an option; takes effect at the next gemel_infer. Errors: EINVAL. */
gemel_status gemel_set_option(gemel_ctx *ctx, int32_t key, int64_t value);

/* Kernel families reported by gemel_profile. */
enum {
    GEMEL_K_CONV_MFMA = 0,   /* bf16 implicit-GEMM convolution (MFMA)       */
    GEMEL_K_CONV_F32 = 1,    /* fp32 direct convolution                     */
    GEMEL_K_SPLITK_REDUCE = 2, /* split-K reduction + epilogue (conv, FC)   */
    GEMEL_K_FC = 3,          /* weight-streaming fully connected            */
    GEMEL_K_PACK = 4,        /* NCHW f32 frames -> NHWC                     */
    GEMEL_K_POOL = 5,        /* max and global average pooling              */
    GEMEL_K_ROUTE = 6,       /* upsample and concat                         */
    GEMEL_K_EXPORT = 7,      /* internal tensor -> NCHW f32 output          */
    GEMEL_K_CONV_MERGED = 8, /* the GEMEL_K_CONV_MFMA launches that run a
                                merged layer over the frames of several
                                models (a subset: also counted in
                                GEMEL_K_CONV_MFMA)                          */
    GEMEL_K_COUNT = 9
};

/* Per-round statistics of one kernel family, averaged over the rounds run
 * with GEMEL_OPT_PROFILE on. flops and bytes are algorithmic: 2 x MAC of
 * the logical (unpadded) layer shapes, and every weight, input, residual
 * and output byte counted once. */
typedef struct gemel_kernel_stat {
    int32_t kind;        /* GEMEL_K_*                                       */
    int32_t launches;    /* launches per round                              */
    double flops;        /* algorithmic FLOPs per round                     */
    double bytes;        /* algorithmic bytes per round                     */
    double ms;           /* summed kernel time per round (HIP events on
                            each kernel's own start and end)                */
} gemel_kernel_stat;

/*
 * Read the profile: stats must hold GEMEL_K_COUNT entries (one per family,
 * in GEMEL_K_* order); *rounds receives the number of profiled rounds the
 * averages cover. Waits for the profiled rounds to finish on the device.
 * Errors: EINVAL (null pointers), ESTATE (profiling never enabled), EDEVICE.
 */
gemel_status gemel_profile(gemel_ctx *ctx, gemel_kernel_stat *stats,
                           int32_t *rounds);

/* Description of the last error (see general conventions). */
const char *gemel_last_error(const gemel_ctx *ctx);

/* Synchronise the device, free all device and host resources. ctx may be
 * NULL. Errors: EDEVICE if a pending device fault is found (resources are
 * released regardless). */
gemel_status gemel_destroy(gemel_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* GEMEL_H */
