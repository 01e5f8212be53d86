// Device placement of weights, execution plans and the inference round.
//
// Placement (materialise): every distinct parameter copy in use (one per
// merged group, one per unmerged layer) is either resident in one device
// pool or, when a weight budget does not fit, kept in pinned host memory
// and streamed through a ring of staging slots every round. Merged copies
// are made resident first: they serve several models (the paper's edge
// scheduler never evicts layers still needed by other models, Appendix
// A.4); the remaining budget is filled largest-first.
//
// Plan: for one set of (model, frame count) the layers of all models
// become launch nodes. The members of a merge group that agree on input
// shape and epilogue form ONE node (one launch over their concatenated
// frames, reading the single shared weight copy); every other layer is a
// node of its own. Nodes run in a topological order of their dependencies.
// Activations live in one arena whose offsets are assigned from tensor
// lifetimes (tensors whose lifetimes overlap never share bytes).
//
// Round: the plan's launches are enqueued on the caller's stream (or a HIP
// graph of them, whose edges are the launches' data dependencies, is
// replayed). Streamed weights are copied on a side stream: copy i waits for
// the consumer of the chunk that last used its slot, and consumer i waits
// for copy i.
#include <algorithm>
#include <functional>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <numeric>
#include <queue>
#include <set>

#include "internal.h"

namespace gemel {

#define HIPCHK(call, what)                                                                   \
    do {                                                                                     \
        hipError_t e_ = (call);                                                              \
        if (e_ != hipSuccess)                                                                \
            return fail(ctx, GEMEL_EDEVICE, std::string(what) + ": " + hipGetErrorString(e_)); \
    } while (0)

// Device and pinned-host allocations of the library, counted so that a
// test can make the n-th one fail (GEMEL_OPT_FAIL_ALLOC_AT).
hipError_t alloc_device(gemel_ctx *ctx, void **p, size_t bytes) {
    ctx->allocs_issued++;
    if (ctx->opt.fail_alloc_at && ctx->allocs_issued == ctx->opt.fail_alloc_at) {
        ctx->opt.fail_alloc_at = 0;
        *p = nullptr;
        return hipErrorOutOfMemory;
    }
    return hipMalloc(p, bytes);
}
static hipError_t alloc_pinned(gemel_ctx *ctx, void **p, size_t bytes) {
    ctx->allocs_issued++;
    if (ctx->opt.fail_alloc_at && ctx->allocs_issued == ctx->opt.fail_alloc_at) {
        ctx->opt.fail_alloc_at = 0;
        *p = nullptr;
        return hipErrorOutOfMemory;
    }
    return hipHostMalloc(p, bytes, hipHostMallocDefault);
}

namespace {

struct DeviceScope {
    int prev = -1;
    explicit DeviceScope(int d) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        (void)hipSetDevice(d);
    }
    ~DeviceScope() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

gemel_status ensure_device(gemel_ctx *ctx) {
    if (ctx->dev_ready) return GEMEL_OK;
    int n = 0;
    HIPCHK(hipGetDeviceCount(&n), "hipGetDeviceCount");
    if (ctx->device >= n) return fail(ctx, GEMEL_EINVAL, "device index beyond the visible devices");
    HIPCHK(hipSetDevice(ctx->device), "hipSetDevice");
    hipDeviceProp_t prop;
    HIPCHK(hipGetDeviceProperties(&prop, ctx->device), "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(ctx, GEMEL_EDEVICE, std::string("libgemel is built for gfx950; device is ") + prop.gcnArchName);
    HIPCHK(hipStreamCreateWithFlags(&ctx->side, hipStreamNonBlocking), "hipStreamCreate");
    for (int i = 0; i < 7; ++i) {
        hipStream_t w = nullptr;
        HIPCHK(hipStreamCreateWithFlags(&w, hipStreamNonBlocking), "hipStreamCreate");
        ctx->workers.push_back(w);
    }
    HIPCHK(hipEventCreateWithFlags(&ctx->ev_round_done, hipEventDisableTiming), "hipEventCreate");
    HIPCHK(hipEventCreateWithFlags(&ctx->ev_side_join, hipEventDisableTiming), "hipEventCreate");
    ctx->round_seen = false;
    ctx->round_stream = nullptr;
    ctx->dev_ready = true;
    return GEMEL_OK;
}

void free_placement(gemel_ctx *ctx) {
    for (auto &b : ctx->placed) {
        if (b->w_pinned) (void)hipHostFree(b->w_pinned);
        if (b->ev_loaded) (void)hipEventDestroy(b->ev_loaded);
        b->w_pinned = nullptr;
        b->w_dev = nullptr;
        b->aff_dev = nullptr;
        b->ev_loaded = nullptr;
        b->index = -1;
        b->cache_off = -1;
        b->loaded_round = -1;
        b->used_round = -1;
    }
    for (int i = 0; i < 2; ++i) {
        if (ctx->ev_cache_done[i]) (void)hipEventDestroy(ctx->ev_cache_done[i]);
        ctx->ev_cache_done[i] = nullptr;
        ctx->cache_done_round[i] = -1;
    }
    ctx->cache_freed.clear();
    ctx->cache_mode = false;
    ctx->cache_base = nullptr;
    ctx->cache_cap = 0;
    ctx->cache_round = 0;
    ctx->placed.clear();
    if (ctx->wpool) (void)hipFree(ctx->wpool);
    if (ctx->staging) (void)hipFree(ctx->staging);
    ctx->wpool = ctx->staging = nullptr;
    ctx->zero_page = nullptr;
    ctx->wpool_bytes = 0;
    for (auto e : ctx->ev_copied)
        if (e) (void)hipEventDestroy(e);
    ctx->ev_copied.clear();
    ctx->slot_users.clear();
    ctx->staging_slots = 0;
    ctx->resident_bytes = 0;
    ctx->weights_ready = false;
}

}  // namespace

void drop_plans(gemel_ctx *ctx) {
    if (!ctx->plans.empty()) (void)hipDeviceSynchronize();
    for (auto &kv : ctx->plans) {
        Plan &p = *kv.second;
        for (auto g : p.graph)
            if (g) (void)hipGraphExecDestroy(g);
        for (auto &sg : p.segs)
            if (sg.exec) (void)hipGraphExecDestroy(sg.exec);
        for (auto ev : p.tune_ev)
            if (ev) (void)hipEventDestroy(ev);
        for (auto ev : p.events)
            if (ev) (void)hipEventDestroy(ev);
        if (p.ev_fork) (void)hipEventDestroy(p.ev_fork);
        for (auto ev : p.ev_join)
            if (ev) (void)hipEventDestroy(ev);
        for (auto ev : p.ev_chunk)
            if (ev) (void)hipEventDestroy(ev);
        if (p.image) (void)hipHostFree(p.image);
        if (!p.static_mem) {
            if (p.arena) (void)hipFree(p.arena);
            if (p.partial) (void)hipFree(p.partial);
            if (p.counters) (void)hipFree(p.counters);
        }
    }
    ctx->plans.clear();
    ctx->last_plan = nullptr;
    for (auto &u : ctx->slot_users) u.clear();   // events of the dropped plans
}

void release_device(gemel_ctx *ctx) {
    drop_plans(ctx);
    free_placement(ctx);
    if (ctx->tune_stream) (void)hipStreamSynchronize(ctx->tune_stream);
    if (ctx->tune_stream) (void)hipStreamDestroy(ctx->tune_stream);
    ctx->tune_stream = nullptr;
    for (auto &ev : ctx->tune_ev) {
        if (ev) (void)hipEventDestroy(ev);
        ev = nullptr;
    }
    if (ctx->tune_partial) (void)hipFree(ctx->tune_partial);
    if (ctx->tune_ctr) (void)hipFree(ctx->tune_ctr);
    if (ctx->tune_w) (void)hipFree(ctx->tune_w);
    ctx->tune_partial = ctx->tune_ctr = ctx->tune_w = nullptr;
    ctx->tune_partial_bytes = ctx->tune_ctr_bytes = ctx->tune_w_bytes = 0;
    if (ctx->side) (void)hipStreamDestroy(ctx->side);
    ctx->side = nullptr;
    for (hipEvent_t *ev : {&ctx->ev_round_done, &ctx->ev_side_join}) {
        if (*ev) (void)hipEventDestroy(*ev);
        *ev = nullptr;
    }
    ctx->round_seen = false;
    ctx->round_stream = nullptr;
    for (auto w : ctx->workers) (void)hipStreamDestroy(w);
    ctx->workers.clear();
    ctx->dev_ready = false;
}

// Tensor storage of every model under the current options and sharing
// map: which conv outputs are kept as bf16 (hi, lo) pairs, the physical
// channels per pixel of every tensor, and the parameters each conv reads
// (its effective parameters, or a copy whose input-channel columns follow
// the physical layout of a paired input).
//
// With GEMEL_OPT_PAIRED_ACTS, the output of an unmerged conv (not an output,
// not a residual, not reading an 8-channel input) is paired when every
// consumer can read pairs: an unmerged conv through its main input, or an
// upsample / concat (not an output) whose own consumers all can. A conv
// that reads a paired tensor multiplies both halves by the same weights
// (its weight columns duplicated), so it sums hi * w + lo * w in fp32.
static void assign_layouts(gemel_ctx *ctx) {
    const bool on = ctx->opt.paired_acts && ctx->dtype == GEMEL_BF16;
    for (auto &mp : ctx->models) {
        Model &m = *mp;
        const int n = (int)m.layers.size();
        // consumers of each layer: (consumer, 0 = src0, 1 = src1, 2 = residual)
        std::vector<std::vector<std::pair<int, int>>> cons((size_t)n);
        for (int c = 0; c < n; ++c) {
            const Layer &C = m.layers[(size_t)c];
            if (C.src0 >= 0) cons[(size_t)C.src0].push_back({c, 0});
            if (C.op == GEMEL_OP_CONCAT && C.src1 >= 0) cons[(size_t)C.src1].push_back({c, 1});
            if (C.res >= 0) cons[(size_t)C.res].push_back({c, 2});
        }
        std::function<bool(int, int)> reads_pairs = [&](int c, int role) -> bool {
            const Layer &C = m.layers[(size_t)c];
            if (role == 2) return false;
            if (C.op == GEMEL_OP_CONV) return role == 0 && C.group < 0;
            if (C.op != GEMEL_OP_UPSAMPLE2X && C.op != GEMEL_OP_CONCAT) return false;
            if (C.is_output || cons[(size_t)c].empty()) return false;
            for (auto [d, r] : cons[(size_t)c])
                if (!reads_pairs(d, r)) return false;
            return true;
        };
        // logical channel held by each physical channel of a tensor (-1: padding)
        auto plain = [](int c, int cp) {
            std::vector<int> v((size_t)cp, -1);
            for (int i = 0; i < c; ++i) v[(size_t)i] = i;
            return v;
        };
        const std::vector<int> in_map = plain(m.in_c, m.in_cp);
        std::vector<std::vector<int>> cmap((size_t)n);
        for (int l = 0; l < n; ++l) {
            Layer &L = m.layers[(size_t)l];
            const std::vector<int> &m0 = L.src0 < 0 ? in_map : cmap[(size_t)L.src0];
            L.in_phys = (int)m0.size();
            L.src1_phys = 0;
            L.out_paired = on && L.op == GEMEL_OP_CONV && L.group < 0 && !L.is_output && L.res < 0 &&
                           L.in_phys != 8 && !cons[(size_t)l].empty();
            for (auto [c, r] : cons[(size_t)l]) L.out_paired = L.out_paired && reads_pairs(c, r);
            std::vector<int> &out = cmap[(size_t)l];
            if (L.op == GEMEL_OP_UPSAMPLE2X) {
                out = m0;
            } else if (L.op == GEMEL_OP_CONCAT) {
                const std::vector<int> &m1 = L.src1 < 0 ? in_map : cmap[(size_t)L.src1];
                L.src1_phys = (int)m1.size();
                out = m0;
                for (int x : m1) out.push_back(x < 0 ? -1 : x + L.in_c);
            } else {
                out = plain(L.out_c, L.out_cp);
                if (L.out_paired) {
                    const std::vector<int> hi = out;
                    out.insert(out.end(), hi.begin(), hi.end());
                }
            }
            L.out_phys = (int)out.size();
            L.exec = L.eff;
            if (L.op == GEMEL_OP_CONV && L.eff && L.in_phys != L.in_cp) {
                // weight columns gathered to the input's physical channels
                const Blob &B = *L.eff;
                auto nb = std::make_shared<Blob>();
                nb->rows = B.rows;
                nb->elem = B.elem;
                nb->k = (int64_t)L.kh * L.kw * L.in_phys;
                nb->scale = B.scale;
                nb->shift = B.shift;
                nb->w.assign((size_t)(nb->rows * nb->k) * nb->elem, 0);
                for (int64_t o = 0; o < B.rows; ++o)
                    for (int64_t t = 0; t < (int64_t)L.kh * L.kw; ++t)
                        for (int j = 0; j < L.in_phys; ++j) {
                            const int c = m0[(size_t)j];
                            if (c < 0) continue;
                            std::memcpy(&nb->w[(size_t)((o * nb->k + t * L.in_phys + j) * (int64_t)nb->elem)],
                                        &B.w[(size_t)((o * B.k + t * L.in_cp + c) * (int64_t)B.elem)], B.elem);
                        }
                L.exec = nb;
            }
        }
    }
}

gemel_status materialise(gemel_ctx *ctx) {
    if (ctx->weights_ready) return GEMEL_OK;
    gemel_status st = ensure_device(ctx);
    if (st) return st;
    drop_plans(ctx);
    free_placement(ctx);
    assign_layouts(ctx);

    // distinct copies in use, in registration order, with their user counts
    std::vector<std::shared_ptr<Blob>> blobs;
    std::set<Blob *> seen;
    for (auto &m : ctx->models)
        for (auto &l : m->layers)
            if (l.exec) {
                if (seen.insert(l.exec.get()).second) {
                    l.exec->users = 0;
                    blobs.push_back(l.exec);
                }
                l.exec->users++;
            }
    size_t w_total = 0, aff_total = 0, max_final = 0;
    for (auto &b : blobs) {
        w_total += (size_t)round_up((int64_t)b->w_bytes(), 256);
        aff_total += (size_t)round_up((int64_t)b->aff_bytes(), 256);
    }
    for (auto &m : ctx->models)
        for (auto &l : m->layers)
            if (l.exec && l.is_output && l.consumers == 0) max_final = std::max(max_final, l.exec->w_bytes());

    std::vector<char> resident(blobs.size(), 1);
    size_t staging_bytes = 0;
    int slots = 0;
    int64_t slot_bytes = 0;
    // weight cache: scale/shift resident, every weight blob in pinned host
    // memory and loaded into the cache (the rest of the budget) when a
    // round needs it
    const bool cache = ctx->opt.swap_cache && ctx->budget;
    size_t cache_cap = 0;
    if (cache) {
        if (aff_total >= ctx->budget)
            return fail(ctx, GEMEL_EBUDGET, "weight budget smaller than the scale/shift vectors");
        cache_cap = (size_t)(ctx->budget - aff_total) / 256 * 256;
        std::fill(resident.begin(), resident.end(), 0);
    } else if (ctx->budget && w_total + aff_total > ctx->budget) {
        slots = ctx->opt.slots;
        slot_bytes = std::max<int64_t>(ctx->opt.slot_bytes, round_up((int64_t)max_final, 256));
        staging_bytes = (size_t)slots * (size_t)slot_bytes;
        if (aff_total + staging_bytes > ctx->budget)
            return fail(ctx, GEMEL_EBUDGET, "weight budget smaller than scale/shift vectors plus staging slots");
        size_t avail = ctx->budget - aff_total - staging_bytes;
        std::vector<size_t> order(blobs.size());
        std::iota(order.begin(), order.end(), 0);
        std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) {
            const bool sa = blobs[a]->users > 1, sb = blobs[b]->users > 1;
            if (sa != sb) return sa;
            return blobs[a]->w_bytes() > blobs[b]->w_bytes();
        });
        std::fill(resident.begin(), resident.end(), 0);
        for (size_t i : order) {
            const size_t need = (size_t)round_up((int64_t)blobs[i]->w_bytes(), 256);
            if (need <= avail) {
                resident[i] = 1;
                avail -= need;
            }
        }
        for (size_t i = 0; i < blobs.size(); ++i)
            if (!resident[i] && blobs[i]->k * (int64_t)blobs[i]->elem * 8 > slot_bytes)
                return fail(ctx, GEMEL_EBUDGET, "a weight row block does not fit one staging slot");
    }

    size_t pool = aff_total + GEMEL_ZERO_PAGE_BYTES + cache_cap;  // + zero page
    for (size_t i = 0; i < blobs.size(); ++i)
        if (resident[i]) pool += (size_t)round_up((int64_t)blobs[i]->w_bytes(), 256);
    if (alloc_device(ctx, &ctx->wpool, pool) != hipSuccess) {
        ctx->wpool = nullptr;
        (void)hipGetLastError();
        return fail(ctx, GEMEL_ENOMEM, "device allocation of the weight pool failed");
    }
    ctx->wpool_bytes = pool;
    {
        static const uint8_t zeros[GEMEL_ZERO_PAGE_BYTES] = {};
        ctx->zero_page = ctx->wpool;
        if (hipMemcpy(ctx->zero_page, zeros, sizeof(zeros), hipMemcpyHostToDevice) != hipSuccess) {
            free_placement(ctx);
            return fail(ctx, GEMEL_EDEVICE, "zero page upload failed");
        }
    }
    size_t off = GEMEL_ZERO_PAGE_BYTES;
    for (size_t i = 0; i < blobs.size(); ++i) {
        Blob &b = *blobs[i];
        ctx->placed.push_back(blobs[i]);
        b.aff_dev = (float *)((char *)ctx->wpool + off);
        hipError_t e = hipMemcpy(b.aff_dev, b.scale.data(), b.scale.size() * 4, hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = hipMemcpy(b.aff_dev + b.rows, b.shift.data(), b.shift.size() * 4, hipMemcpyHostToDevice);
        off += (size_t)round_up((int64_t)b.aff_bytes(), 256);
        if (e == hipSuccess && resident[i]) {
            b.w_dev = (char *)ctx->wpool + off;
            e = hipMemcpy(b.w_dev, b.w.data(), b.w_bytes(), hipMemcpyHostToDevice);
            off += (size_t)round_up((int64_t)b.w_bytes(), 256);
        } else if (e == hipSuccess) {
            e = alloc_pinned(ctx, (void **)&b.w_pinned, b.w_bytes());
            if (e == hipSuccess) std::memcpy(b.w_pinned, b.w.data(), b.w_bytes());
            else b.w_pinned = nullptr;
        }
        if (e == hipSuccess && cache) {
            b.index = (int)i;
            e = hipEventCreateWithFlags(&b.ev_loaded, hipEventDisableTiming);
            if (e != hipSuccess) b.ev_loaded = nullptr;
        }
        if (e != hipSuccess) {
            free_placement(ctx);
            return fail(ctx, GEMEL_ENOMEM, std::string("placing weights: ") + hipGetErrorString(e));
        }
    }
    if (cache) {
        ctx->cache_mode = true;
        ctx->cache_base = (char *)ctx->wpool + off;
        ctx->cache_cap = cache_cap;
        ctx->cache_round = 0;
        for (int k = 0; k < 2; ++k)
            if (hipEventCreateWithFlags(&ctx->ev_cache_done[k], hipEventDisableTiming) != hipSuccess) {
                ctx->ev_cache_done[k] = nullptr;
                free_placement(ctx);
                return fail(ctx, GEMEL_EDEVICE, "event creation failed");
            }
    }
    if (slots) {
        if (alloc_device(ctx, &ctx->staging, staging_bytes) != hipSuccess) {
            ctx->staging = nullptr;
            free_placement(ctx);
            return fail(ctx, GEMEL_ENOMEM, "device allocation of the staging slots failed");
        }
        ctx->staging_slots = slots;
        ctx->staging_slot_bytes = slot_bytes;
        ctx->ev_copied.resize((size_t)slots);
        ctx->slot_users.assign((size_t)slots, {});
        for (int i = 0; i < slots; ++i) {
            if (hipEventCreateWithFlags(&ctx->ev_copied[(size_t)i], hipEventDisableTiming) != hipSuccess) {
                free_placement(ctx);
                return fail(ctx, GEMEL_EDEVICE, "event creation failed");
            }
        }
    }
    size_t res_w = 0;
    for (size_t i = 0; i < blobs.size(); ++i)
        if (resident[i]) res_w += blobs[i]->bytes();
        else res_w += blobs[i]->aff_bytes();
    ctx->resident_bytes = res_w;
    ctx->peak_bytes = std::max(ctx->peak_bytes, pool + staging_bytes);
    ctx->weights_ready = true;
    return GEMEL_OK;
}

// ----------------------------------------------------------------------------
// plan construction
// ----------------------------------------------------------------------------
namespace {

struct TRef {
    int slot, layer;  // layer -1 = the slot's packed input
    bool operator<(const TRef &o) const { return slot != o.slot ? slot < o.slot : layer < o.layer; }
};

struct Tensor {
    size_t bytes = 0;
    int first = 0, last = 0;
    size_t off = 0;
};

struct Node {
    int op;
    std::vector<std::pair<int, int>> mem;  // (slot, layer)
};

bool direct_output(const Layer &l) {
    return l.is_output && l.consumers == 0 && (l.op == GEMEL_OP_CONV || l.op == GEMEL_OP_FC);
}

// Launch configuration of a bf16 implicit-GEMM conv of size M x N x K:
// the tile shape and split-K factor with the smallest estimated time.
// Model (fitted to measured times of every tile shape on the conv shapes of
// the ResNet, VGG and Darknet workloads): tiles run in waves of (256 CUs x
// resident tiles per CU); a wave costs its tiles' FLOPs at the tile shape's
// MFMA efficiency plus a per-wave latency; split-K adds the partial-sum
// round trip through memory.
struct TileCost {
    int tile;
    double eff;   // MFMA efficiency of the tile shape
    int occ;      // tiles resident per CU
    double lat;   // seconds of latency per wave of tiles
};
static const TileCost kTileCost[] = {
    {TILE_128x128, 0.441, 2, 5.61e-6},
    {TILE_128x64, 0.311, 2, 3.88e-6},
    {TILE_64x64, 0.375, 4, 2.79e-6},
    {TILE_256x256, 0.469, 1, 11.42e-6},
    {TILE_256x128, 0.351, 1, 6.62e-6},
    {TILE_256x64, 0.217, 1, 5.53e-6},
    {TILE_64x64_D2, 0.301, 3, 2.48e-6},
    {TILE_128x64_D2, 0.313, 2, 4.03e-6},
    {TILE_64x128, 0.332, 2, 3.60e-6},
    {TILE_DMA_256x256, 0.529, 1, 7.94e-6},
    {TILE_DMA_256x128, 0.330, 1, 7.72e-6},
    {TILE_DMA_128x128, 0.526, 2, 4.83e-6},
    {TILE_DMA_128x64, 0.379, 3, 5.06e-6},
    {TILE_DMA64_256x256, 0.520, 1, 7.94e-6},
    {TILE_DMA64_256x128, 0.320, 1, 7.72e-6},
    {TILE_DMA64_128x128, 0.520, 1, 4.83e-6},
    {TILE_DMA64_128x64, 0.370, 3, 5.06e-6},
    {TILE_DMA_64x64, 0.380, 4, 2.50e-6},
    {TILE_DMA64_64x64, 0.420, 2, 2.20e-6},
    {TILE_DMA_256x128W8, 0.560, 1, 7.00e-6},
    {TILE_DMA_128x256W8, 0.560, 1, 7.00e-6},
    {TILE_DMA_256x64, 0.500, 2, 5.00e-6},
    {TILE_DMA_64x256, 0.500, 2, 5.00e-6},
};

// Partial sums of one split-K launch are addressed with 32-bit byte offsets.
constexpr int64_t kMaxPartialBytes = 0x7fffffff;

// One launch configuration of a conv and its estimated time.
struct ConvCand {
    double est;
    int tile, splits;
};

// Every (tile, split-K) configuration the conv may use, fastest estimate
// first. dma_depth: deepest LDS-DMA step the conv allows (0: no DMA tile,
// 32 or 64); force >= 0 restricts the tile; dma_only: LDS-DMA tiles only
// (a fused pool, segments of mixed sizes); no_split: no split-K (a fused
// pool).
std::vector<ConvCand> conv_candidates(int64_t M, int64_t N, int64_t K, int dma_depth, int force, bool dma_only,
                                      bool no_split) {
    const double cu_flops = 4096.0 * 2.4e9;   // per CU, dense bf16
    std::vector<ConvCand> out;
    for (const TileCost &tc : kTileCost) {
        if (force >= 0 && tc.tile != force) continue;
        if (force < 0 && tile_is_dma(tc.tile) && tile_dma_depth(tc.tile) > dma_depth) continue;
        if (dma_only && (!tile_is_dma(tc.tile) || tile_dma_depth(tc.tile) > dma_depth)) continue;
        const int64_t bm = conv_tile_bm(tc.tile), bn = conv_tile_bn(tc.tile);
        const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
        int last = 0;
        for (int s = 1; s <= 16; s *= 2) {
            if (s > 1 && K / s < 4 * CONV_BK) break;
            const int64_t k_s = round_up((K + s - 1) / s, CONV_BK);
            const int64_t s_eff = (K + k_s - 1) / k_s;
            if (s_eff > 1 && s_eff * M * N * 4 > kMaxPartialBytes) break;
            if (s_eff == last) continue;
            if (no_split && s_eff > 1) break;
            last = (int)s_eff;
            const double waves = std::ceil((double)(tiles * s_eff) / (256.0 * tc.occ));
            double t = waves * (tc.occ * (2.0 * bm * bn * k_s) / (cu_flops * tc.eff) + tc.lat);
            if (s_eff > 1) t += (double)s_eff * M * N * 4.0 * 2.0 / 4e12 + 2e-6;
            out.push_back({t, tc.tile, (int)s_eff});
        }
    }
    std::stable_sort(out.begin(), out.end(), [](const ConvCand &x, const ConvCand &y) { return x.est < y.est; });
    return out;
}

// Depth per split for `splits` splits (a multiple of the conv step); the
// split count is then the number of splits that depth needs.
void conv_split_depth(int64_t K, int &splits, int &kps) {
    kps = (int)round_up((K + splits - 1) / splits, CONV_BK);
    splits = (int)((K + kps - 1) / kps);
}

// Launch configuration of a bf16 implicit-GEMM conv of size M x N x K:
// the candidate with the smallest estimated time (or the forced tile /
// split count).
void pick_conv_config(int64_t M, int64_t N, int64_t K, int dma_depth, int force, int force_splits, bool dma_only,
                      bool pooled, int &tile, int &splits, int &kps) {
    const std::vector<ConvCand> c = conv_candidates(M, N, K, dma_depth, force, dma_only || pooled, pooled);
    tile = c.empty() ? (force >= 0 ? force : TILE_64x64) : c[0].tile;
    splits = c.empty() ? 1 : c[0].splits;
    if (force_splits > 0 && !pooled) splits = (int)std::min<int64_t>(force_splits, (K + CONV_BK - 1) / CONV_BK);
    while (splits > 1 && (int64_t)splits * M * N * 4 > kMaxPartialBytes) --splits;
    conv_split_depth(K, splits, kps);
}

// Split-K partial sums reduced inside the GEMM launch (by the last split of
// each tile): only as many workgroups as tiles share that work, so with
// fewer tiles than compute units a separate reduction launch (one
// workgroup per 2048 outputs) is faster (measured).
bool fuse_splitk(const gemel_ctx *ctx, int tiles) {
    return ctx->opt.splitk_fused == 2 || (ctx->opt.splitk_fused == 1 && tiles >= 256);
}

// Argument block of the separate split-K reduction of conv launch a.
ReduceArgs reduce_args(const ConvArgs &a) {
    ReduceArgs r{};
    r.partial = a.partial;
    r.M = a.M; r.N = a.N; r.splits = a.k_splits; r.HWo = a.Ho * a.Wo;
    r.out_cs = a.out_cs; r.cout = a.cout; r.act = a.act; r.slope = a.slope;
    r.res_mode = a.res_mode; r.has_res = a.has_res; r.out_mode = a.out_mode;
    r.out_pair = a.out_pair;
    r.nseg = a.nseg;
    for (int i = 0; i < a.nseg; ++i) r.seg[i] = a.seg[i];
    return r;
}

// Measured choice among the best-estimated configurations of one conv
// launch: each candidate runs on the context's tuning stream over the
// plan's own tensors (their contents are overwritten by every round), timed
// launch by launch with HIP events bound to the kernels' own start and end
// (hipExtLaunchKernel: the gap before the dispatch is not counted); the
// smallest median wins. Results
// are cached per conv shape for the life of the context. Returns false
// (leaving tile/splits/kps alone) if nothing could be timed.
bool tune_conv(gemel_ctx *ctx, const ConvArgs &a0, int dma_depth, bool bf16, int &tile, int &splits, int &kps) {
    std::vector<int64_t> key = {a0.M, a0.N, a0.K, a0.H, a0.W, a0.Cin, a0.in_cs, a0.kh, a0.kw, a0.stride, a0.pad,
                                a0.out_cs, a0.has_res, a0.out_mode, a0.nseg > 1, dma_depth, ctx->opt.splitk_fused,
                                a0.hetero, a0.grouped, a0.out_pair};
    auto hit = ctx->tune_cache.find(key);
    if (hit != ctx->tune_cache.end()) {
        tile = hit->second.first;
        splits = hit->second.second;
        conv_split_depth(a0.K, splits, kps);
        return true;
    }
    const bool pooled = a0.out_mode == OUT_NHWC_POOL2;
    std::vector<ConvCand> c = conv_candidates(a0.M, a0.N, a0.K, dma_depth, -1, pooled || a0.hetero || a0.grouped, pooled);
    if (c.empty()) return false;
    const double cut = 2.0 * c[0].est;
    size_t n = 0;
    while (n < c.size() && n < (size_t)ctx->opt.tune_candidates && c[n].est <= cut) ++n;
    if (n < 2) return false;
    c.resize(n);
    // scratch: partial sums and arrival counters of the largest candidate
    size_t pbytes = 0, cbytes = 0;
    for (const ConvCand &k : c) {
        const int64_t bm = conv_tile_bm(k.tile), bn = conv_tile_bn(k.tile);
        if (k.splits > 1) pbytes = std::max(pbytes, (size_t)k.splits * a0.M * a0.N * 4);
        cbytes = std::max(cbytes, (size_t)conv_tiles(a0, (int)bm, (int)bn) * 4);
    }
    if (!ctx->tune_stream && hipStreamCreateWithFlags(&ctx->tune_stream, hipStreamNonBlocking) != hipSuccess)
        return false;
    if (!ctx->tune_ev[0] && (hipEventCreate(&ctx->tune_ev[0]) != hipSuccess ||
                             hipEventCreate(&ctx->tune_ev[1]) != hipSuccess))
        return false;
    if (pbytes > ctx->tune_partial_bytes) {
        if (ctx->tune_partial) (void)hipFree(ctx->tune_partial);
        ctx->tune_partial = nullptr;
        ctx->tune_partial_bytes = 0;
        if (alloc_device(ctx, &ctx->tune_partial, pbytes) != hipSuccess) {
            (void)hipGetLastError();
            return false;
        }
        ctx->tune_partial_bytes = pbytes;
    }
    // cached weights may still be in flight on the copy stream, or not be
    // cached at all: time the candidates over a zeroed buffer of the same
    // size instead (the kernels' timing does not depend on the values)
    const size_t wbytes = ctx->cache_mode ? (size_t)a0.N * a0.K * (bf16 ? 2 : 4) : 0;
    if (wbytes > ctx->tune_w_bytes) {
        if (ctx->tune_w) (void)hipFree(ctx->tune_w);
        ctx->tune_w = nullptr;
        ctx->tune_w_bytes = 0;
        if (alloc_device(ctx, &ctx->tune_w, wbytes) != hipSuccess) {
            (void)hipGetLastError();
            return false;
        }
        const std::vector<char> zeros(wbytes, 0);
        if (hipMemcpy(ctx->tune_w, zeros.data(), wbytes, hipMemcpyHostToDevice) != hipSuccess) return false;
        ctx->tune_w_bytes = wbytes;
    }
    if (cbytes > ctx->tune_ctr_bytes) {
        if (ctx->tune_ctr) (void)hipFree(ctx->tune_ctr);
        ctx->tune_ctr = nullptr;
        ctx->tune_ctr_bytes = 0;
        if (alloc_device(ctx, &ctx->tune_ctr, cbytes) != hipSuccess) {
            (void)hipGetLastError();
            return false;
        }
        const std::vector<char> zeros(cbytes, 0);
        if (hipMemcpy(ctx->tune_ctr, zeros.data(), cbytes, hipMemcpyHostToDevice) != hipSuccess) return false;
        ctx->tune_ctr_bytes = cbytes;
    }
    Sink sk;
    sk.stream = ctx->tune_stream;
    // launch of candidate i; timed: the events take the kernels' own start
    // and end (the reduction's end where a separate launch reduces)
    auto once = [&](size_t i, bool timed = false) {
        ConvArgs a = a0;
        if (wbytes) {
            a.w = ctx->tune_w;
            if (a.grouped)
                for (int g = 0; g < a.nseg; ++g) a.seg[g].w = ctx->tune_w;
        }
        int sp = c[i].splits, kp = 0;
        conv_split_depth(a.K, sp, kp);
        a.k_splits = sp;
        a.k_per_split = kp;
        const int64_t bm = conv_tile_bm(c[i].tile), bn = conv_tile_bn(c[i].tile);
        const int tiles = (int)conv_tiles(a, (int)bm, (int)bn);
        const bool fuse = sp > 1 && fuse_splitk(ctx, tiles);
        a.partial = sp > 1 ? (float *)ctx->tune_partial : nullptr;
        a.counters = fuse ? (int32_t *)ctx->tune_ctr : nullptr;
        const bool two = sp > 1 && !fuse;
        Sink s1 = sk, s2 = sk;
        if (timed) {
            s1.ev_start = ctx->tune_ev[0];
            (two ? s2 : s1).ev_stop = ctx->tune_ev[1];
        }
        hipError_t e = launch_conv_bf16(a, c[i].tile, s1);
        if (e == hipSuccess && two) e = launch_conv_reduce(reduce_args(a), bf16, s2);
        return e;
    };
    // one untimed pass over every candidate, then kTuneReps passes timing
    // each launch on its own with the candidates interleaved (a clock that
    // is still rising, or any other drift, then affects all of them alike);
    // the median of a candidate's times decides
    constexpr int kTuneReps = 7;
    std::vector<bool> ok(c.size(), true);
    std::vector<std::vector<float>> ms(c.size());
    for (size_t i = 0; i < c.size(); ++i) ok[i] = once(i) == hipSuccess;
    for (int rep = 0; rep < kTuneReps; ++rep) {
        for (size_t i = 0; i < c.size(); ++i) {
            if (!ok[i]) continue;
            float t = 0.f;
            ok[i] = once(i, true) == hipSuccess && hipEventSynchronize(ctx->tune_ev[1]) == hipSuccess &&
                    hipEventElapsedTime(&t, ctx->tune_ev[0], ctx->tune_ev[1]) == hipSuccess;
            if (ok[i]) ms[i].push_back(t);
        }
    }
    (void)hipGetLastError();
    double best = 1e300;
    int bi = -1;
    for (size_t i = 0; i < c.size(); ++i) {
        if (!ok[i] || ms[i].empty()) continue;
        std::vector<float> v = ms[i];
        std::nth_element(v.begin(), v.begin() + v.size() / 2, v.end());
        if (v[v.size() / 2] < best) {
            best = v[v.size() / 2];
            bi = (int)i;
        }
    }
    if (hipStreamSynchronize(ctx->tune_stream) != hipSuccess || bi < 0) return false;
    tile = c[(size_t)bi].tile;
    splits = c[(size_t)bi].splits;
    conv_split_depth(a0.K, splits, kps);
    ctx->tune_cache[key] = {tile, c[(size_t)bi].splits};
    return true;
}

// Split-K of the small-batch FC kernel: enough workgroups to keep HBM busy
// (about 1024), with each split's input slice (16-frame blocks x depth) fitting
// the kernel's 64 KB of LDS.
void pick_fc_config(int64_t M, int64_t N, int64_t K, int &splits, int &kps) {
    // M: frames of the largest grid slice (a grouped launch takes the
    // configuration of one member's launch, so that its results are those
    // of separate launches)
    const int64_t blocks = (N + 63) / 64;
    const int64_t want = (1024 + blocks - 1) / blocks;
    const int64_t maxs = std::max<int64_t>(1, K / 1024);
    // frames staged in LDS (as the kernel computes them) and the depth that
    // fits: kps * mp elements plus the last 64-slot run
    const int64_t mp = M > 16 ? (M + 15) / 16 * 16 : M > 8 ? 16 : M > 4 ? 8 : M > 2 ? 4 : M;
    const int64_t kps_cap = std::max<int64_t>(128, (32768 / mp - 64) / 128 * 128);
    splits = (int)std::max<int64_t>(1, std::min(want, maxs));
    splits = (int)std::max<int64_t>(splits, (K + kps_cap - 1) / kps_cap);
    kps = (int)round_up((K + splits - 1) / splits, 128);
    splits = (int)((K + kps - 1) / kps);
}

}  // namespace

// can_tune: conv configurations may be timed on the device (not while the
// caller's stream is being captured into a graph).
// static_base: the arena, split-K partial sums and counters are laid out in
// these static_cap bytes (the static scratch) instead of being allocated.
static gemel_status build_plan(gemel_ctx *ctx, const std::vector<int> &ids, const std::vector<int> &nfr,
                               Plan &P, bool can_tune, void *static_base = nullptr, size_t static_cap = 0) {
    const bool bf16 = ctx->dtype == GEMEL_BF16;
    const size_t esz = bf16 ? 2 : 4;
    const int S = (int)ids.size();
    P.model_ids = ids;
    P.n_frames = nfr;
    P.out_base.resize((size_t)S);
    for (int s = 0, ob = 0; s < S; ++s) {
        P.out_base[(size_t)s] = ob;
        ob += (int)ctx->models[(size_t)ids[(size_t)s]]->outputs.size();
    }
    auto model = [&](int s) -> const Model & { return *ctx->models[(size_t)ids[(size_t)s]]; };
    auto layer = [&](int s, int l) -> const Layer & { return model(s).layers[(size_t)l]; };

    // ---- 2x2 max pools fused into their conv: pool_of[s][l] is the pool
    // that conv (s, l) writes from its epilogue (-1: none). The conv is its
    // pool's only producer input, the pool its only consumer; the pool
    // layer then belongs to the conv's node and has no launch of its own ----
    std::vector<std::vector<int>> pool_of((size_t)S), fused_into((size_t)S);
    const int forced = ctx->opt.conv_tile;
    for (int s = 0; s < S; ++s) {
        const Model &m = model(s);
        pool_of[(size_t)s].assign(m.layers.size(), -1);
        fused_into[(size_t)s].assign(m.layers.size(), -1);
        if (!bf16 || !ctx->opt.fuse_pool || (forced >= 0 && !tile_is_dma(forced))) continue;
        for (int p = 0; p < (int)m.layers.size(); ++p) {
            const Layer &Pl = m.layers[(size_t)p];
            if (Pl.op != GEMEL_OP_MAXPOOL || Pl.kh != 2 || Pl.kw != 2 || Pl.stride != 2 || Pl.pad != 0 || Pl.src0 < 0)
                continue;
            const int l = Pl.src0;
            const Layer &L = m.layers[(size_t)l];
            // the LDS-DMA kernel's requirements (as for its tiles below)
            const bool dma = L.in_phys % 32 == 0 && (int64_t)L.in_phys * 2 + 128 <= GEMEL_ZERO_PAGE_BYTES &&
                             (forced < 0 || tile_dma_depth(forced) == 32 || L.in_phys % 64 == 0);
            if (L.op != GEMEL_OP_CONV || L.res >= 0 || L.is_output || L.consumers != 1 || !dma || L.out_h % 2 ||
                L.out_w % 2 || L.out_h < 2 || L.out_w < 2)
                continue;
            pool_of[(size_t)s][(size_t)l] = p;
            fused_into[(size_t)s][(size_t)p] = l;
        }
    }

    // ---- nodes: merged groups batched when compatible ----
    // A node batches at most one appearance of a group per model: the k-th
    // appearance in each model goes with the k-th of the others (appearances
    // within one model may depend on each other, e.g. repeated blocks).
    std::vector<Node> nodes;
    std::map<std::vector<int64_t>, int> group_node;
    std::map<std::pair<int, int>, int> occurrence;   // (model slot, group) -> appearances so far
    std::map<std::pair<int, std::vector<int64_t>>, int> ungrouped_seen;  // (slot, signature) -> appearances
    // an unmerged bf16 conv that a grouped launch can take: the LDS-DMA
    // kernel's input conditions, resident weights, no mixed sizes
    auto groupable = [&](int s, int l) {
        const Layer &L = layer(s, l);
        if (!ctx->opt.group_unmerged || !bf16 || L.group >= 0 || !L.exec || !(L.exec->w_dev || ctx->cache_mode))
            return false;
        // the FC kernel over at most 64 frames in all; a layer whose weights
        // alone fill the GPU's memory bandwidth keeps its own launch
        if (L.op == GEMEL_OP_FC) return L.exec->w_bytes() <= ((size_t)64 << 20);
        return L.op == GEMEL_OP_CONV && L.in_phys % 32 == 0 && (int64_t)L.in_phys * 2 + 128 <= GEMEL_ZERO_PAGE_BYTES &&
               (forced < 0 || (tile_is_dma(forced) && (tile_dma_depth(forced) == 32 || L.in_phys % 64 == 0)));
    };
    std::map<int, int64_t> node_frames;   // frames of a grouped FC node so far
    std::vector<std::vector<int>> node_of((size_t)S);
    for (int s = 0; s < S; ++s) {
        const Model &m = model(s);
        node_of[(size_t)s].assign(m.layers.size(), -1);
        for (int l = 0; l < (int)m.layers.size(); ++l) {
            const Layer &L = m.layers[(size_t)l];
            if (fused_into[(size_t)s][(size_t)l] >= 0) {   // a fused pool: part of its conv's node
                node_of[(size_t)s][(size_t)l] = node_of[(size_t)s][(size_t)fused_into[(size_t)s][(size_t)l]];
                continue;
            }
            int nid = -1;
            if (L.group >= 0 && !ctx->opt.split_merged) {
                // members of different spatial sizes share a launch where the
                // LDS-DMA kernel can take them (one weight copy, per-segment
                // sizes): bf16 conv, internal NHWC output, no fused pool
                const bool mixed = ctx->opt.mixed_sizes && bf16 && L.op == GEMEL_OP_CONV && !direct_output(L) &&
                                   pool_of[(size_t)s][(size_t)l] < 0 && L.in_phys % 32 == 0 &&
                                   (int64_t)L.in_phys * 2 + 128 <= GEMEL_ZERO_PAGE_BYTES &&
                                   (forced < 0 || (tile_is_dma(forced) && (tile_dma_depth(forced) == 32 || L.in_phys % 64 == 0)));
                std::vector<int64_t> key = {L.group, mixed ? -1 : L.in_h, mixed ? -1 : L.in_w, L.in_c, L.act,
                                            (int64_t)(L.slope * 1e6f), L.res >= 0, L.res_mode,
                                            direct_output(L), L.src1_phys, L.in_phys, L.out_paired,
                                            pool_of[(size_t)s][(size_t)l] >= 0,
                                            occurrence[{s, L.group}]++};
                auto it = group_node.find(key);
                if (it != group_node.end() && nodes[(size_t)it->second].mem.size() < GEMEL_MAX_SEG) {
                    nid = it->second;
                } else {
                    nid = (int)nodes.size();
                    nodes.push_back(Node{L.op, {}});
                    group_node[key] = nid;
                }
            } else if (groupable(s, l)) {
                // the same unmerged conv of several models (same shape and
                // epilogue, its k-th appearance in each): one grouped launch,
                // each segment with its own weights
                const int pooled = pool_of[(size_t)s][(size_t)l] >= 0;
                std::vector<int64_t> sig = {-1, L.op, L.in_h, L.in_w, L.in_c, L.in_phys, L.out_c, L.out_phys,
                                            L.kh, L.stride, L.pad, L.act, (int64_t)(L.slope * 1e6f), L.res >= 0,
                                            L.res_mode, direct_output(L), L.out_paired, pooled,
                                            (int64_t)L.exec->k};
                sig.push_back(ungrouped_seen[{s, sig}]++);
                auto it = group_node.find(sig);
                const bool fits = L.op != GEMEL_OP_FC ||
                                  (it != group_node.end() && node_frames[it->second] + nfr[(size_t)s] <= 64);
                if (it != group_node.end() && nodes[(size_t)it->second].mem.size() < GEMEL_MAX_SEG && fits) {
                    nid = it->second;
                } else {
                    nid = (int)nodes.size();
                    nodes.push_back(Node{L.op, {}});
                    group_node[sig] = nid;
                }
                node_frames[nid] += nfr[(size_t)s];
            } else {
                nid = (int)nodes.size();
                nodes.push_back(Node{L.op, {}});
            }
            nodes[(size_t)nid].mem.push_back({s, l});
            node_of[(size_t)s][(size_t)l] = nid;
        }
    }

    // ---- topological order of nodes (Kahn) ----
    auto topo = [&](std::vector<int> &order) -> bool {
        const size_t n = nodes.size();
        std::vector<std::set<int>> out(n);
        std::vector<int> indeg(n, 0);
        for (size_t v = 0; v < n; ++v)
            for (auto [s, l] : nodes[v].mem) {
                const Layer &L = layer(s, l);
                for (int p : {L.src0, L.src1, L.res}) {
                    if (p < 0) continue;
                    const int u = node_of[(size_t)s][(size_t)p];
                    if (u != (int)v && out[(size_t)u].insert((int)v).second) indeg[v]++;
                }
            }
        auto key = [&](int v) {
            auto [s, l] = nodes[(size_t)v].mem[0];
            return std::make_pair(l, s);
        };
        auto cmp = [&](int a, int b) { return key(a) > key(b); };
        std::priority_queue<int, std::vector<int>, decltype(cmp)> q(cmp);
        for (size_t v = 0; v < n; ++v)
            if (!indeg[v]) q.push((int)v);
        order.clear();
        while (!q.empty()) {
            const int v = q.top();
            q.pop();
            order.push_back(v);
            for (int w : out[(size_t)v])
                if (--indeg[(size_t)w] == 0) q.push(w);
        }
        return order.size() == n;
    };
    // a merged node that takes part in a cycle (its members' models order
    // their layers differently) runs its members separately: the nodes Kahn
    // leaves unordered are on a cycle or behind one, and each round splits
    // the merged ones among them until an order exists
    std::vector<int> order;
    while (!topo(order)) {
        std::vector<char> done(nodes.size(), 0);
        for (int v : order) done[(size_t)v] = 1;
        std::vector<Node> next;
        bool split = false;
        for (size_t v = 0; v < nodes.size(); ++v) {
            if (!done[v] && nodes[v].mem.size() > 1) {
                split = true;
                for (auto &mb : nodes[v].mem) next.push_back(Node{nodes[v].op, {mb}});
            } else {
                next.push_back(nodes[v]);
            }
        }
        if (!split) return fail(ctx, GEMEL_ESTATE, "internal: layer graph has a cycle");
        nodes.swap(next);
        for (size_t v = 0; v < nodes.size(); ++v)
            for (auto &mb : nodes[v].mem) node_of[(size_t)mb.first][(size_t)mb.second] = (int)v;
        for (int s = 0; s < S; ++s)
            for (size_t p = 0; p < fused_into[(size_t)s].size(); ++p)
                if (fused_into[(size_t)s][p] >= 0)
                    node_of[(size_t)s][p] = node_of[(size_t)s][(size_t)fused_into[(size_t)s][p]];
    }

    // ---- steps: the ordered nodes, then one export step per output that is
    // not written directly by its conv/FC epilogue ----
    const int NN = (int)order.size();
    std::vector<int> pos(nodes.size());
    for (int i = 0; i < NN; ++i) pos[(size_t)order[(size_t)i]] = i;
    std::vector<std::pair<int, int>> exports;  // (slot, layer)
    for (int s = 0; s < S; ++s)
        for (int l : model(s).outputs)
            if (!direct_output(layer(s, l))) exports.push_back({s, l});
    const int NS = NN + (int)exports.size();
    auto step_of = [&](int s, int l) { return pos[(size_t)node_of[(size_t)s][(size_t)l]]; };
    std::vector<std::vector<int>> preds((size_t)NS);
    std::vector<double> est((size_t)NS, 5e-6);
    for (int i = 0; i < NN; ++i) {
        std::set<int> ps;
        {   // the node's weights are read once, whatever its member count
            const auto [s0, l0] = nodes[(size_t)order[(size_t)i]].mem[0];
            const Layer &L0 = layer(s0, l0);
            if (L0.exec) est[(size_t)i] += (double)L0.exec->rows * L0.exec->k * L0.exec->elem / 4e12;
        }
        for (auto [s, l] : nodes[(size_t)order[(size_t)i]].mem) {
            const Layer &L = layer(s, l);
            if (L.src0 >= 0) ps.insert(step_of(s, L.src0));
            if (L.op == GEMEL_OP_CONCAT && L.src1 >= 0) ps.insert(step_of(s, L.src1));
            if (L.res >= 0) ps.insert(step_of(s, L.res));
            const double n = nfr[(size_t)s];
            const double kd = L.op == GEMEL_OP_CONV ? (double)L.kh * L.kw * L.cin : (double)L.cin;
            if (L.op == GEMEL_OP_CONV || L.op == GEMEL_OP_FC)
                est[(size_t)i] += 2.0 * n * L.out_h * L.out_w * L.out_c * kd / 1e15;
            est[(size_t)i] += n * L.out_h * L.out_w * L.out_phys * esz / 4e12;
        }
        preds[(size_t)i].assign(ps.begin(), ps.end());
    }
    for (size_t e = 0; e < exports.size(); ++e) preds[(size_t)NN + e] = {step_of(exports[e].first, exports[e].second)};

    // ---- happens-before: ancestors of each step in the dependency graph ----
    const size_t WDS = ((size_t)NS + 63) / 64;
    std::vector<uint64_t> anc((size_t)NS * WDS, 0);
    for (int i = 0; i < NS; ++i)
        for (int p : preds[(size_t)i]) {
            uint64_t *dst = &anc[(size_t)i * WDS];
            const uint64_t *src = &anc[(size_t)p * WDS];
            for (size_t w = 0; w < WDS; ++w) dst[w] |= src[w];
            dst[(size_t)p / 64] |= 1ull << (p % 64);
        }

    // ---- streams: each step continues the stream of a predecessor it directly
    // follows. A step that starts a branch opens the least loaded stream only
    // when the work it dominates (the steps reachable from the round's start
    // only through it: what can overlap with other branches before they
    // join) is worth a fork, a cross-stream wait costing a few microseconds;
    // else it queues behind its first predecessor. Cross-stream edges become
    // event waits (graph edges in a graph round) ----
    std::vector<int> idom((size_t)NS, -1), depth((size_t)NS, 0);  // -1: the round's start
    for (int i = 0; i < NS; ++i) {
        const auto &pr = preds[(size_t)i];
        const bool from_start = pr.empty() || (i < NN && [&] {
            for (auto [s, l] : nodes[(size_t)order[(size_t)i]].mem) {
                const Layer &L = layer(s, l);
                if (L.src0 < 0 || (L.op == GEMEL_OP_CONCAT && L.src1 < 0)) return true;
            }
            return false;
        }());
        int d = from_start ? -1 : pr[0];
        for (size_t k = 1; k < pr.size() && d >= 0; ++k) {  // nearest common dominator
            int x = d, y = pr[k];
            while (x != y && x >= 0 && y >= 0) {
                if (depth[(size_t)x] >= depth[(size_t)y]) x = idom[(size_t)x];
                else y = idom[(size_t)y];
            }
            d = (x == y) ? x : -1;
        }
        idom[(size_t)i] = d;
        depth[(size_t)i] = d < 0 ? 1 : depth[(size_t)d] + 1;
    }
    std::vector<double> owned(est);  // estimated work of the dominator subtree
    std::vector<int> owned_steps((size_t)NS, 1);
    for (int i = NS - 1; i >= 0; --i)
        if (idom[(size_t)i] >= 0) {
            owned[(size_t)idom[(size_t)i]] += owned[(size_t)i];
            owned_steps[(size_t)idom[(size_t)i]] += owned_steps[(size_t)i];
        }
    // a chain of 3 or more launches overlaps usefully even when its FLOPs are
    // few: small launches are latency bound
    const double fork_work = ctx->opt.fork_us * 1e-6;
    auto worth_fork = [&](int i) { return owned[(size_t)i] >= fork_work || owned_steps[(size_t)i] >= 3; };
    const int SMAX = std::max(1, std::min(ctx->opt.streams, 1 + (int)ctx->workers.size()));
    std::vector<int> stream_of((size_t)NS, 0), tail((size_t)SMAX, -2);
    std::vector<double> load((size_t)SMAX, 0.0);
    for (int i = 0; i < NS; ++i) {
        int st = -1;
        for (int p : preds[(size_t)i])
            if (tail[(size_t)stream_of[(size_t)p]] == p) {
                st = stream_of[(size_t)p];
                break;
            }
        if (st < 0 && !preds[(size_t)i].empty() && !worth_fork(i)) st = stream_of[(size_t)preds[(size_t)i][0]];
        if (st < 0) {
            st = 0;
            for (int k = 1; k < SMAX; ++k)
                if (load[(size_t)k] < load[(size_t)st]) st = k;
        }
        stream_of[(size_t)i] = st;
        tail[(size_t)st] = i;
        load[(size_t)st] += est[(size_t)i];
    }
    std::vector<int> event_of((size_t)NS, -1);
    int n_events = 0;
    P.n_streams = 1;
    for (int i = 0; i < NS; ++i) {
        P.n_streams = std::max(P.n_streams, stream_of[(size_t)i] + 1);
        for (int p : preds[(size_t)i])
            if (stream_of[(size_t)p] != stream_of[(size_t)i] && event_of[(size_t)p] < 0) event_of[(size_t)p] = n_events++;
    }

    auto before = [&](int a_, int b_) {  // step a_ strictly precedes step b_
        if (a_ < 0) return b_ >= 0;          // the pack precedes every step
        if (b_ < 0) return false;
        return ((anc[(size_t)b_ * WDS + (size_t)a_ / 64] >> (a_ % 64)) & 1ull) != 0;
    };

    // ---- tensors: producer step (-1 = pack), user steps; two tensors share
    // bytes only when every use of one precedes the other's producer ----
    struct TInfo {
        size_t bytes = 0, off = 0;
        int prod = -1;
        std::vector<int> users;
    };
    std::map<TRef, TInfo> T;
    for (int s = 0; s < S; ++s) {
        const Model &m = model(s);
        T[{s, -1}].bytes = (size_t)nfr[(size_t)s] * m.in_h * m.in_w * m.in_cp * esz;
    }
    for (int i = 0; i < NN; ++i)
        for (auto [s, l] : nodes[(size_t)order[(size_t)i]].mem) {
            const Layer &L = layer(s, l);
            const int p = pool_of[(size_t)s][(size_t)l];
            if (p >= 0) {   // the conv writes its pool's (pooled) tensor only
                const Layer &Pl = layer(s, p);
                TInfo &t = T[{s, p}];
                t.bytes = (size_t)nfr[(size_t)s] * Pl.out_h * Pl.out_w * Pl.out_phys * esz;
                t.prod = i;
            } else if (!direct_output(L)) {
                TInfo &t = T[{s, l}];
                t.bytes = (size_t)nfr[(size_t)s] * L.out_h * L.out_w * L.out_phys * esz;
                t.prod = i;
            }
        }
    auto use = [&](int s, int p, int i) {
        auto it = T.find({s, p});
        if (it != T.end()) it->second.users.push_back(i);
    };
    for (int i = 0; i < NN; ++i)
        for (auto [s, l] : nodes[(size_t)order[(size_t)i]].mem) {
            const Layer &L = layer(s, l);
            use(s, L.src0, i);
            if (L.op == GEMEL_OP_CONCAT) use(s, L.src1, i);
            if (L.res >= 0) use(s, L.res, i);
        }
    for (size_t e = 0; e < exports.size(); ++e) use(exports[e].first, exports[e].second, NN + (int)e);
    auto done_before = [&](const TInfo &t, const TInfo &u) {
        if (u.prod < 0) return false;
        if (t.users.empty()) return before(t.prod, u.prod);
        for (int x : t.users)
            if (!before(x, u.prod)) return false;
        return true;
    };
    std::vector<TInfo *> tv;
    for (auto &kv : T)
        if (kv.second.bytes) tv.push_back(&kv.second);
    std::stable_sort(tv.begin(), tv.end(), [](TInfo *x, TInfo *y) { return x->bytes > y->bytes; });
    std::vector<TInfo *> placed;
    size_t arena = 0;
    for (TInfo *t : tv) {
        std::vector<std::pair<size_t, size_t>> busy;
        for (TInfo *o : placed)
            if (!done_before(*o, *t) && !done_before(*t, *o)) busy.push_back({o->off, o->off + o->bytes});
        std::sort(busy.begin(), busy.end());
        size_t cand = 0;
        for (auto &bz : busy) {
            if (cand + t->bytes <= bz.first) break;
            cand = std::max(cand, (size_t)round_up((int64_t)bz.second, 256));
        }
        t->off = cand;
        arena = std::max(arena, cand + (size_t)round_up((int64_t)t->bytes, 256));
        placed.push_back(t);
    }
    P.arena_bytes = arena;
    P.static_mem = static_base != nullptr;
    size_t static_used = (size_t)round_up((int64_t)arena, 256);
    if (static_base) {
        if (static_used > static_cap)
            return fail(ctx, GEMEL_EBUDGET,
                        "the activations of this model set and frame count (" + std::to_string(arena) +
                            " bytes) exceed the static scratch of " + std::to_string(static_cap) + " bytes");
        P.arena = static_base;
    } else if (arena && alloc_device(ctx, &P.arena, arena) != hipSuccess) {
        P.arena = nullptr;
        (void)hipGetLastError();
        return fail(ctx, GEMEL_ENOMEM, "device allocation of the activation arena failed");
    }
    auto tptr = [&](int s, int l) -> void * {
        auto it = T.find({s, l});
        if (it == T.end() || !it->second.bytes) return nullptr;
        return (char *)P.arena + it->second.off;
    };
    P.events.assign((size_t)n_events, nullptr);
    for (auto &ev : P.events)
        if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess)
            return fail(ctx, GEMEL_EDEVICE, "event creation failed");
    if (P.n_streams > 1) {
        if (hipEventCreateWithFlags(&P.ev_fork, hipEventDisableTiming) != hipSuccess)
            return fail(ctx, GEMEL_EDEVICE, "event creation failed");
        P.ev_join.assign((size_t)P.n_streams, nullptr);
        for (int k = 1; k < P.n_streams; ++k)
            if (hipEventCreateWithFlags(&P.ev_join[(size_t)k], hipEventDisableTiming) != hipSuccess)
                return fail(ctx, GEMEL_EDEVICE, "event creation failed");
    }
    // stream, waits and event record of the launches of step i
    std::vector<std::pair<size_t, size_t>> step_range((size_t)NS, {0, 0});
    auto tag_launches = [&](size_t first, int i) {
        step_range[(size_t)i] = {first, P.launches.size()};
        if (first >= P.launches.size()) return;
        for (size_t k = first; k < P.launches.size(); ++k) {
            P.launches[k].stream = stream_of[(size_t)i];
            P.launches[k].step = i;
        }
        for (int p : preds[(size_t)i])
            if (stream_of[(size_t)p] != stream_of[(size_t)i]) P.launches[first].waits.push_back(event_of[(size_t)p]);
        P.launches.back().record = event_of[(size_t)i];
    };

    // ---- launches ----
    std::vector<size_t> step_partial((size_t)NS, 0);  // split-K bytes per step
    // input pack, grouped by input shape, at most GEMEL_MAX_SEG models each
    {
        std::map<std::vector<int>, std::vector<int>> by_shape;
        for (int s = 0; s < S; ++s) {
            const Model &m = model(s);
            by_shape[{m.in_c, m.in_h, m.in_w, m.in_cp}].push_back(s);
        }
        for (auto &kv : by_shape)
            for (size_t b = 0; b < kv.second.size(); b += GEMEL_MAX_SEG) {
                Launch L;
                L.type = L_PACK;
                L.kind = GEMEL_K_PACK;
                L.bf16 = bf16;
                EwArgs &a = L.ew;
                a.H = kv.first[1]; a.W = kv.first[2]; a.Co = kv.first[3]; a.c_logical = kv.first[0];
                a.nseg = 0;
                for (size_t i = b; i < std::min(kv.second.size(), b + GEMEL_MAX_SEG); ++i) {
                    const int s = kv.second[i];
                    EwSeg &sg = a.seg[a.nseg];
                    sg.in0 = nullptr;
                    sg.in1 = nullptr;
                    sg.out = tptr(s, -1);
                    sg.frames = nfr[(size_t)s];
                    a.max_frames = std::max(a.max_frames, sg.frames);
                    L.patches.push_back({Patch::FRAMES, s, 0, a.nseg});
                    L.bytes += (double)sg.frames * a.H * a.W * a.c_logical * (4.0 + esz);
                    a.nseg++;
                }
                P.launches.push_back(L);
            }
    }
    P.n_pack = (int)P.launches.size();
    auto in_ptr = [&](int s, int p) { return p < 0 ? tptr(s, -1) : tptr(s, p); };

    for (int step = 0; step < NN; ++step) {
        const size_t first_launch = P.launches.size();
        struct Tagger {
            std::function<void()> f;
            ~Tagger() { f(); }
        } tagger{[&, first_launch, step] { tag_launches(first_launch, step); }};
        const Node &nd = nodes[(size_t)order[(size_t)step]];
        const auto [s0, l0] = nd.mem[0];
        const Layer &L0 = layer(s0, l0);
        if (L0.op == GEMEL_OP_CONV || L0.op == GEMEL_OP_FC) {
            Blob *blob = L0.exec.get();
            const bool pooled = pool_of[(size_t)s0][(size_t)l0] >= 0;   // alike for every member
            int64_t M = 0;
            for (auto [s, l] : nd.mem) M += (int64_t)nfr[(size_t)s] * layer(s, l).out_h * layer(s, l).out_w;
            const bool direct = direct_output(L0);
            const bool fc_small = L0.op == GEMEL_OP_FC && bf16 && M <= 64;
            const bool fc_f32 = L0.op == GEMEL_OP_FC && !bf16;
            // weight chunks: a resident blob is one chunk with no copy
            std::vector<std::pair<int64_t, int64_t>> rows;  // (row0, nrows)
            if (blob->w_dev || ctx->cache_mode) {   // resident, or cached when the round runs
                rows.push_back({0, blob->rows});
            } else {
                const int64_t row_bytes = blob->k * (int64_t)blob->elem;
                int64_t per = ctx->staging_slot_bytes / row_bytes;
                per = per >= 128 ? per / 128 * 128 : per / 8 * 8;
                if (direct && per < blob->rows)
                    return fail(ctx, GEMEL_EBUDGET, "an output layer's weights exceed one staging slot");
                for (int64_t r0 = 0; r0 < blob->rows; r0 += per) rows.push_back({r0, std::min(per, blob->rows - r0)});
            }
            double in_elems = 0;
            for (auto [s, l] : nd.mem)
                in_elems += (double)nfr[(size_t)s] * layer(s, l).in_h * layer(s, l).in_w * layer(s, l).in_c;
            const double kdepth = L0.op == GEMEL_OP_CONV ? (double)L0.kh * L0.kw * L0.cin : (double)L0.cin;
            int members = 0;
            for (auto [s, l] : nd.mem) members += nfr[(size_t)s] > 0 ? 1 : 0;
            // unmerged layers of several models in one node: a grouped
            // launch, every member with its own weights
            const bool grouped = nd.mem.size() > 1 && L0.group < 0;
            for (auto [row0, nrows] : rows) {
                Launch Lc;
                Lc.bf16 = bf16;
                Lc.merged = members > 1 && !grouped;
                const double co = (double)std::max<int64_t>(0, std::min<int64_t>(nrows, L0.out_c - row0));
                Lc.flops = 2.0 * (double)M * co * kdepth;
                Lc.bytes = co * kdepth * esz * (grouped ? members : 1) + in_elems * esz +
                           (double)M * co * (direct ? 4.0 : esz) / (pooled ? 4.0 : 1.0) +
                           (L0.res >= 0 ? (double)M * co * esz : 0.0);
                if (ctx->cache_mode) {
                    // the weights' cache address is set when the round runs
                    if (!grouped) Lc.wblobs.push_back(blob);
                } else if (!blob->w_dev) {
                    Lc.chunk = (int)P.chunks.size();
                    P.chunks.push_back(Chunk{blob, row0, nrows});
                    P.streamed_bytes += P.chunks.back().bytes();
                }
                const void *wptr = blob->w_dev ? (const void *)((const char *)blob->w_dev) : nullptr;
                if (fc_small || fc_f32) {
                    FcArgs &a = Lc.fc;
                    a.w = wptr;
                    a.M = (int)M; a.N = (int)nrows; a.K = (int)blob->k;
                    a.out_cs = L0.out_phys; a.cout = L0.out_c;
                    a.act = L0.act; a.slope = L0.slope;
                    a.out_mode = direct ? OUT_NCHW_F32 : OUT_NHWC;
                    a.nseg = 0;
                    int f = 0;
                    int64_t slice_frames = 0;
                    for (auto [s, l] : nd.mem) {
                        if (!nfr[(size_t)s]) continue;
                        FcSeg &sg = a.seg[a.nseg];
                        // a grouped launch: each member with its own weights
                        // and scale/shift
                        Blob *mb = grouped ? layer(s, l).exec.get() : blob;
                        if (grouped && ctx->cache_mode) Lc.wblobs.push_back(mb);
                        sg.in = in_ptr(s, layer(s, l).src0);
                        sg.out = direct ? nullptr : (void *)((char *)tptr(s, l) + row0 * esz);
                        sg.scale = mb->aff_dev + row0;
                        sg.shift = mb->aff_dev + mb->rows + row0;
                        sg.w = grouped ? mb->w_dev : nullptr;
                        sg.f_start = f;
                        slice_frames = grouped ? std::max<int64_t>(slice_frames, nfr[(size_t)s]) : M;
                        if (direct) Lc.patches.push_back({Patch::OUTPUT, s, layer(s, l).out_index, a.nseg});
                        f += nfr[(size_t)s];
                        a.nseg++;
                    }
                    Lc.kind = GEMEL_K_FC;
                    a.grouped = grouped ? 1 : 0;
                    if (fc_f32) {
                        a.k_splits = 1;
                        a.k_per_split = a.K;
                        Lc.type = L_FC_F32;
                    } else {
                        pick_fc_config(slice_frames, a.N, a.K, a.k_splits, a.k_per_split);
                        Lc.type = L_FC_BF16;
                        if (a.k_splits > 1) {
                            step_partial[(size_t)step] = std::max(step_partial[(size_t)step], (size_t)a.k_splits * a.M * a.N * 4);
                            if (ctx->opt.splitk_fused)
                                Lc.ctr_n = (a.N + 63) / 64 * (grouped ? a.nseg : 1);
                        }
                    }
                    P.launches.push_back(Lc);
                    if (Lc.type == L_FC_BF16 && a.k_splits > 1 && !Lc.ctr_n) {
                        Launch R = Lc;
                        R.type = L_FC_REDUCE;
                        R.kind = GEMEL_K_SPLITK_REDUCE;
                        R.flops = 0;
                        R.bytes = (double)a.k_splits * a.M * a.N * 4.0;
                        R.chunk = -1;
                        P.launches.push_back(R);
                    }
                    continue;
                }
                ConvArgs &a = Lc.conv;
                a.w = wptr;
                a.zero = ctx->zero_page;
                a.M = (int)M; a.N = (int)nrows; a.K = (int)blob->k;
                if (L0.op == GEMEL_OP_CONV) {
                    a.H = L0.in_h; a.W = L0.in_w; a.Cin = L0.in_phys; a.in_cs = L0.in_phys;
                    a.Ho = L0.out_h; a.Wo = L0.out_w;
                    a.kh = L0.kh; a.kw = L0.kw; a.stride = L0.stride; a.pad = L0.pad;
                } else {  // FC over many frames: a 1x1 conv on a 1x1 map with Cin = K
                    a.H = a.W = 1; a.Cin = a.in_cs = (int)blob->k;
                    a.Ho = a.Wo = 1;
                    a.kh = a.kw = 1; a.stride = 1; a.pad = 0;
                }
                a.out_cs = L0.out_phys;
                a.out_pair = L0.out_paired ? L0.out_cp : 0;
                a.cout = direct ? std::min<int>((int)nrows, L0.out_c - (int)row0) : L0.out_c;
                a.act = L0.act; a.slope = L0.slope;
                a.res_mode = L0.res_mode; a.has_res = L0.res >= 0;
                a.out_mode = direct ? OUT_NCHW_F32 : pooled ? OUT_NHWC_POOL2 : OUT_NHWC;
                a.nseg = 0;
                a.hetero = 0;
                int f = 0;
                int64_t m_acc = 0;
                for (auto [s, l] : nd.mem) {
                    if (!nfr[(size_t)s]) continue;
                    const Layer &L = layer(s, l);
                    ConvSeg &sg = a.seg[a.nseg];
                    sg.in = in_ptr(s, L.src0);
                    sg.res = L.res >= 0 ? (const void *)((char *)tptr(s, L.res) + row0 * esz) : nullptr;
                    const int wl = pooled ? pool_of[(size_t)s][(size_t)l] : l;   // the tensor written
                    sg.out = direct ? nullptr : (void *)((char *)tptr(s, wl) + row0 * esz);
                    Blob *mb = L.exec.get();   // the member's own parameters (grouped)
                    sg.w = grouped ? mb->w_dev : nullptr;
                    if (grouped && ctx->cache_mode) Lc.wblobs.push_back(mb);
                    sg.scale = mb->aff_dev + row0;
                    sg.shift = mb->aff_dev + mb->rows + row0;
                    sg.f_start = f;
                    sg.m_start = (int32_t)m_acc;
                    sg.H = L.in_h; sg.W = L.in_w; sg.Ho = L.out_h; sg.Wo = L.out_w;
                    if (L.in_h != L0.in_h || L.in_w != L0.in_w || L.out_h != L0.out_h || L.out_w != L0.out_w)
                        a.hetero = 1;
                    m_acc += (int64_t)nfr[(size_t)s] * L.out_h * L.out_w;
                    if (direct) Lc.patches.push_back({Patch::OUTPUT, s, L.out_index, a.nseg});
                    f += nfr[(size_t)s];
                    a.nseg++;
                }
                if (!a.nseg) continue;
                a.grouped = grouped ? 1 : 0;
                a.uni_affine = 1;
                for (int i = 1; i < a.nseg; ++i)
                    if (a.seg[i].scale != a.seg[0].scale || a.seg[i].shift != a.seg[0].shift) a.uni_affine = 0;
                if (bf16) {
                    // DMA tiles: masked rows read the zero page at their
                    // channel offset, so the pixel stride must fit it
                    const bool dma_ok = a.in_cs % 8 == 0 && (a.uni_affine || a.grouped) &&
                                        (int64_t)a.in_cs * 2 + 128 <= GEMEL_ZERO_PAGE_BYTES;
                    const int dma_depth = !dma_ok ? 0 : a.Cin % 64 == 0 ? 64 : a.Cin % 32 == 0 ? 32 : 0;
                    // 8-channel inputs (the RGB stems) take the stem kernel
                    const bool stem = a.Cin == 8 && a.in_cs == 8 && a.kh * a.kw <= STEM_MAX_TAPS && a.uni_affine &&
                                      (ctx->opt.conv_tile < 0 || ctx->opt.conv_tile == TILE_STEM);
                    if (stem) {
                        Lc.tile = TILE_STEM;
                        a.k_splits = 1;
                        a.k_per_split = a.K;
                    } else {
                        pick_conv_config(a.M, a.N, a.K, dma_depth, ctx->opt.conv_tile == TILE_STEM ? TILE_64x64 : ctx->opt.conv_tile,
                                         ctx->opt.conv_splits, a.hetero != 0 || a.grouped != 0, pooled, Lc.tile, a.k_splits,
                                         a.k_per_split);
                        // measured choice where nothing is forced and the
                        // launch's tensors all exist at plan time
                        if (ctx->opt.tune && can_tune && ctx->opt.conv_tile < 0 && (ctx->opt.conv_splits <= 0 || pooled) &&
                            !direct && (blob->w_dev || ctx->cache_mode))
                            tune_conv(ctx, a, dma_depth, bf16, Lc.tile, a.k_splits, a.k_per_split);
                    }
                    if (tile_is_dma(Lc.tile) && !conv_dma_supported(a, Lc.tile)) {
                        if (pooled || a.hetero || a.grouped)
                            return fail(ctx, GEMEL_ESTATE,
                                        "internal: fused pool, mixed sizes or grouped launch without an LDS-DMA tile");
                        Lc.tile = TILE_64x64;
                    }
                    Lc.type = L_CONV_BF16;
                    Lc.kind = L0.op == GEMEL_OP_CONV ? GEMEL_K_CONV_MFMA : GEMEL_K_FC;
                } else {
                    a.k_splits = 1;
                    a.k_per_split = a.K;
                    Lc.type = L_CONV_F32;
                    Lc.kind = L0.op == GEMEL_OP_CONV ? GEMEL_K_CONV_F32 : GEMEL_K_FC;
                }
                if (a.k_splits > 1) {
                    step_partial[(size_t)step] = std::max(step_partial[(size_t)step], (size_t)a.k_splits * a.M * a.N * 4);
                    const int bm = conv_tile_bm(Lc.tile), bn = conv_tile_bn(Lc.tile);
                    const int tiles = (int)conv_tiles(a, bm, bn);
                    if (fuse_splitk(ctx, tiles)) Lc.ctr_n = tiles;
                }
                P.launches.push_back(Lc);
                if (a.k_splits > 1 && !Lc.ctr_n) {
                    Launch R;
                    R.type = L_CONV_REDUCE;
                    R.kind = GEMEL_K_SPLITK_REDUCE;
                    R.bytes = (double)a.k_splits * a.M * a.N * 4.0;
                    R.bf16 = bf16;
                    R.patches = Lc.patches;
                    R.red = reduce_args(a);
                    P.launches.push_back(R);
                }
            }
            continue;
        }
        // memory-bound ops: one launch with one segment per member
        Launch Le;
        Le.bf16 = bf16;
        EwArgs &a = Le.ew;
        a.H = L0.in_h; a.W = L0.in_w; a.C = L0.in_phys;
        a.Ho = L0.out_h; a.Wo = L0.out_w; a.Co = L0.out_phys;
        a.k = L0.kh; a.stride = L0.stride; a.pad = L0.pad;
        a.C1 = L0.src1_phys;
        a.nseg = 0;
        for (auto [s, l] : nd.mem) {
            if (!nfr[(size_t)s]) continue;
            const Layer &L = layer(s, l);
            EwSeg &sg = a.seg[a.nseg++];
            sg.in0 = in_ptr(s, L.src0);
            sg.in1 = L.op == GEMEL_OP_CONCAT ? in_ptr(s, L.src1) : nullptr;
            sg.out = tptr(s, l);
            sg.frames = nfr[(size_t)s];
            a.max_frames = std::max(a.max_frames, sg.frames);
        }
        if (!a.nseg) continue;
        switch (L0.op) {
        case GEMEL_OP_MAXPOOL: Le.type = L_MAXPOOL; Le.kind = GEMEL_K_POOL; break;
        case GEMEL_OP_AVGPOOL: Le.type = L_AVGPOOL; Le.kind = GEMEL_K_POOL; break;
        case GEMEL_OP_UPSAMPLE2X: Le.type = L_UPSAMPLE; Le.kind = GEMEL_K_ROUTE; break;
        default: Le.type = L_CONCAT; Le.kind = GEMEL_K_ROUTE; break;
        }
        for (int i = 0; i < a.nseg; ++i)
            Le.bytes += (double)a.seg[i].frames * esz *
                        ((double)L0.in_h * L0.in_w * L0.in_c + (double)L0.out_h * L0.out_w * L0.out_c);
        P.launches.push_back(Le);
    }
    // outputs that are also read internally (or not conv/fc): export to NCHW f32
    for (size_t e = 0; e < exports.size(); ++e) {
        const auto [s, l] = exports[e];
        const Layer &L = model(s).layers[(size_t)l];
        const size_t first_launch = P.launches.size();
        Launch Le;
        Le.type = L_EXPORT;
        Le.kind = GEMEL_K_EXPORT;
        Le.bytes = (double)nfr[(size_t)s] * L.out_h * L.out_w * L.out_c * (esz + 4.0);
        Le.bf16 = bf16;
        EwArgs &a = Le.ew;
        a.H = L.out_h; a.W = L.out_w; a.C = L.out_phys; a.c_logical = L.out_c;
        a.nseg = 1;
        a.seg[0].in0 = tptr(s, l);
        a.seg[0].in1 = nullptr;
        a.seg[0].out = nullptr;
        a.seg[0].frames = nfr[(size_t)s];
        a.max_frames = a.seg[0].frames;
        Le.patches.push_back({Patch::OUTPUT, s, L.out_index, 0});
        P.launches.push_back(Le);
        tag_launches(first_launch, NN + (int)e);
    }
    if (const char *tr = std::getenv("GEMEL_TRACE_PLAN"); tr && tr[0] == '1') {
        static const char *names[] = {"pack", "conv_bf16", "conv_f32", "conv_reduce", "fc_bf16", "fc_f32",
                                      "fc_reduce", "maxpool", "avgpool", "upsample", "concat", "export"};
        for (size_t i = 0; i < P.launches.size(); ++i) {
            const Launch &L = P.launches[i];
            const bool cv = L.type == L_CONV_BF16 || L.type == L_CONV_F32;
            const bool fcl = L.type == L_FC_BF16 || L.type == L_FC_F32;
            std::fprintf(stderr, "plan %zu %s M=%d N=%d K=%d tile=%d splits=%d segs=%d gflop=%.3f mb=%.2f st=%d\n", i,
                         names[L.type], cv ? L.conv.M : fcl ? L.fc.M : 0, cv ? L.conv.N : fcl ? L.fc.N : 0,
                         cv ? L.conv.K : fcl ? L.fc.K : 0, L.tile,
                         cv ? L.conv.k_splits : fcl ? L.fc.k_splits : 0,
                         cv ? L.conv.nseg : fcl ? L.fc.nseg : L.ew.nseg, L.flops / 1e9, L.bytes / 1e6, L.stream);
        }
    }
    // ---- split-K partial sums: a region per split-K step, first fit; two
    // steps share bytes only when one precedes the other ----
    {
        std::vector<size_t> poff((size_t)NS, 0);
        std::vector<int> ps;
        for (int i = 0; i < NS; ++i)
            if (step_partial[(size_t)i]) ps.push_back(i);
        std::stable_sort(ps.begin(), ps.end(),
                         [&](int x, int y) { return step_partial[(size_t)x] > step_partial[(size_t)y]; });
        std::vector<int> done;
        size_t total = 0;
        for (int i : ps) {
            std::vector<std::pair<size_t, size_t>> busy;
            for (int j : done)
                if (!before(i, j) && !before(j, i)) busy.push_back({poff[(size_t)j], poff[(size_t)j] + step_partial[(size_t)j]});
            std::sort(busy.begin(), busy.end());
            size_t cand = 0;
            for (auto &bz : busy) {
                if (cand + step_partial[(size_t)i] <= bz.first) break;
                cand = std::max(cand, (size_t)round_up((int64_t)bz.second, 256));
            }
            poff[(size_t)i] = cand;
            total = std::max(total, cand + (size_t)round_up((int64_t)step_partial[(size_t)i], 256));
            done.push_back(i);
        }
        if (total) {
            if (static_base) {
                if (static_used + total > static_cap)
                    return fail(ctx, GEMEL_EBUDGET,
                                "activations and split-K partial sums exceed the static scratch of " +
                                    std::to_string(static_cap) + " bytes");
                P.partial = (float *)((char *)static_base + static_used);
                static_used += (size_t)round_up((int64_t)total, 256);
            } else if (alloc_device(ctx, (void **)&P.partial, total) != hipSuccess) {
                P.partial = nullptr;
                (void)hipGetLastError();
                return fail(ctx, GEMEL_ENOMEM, "device allocation of the split-K buffer failed");
            }
            P.partial_bytes = total;
            for (auto &L : P.launches) {
                if (L.step < 0 || !step_partial[(size_t)L.step]) continue;
                float *pp = P.partial + poff[(size_t)L.step] / sizeof(float);
                L.conv.partial = pp;
                L.red.partial = pp;
                L.fc.partial = pp;
            }
        }
    }

    // ---- arrival counters of the fused split-K launches: zeroed once here;
    // each launch leaves its counters at zero again ----
    {
        size_t total = 0;
        for (auto &L : P.launches) total += (size_t)L.ctr_n;
        if (total) {
            P.counters_n = total;
            if (static_base) {
                // cleared by every round: the static scratch is shared
                if (static_used + total * sizeof(int32_t) > static_cap)
                    return fail(ctx, GEMEL_EBUDGET,
                                "activations, split-K partial sums and counters exceed the static scratch of " +
                                    std::to_string(static_cap) + " bytes");
                P.counters = (int32_t *)((char *)static_base + static_used);
                static_used += (size_t)round_up((int64_t)(total * sizeof(int32_t)), 256);
            } else {
                if (alloc_device(ctx, (void **)&P.counters, total * sizeof(int32_t)) != hipSuccess) {
                    P.counters = nullptr;
                    (void)hipGetLastError();
                    return fail(ctx, GEMEL_ENOMEM, "device allocation of the split-K counters failed");
                }
                const std::vector<int32_t> zeros(total, 0);
                if (hipMemcpy(P.counters, zeros.data(), total * sizeof(int32_t), hipMemcpyHostToDevice) != hipSuccess)
                    return fail(ctx, GEMEL_EDEVICE, "clearing the split-K counters failed");
            }
            size_t off = 0;
            for (auto &L : P.launches) {
                if (!L.ctr_n) continue;
                L.conv.counters = P.counters + off;
                L.fc.counters = P.counters + off;
                off += (size_t)L.ctr_n;
            }
        }
    }

    // ---- prefetch: each conv launch reads the weights of the next conv
    // launch of its stream into the caches after its own tiles (resident,
    // ungrouped weights; at most 16 MiB). In a round that moves more bytes
    // than the memory-side cache holds, weights last read a round ago come
    // from HBM, and the latency of those first reads holds up every early
    // depth step of a launch with few steps in flight. A smaller round
    // finds its weights in that cache and would only pay for the reads. ----
    constexpr double kMemSideCacheBytes = 256.0 * (1 << 20);
    double round_bytes = 0;
    for (const Launch &L : P.launches) round_bytes += L.bytes;
    const bool prefetch = ctx->opt.prefetch == 2 || (ctx->opt.prefetch == 1 && round_bytes > kMemSideCacheBytes);
    for (size_t i = 0; i < P.launches.size(); ++i) {
        Launch &L = P.launches[i];
        if (L.type != L_CONV_BF16) continue;
        L.conv.pf = nullptr;
        L.conv.pf_bytes = 0;
        if (!prefetch) continue;
        for (size_t j = i + 1; j < P.launches.size(); ++j) {
            const Launch &M = P.launches[j];
            if (M.stream != L.stream || M.type != L_CONV_BF16) continue;
            if (M.chunk < 0 && M.wblobs.empty() && !M.conv.grouped && M.conv.w) {
                L.conv.pf = M.conv.w;
                L.conv.pf_bytes = (uint32_t)std::min<int64_t>((int64_t)M.conv.N * M.conv.K * 2, 16 << 20) & ~15u;
            }
            break;
        }
    }

    // ---- dependencies of each launch (the edges of a graph round) ----
    {
        std::vector<std::vector<int>> tails((size_t)NS);  // launches that complete step i
        for (int i = 0; i < NS; ++i) {
            std::set<int> d;
            for (int p : preds[(size_t)i]) d.insert(tails[(size_t)p].begin(), tails[(size_t)p].end());
            bool reads_input = false;
            if (i < NN)
                for (auto [s, l] : nodes[(size_t)order[(size_t)i]].mem) {
                    const Layer &L = layer(s, l);
                    reads_input |= L.src0 < 0 || (L.op == GEMEL_OP_CONCAT && L.src1 < 0);
                }
            if (reads_input)
                for (int k = 0; k < P.n_pack; ++k) d.insert(k);
            const auto [f, e] = step_range[(size_t)i];
            if (f < e) {
                P.launches[f].deps.assign(d.begin(), d.end());
                for (size_t k = f + 1; k < e; ++k) P.launches[k].deps = {(int)k - 1};
                tails[(size_t)i] = {(int)e - 1};
            } else {
                tails[(size_t)i].assign(d.begin(), d.end());
            }
        }
    }
    return GEMEL_OK;
}

// ----------------------------------------------------------------------------
// inference round
// ----------------------------------------------------------------------------
namespace {

struct CallPtrs {
    std::vector<const void *> frames;  // per slot
    std::vector<void *> outputs;       // per slot output, flattened by slot
};

hipError_t launch_one(Launch &L, const CallPtrs &cp, const Plan &P, void *wptr, const Sink &st) {
    for (const Patch &p : L.patches) {
        if (p.kind == Patch::FRAMES) {
            L.ew.seg[p.seg].in0 = cp.frames[(size_t)p.slot];
        } else {
            void *o = cp.outputs[(size_t)(P.out_base[(size_t)p.slot] + p.out_idx)];
            switch (L.type) {
            case L_CONV_BF16:
            case L_CONV_F32: L.conv.seg[p.seg].out = o; break;
            case L_CONV_REDUCE: L.red.seg[p.seg].out = o; break;
            case L_FC_BF16:
            case L_FC_F32:
            case L_FC_REDUCE: L.fc.seg[p.seg].out = o; break;
            default: L.ew.seg[p.seg].out = o; break;
            }
        }
    }
    if (wptr) {
        L.conv.w = wptr;
        L.fc.w = wptr;
    }
    switch (L.type) {
    case L_PACK: return launch_pack(L.ew, L.bf16, st);
    case L_CONV_BF16: return launch_conv_bf16(L.conv, L.tile, st);
    case L_CONV_F32: return launch_conv_f32(L.conv, st);
    case L_CONV_REDUCE: return launch_conv_reduce(L.red, L.bf16, st);
    case L_FC_BF16: return launch_fc_bf16(L.fc, st);
    case L_FC_F32: return launch_fc_f32(L.fc, st);
    case L_FC_REDUCE: return launch_fc_reduce(L.fc, L.bf16, st);
    case L_MAXPOOL: return launch_maxpool(L.ew, L.bf16, st);
    case L_AVGPOOL: return launch_avgpool(L.ew, L.bf16, st);
    case L_UPSAMPLE: return launch_upsample2x(L.ew, L.bf16, st);
    case L_CONCAT: return launch_concat(L.ew, L.bf16, st);
    case L_EXPORT: return launch_export(L.ew, L.bf16, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

// After a failure part way through a round: the work already enqueued on
// the worker streams and the side (weight copy) stream is joined back to
// the caller's stream, best effort, so that a synchronisation of that
// stream covers the partial round and the next round's launches are
// ordered after it.
static void join_partial_round(gemel_ctx *ctx, Plan &P, hipStream_t st) {
    for (int k = 1; k < P.n_streams; ++k) {
        if (hipEventRecord(P.ev_join[(size_t)k], ctx->workers[(size_t)k - 1]) == hipSuccess)
            (void)hipStreamWaitEvent(st, P.ev_join[(size_t)k], 0);
    }
    if (ctx->side && hipEventRecord(ctx->ev_side_join, ctx->side) == hipSuccess)
        (void)hipStreamWaitEvent(st, ctx->ev_side_join, 0);
    // the partial round shares the arena and the staging slots with the next
    // round, which, on another stream, waits for this event
    if (ctx->ev_round_done && hipEventRecord(ctx->ev_round_done, st) == hipSuccess) {
        ctx->round_stream = st;
        ctx->round_seen = true;
        const int slot = ctx->cache_round & 1;
        if (ctx->cache_mode && ctx->ev_cache_done[slot] &&
            hipEventRecord(ctx->ev_cache_done[slot], st) == hipSuccess)
            ctx->cache_done_round[slot] = ctx->cache_round;
    }
    (void)hipGetLastError();
}

// Every launch of the plan in plan order on one stream, with no event and
// no other stream (a round captured into the caller's graph). Plan order is
// a topological order of the launches' dependencies, and the plan's arena
// and split-K regions are shared only between launches ordered by those
// dependencies, so one stream is always a valid schedule.
static gemel_status enqueue_serial(gemel_ctx *ctx, Plan &P, const CallPtrs &cp, hipStream_t st) {
    for (Launch &L : P.launches) {
        Sink sk;
        sk.stream = st;
        const hipError_t e = launch_one(L, cp, P, nullptr, sk);
        if (e != hipSuccess) return fail(ctx, GEMEL_EDEVICE, std::string("kernel launch: ") + hipGetErrorString(e));
    }
    return GEMEL_OK;
}

static gemel_status enqueue_body(gemel_ctx *ctx, Plan &P, const CallPtrs &cp, hipStream_t st);

// Weight cache (GEMEL_OPT_SWAP_CACHE): bring every blob the round's models
// need into the cache before their launches. Needed blobs are taken in
// first-use order (models by id, then layers); one that is not cached is
// placed first-fit (lowest offset with a large enough free run, 256-byte
// aligned) after evicting, while no run fits, cached blobs that are not
// pinned, unshared before shared, larger before smaller, lower number
// first. Pinned: the round's blobs and the shared blobs of the models of
// the next round (gemel_set_next_round). The whole decision is made before
// anything changes, so a round whose pinned blobs do not fit changes
// nothing. Copies run on the side stream after the previous round's work
// (their regions may still be read by it); each loaded blob records an
// event its launches wait for.
static gemel_status cache_round(gemel_ctx *ctx, Plan &P, hipStream_t st) {
    ctx->cache_round++;
    std::vector<Blob *> needed;
    std::set<Blob *> in_needed;
    for (int id : P.model_ids)
        for (auto &l : ctx->models[(size_t)id]->layers)
            if (l.exec && in_needed.insert(l.exec.get()).second) needed.push_back(l.exec.get());
    std::set<Blob *> pinned(in_needed);
    for (int id : ctx->next_models)
        if (id >= 0 && id < (int)ctx->models.size())
            for (auto &l : ctx->models[(size_t)id]->layers)
                if (l.exec && l.exec->users > 1) pinned.insert(l.exec.get());
    auto sz = [](const Blob *b) { return (int64_t)round_up((int64_t)b->w_bytes(), 256); };
    std::map<Blob *, int64_t> at;   // the cache after this round
    for (auto &b : ctx->placed)
        if (b->cache_off >= 0) at[b.get()] = b->cache_off;
    std::vector<Blob *> loaded, evicted;
    for (Blob *b : needed) {
        if (at.count(b)) continue;
        const int64_t size = sz(b);
        int64_t off = -1;
        while (true) {
            std::vector<std::pair<int64_t, int64_t>> taken;
            for (auto &kv : at) taken.push_back({kv.second, kv.second + sz(kv.first)});
            std::sort(taken.begin(), taken.end());
            int64_t pos = 0;
            off = -1;
            for (auto &t : taken) {
                if (t.first - pos >= size) {
                    off = pos;
                    break;
                }
                pos = std::max(pos, t.second);
            }
            if (off < 0 && (int64_t)ctx->cache_cap - pos >= size) off = pos;
            if (off >= 0) break;
            Blob *v = nullptr;
            for (auto &kv : at) {
                Blob *c = kv.first;
                if (pinned.count(c)) continue;
                auto key = [&](const Blob *x) { return std::make_tuple(x->users > 1, -sz(x), x->index); };
                if (!v || key(c) < key(v)) v = c;
            }
            if (!v)
                return fail(ctx, GEMEL_EBUDGET,
                            "the weights this round pins do not fit the weight cache of " +
                                std::to_string(ctx->cache_cap) + " bytes");
            at.erase(v);
            evicted.push_back(v);
        }
        at[b] = off;
        loaded.push_back(b);
    }
    // commit
    const int R = ctx->cache_round;
    int64_t lb = 0, eb = 0;
    for (Blob *v : evicted) {
        ctx->cache_freed.push_back({v->cache_off, sz(v), v->used_round});
        v->cache_off = -1;
        v->w_dev = nullptr;
        eb += sz(v);
    }
    for (Blob *b : needed) b->used_round = R;
    // a copy overwrites bytes that earlier rounds may still read: it waits
    // for the end of the latest round that used them (the previous round
    // only if it did; rounds further back are done by then or are waited
    // for through the end of a later round, which follows them)
    auto done_event = [&](int round) -> hipEvent_t {
        const int slot = round & 1;
        return ctx->cache_done_round[slot] == round ? ctx->ev_cache_done[slot] : ctx->ev_round_done;
    };
    int waited = 0;   // the side stream has waited for every round < waited + 1
    auto wait_for = [&](int round) -> gemel_status {
        if (round < 1 || round <= waited || !ctx->round_seen) return GEMEL_OK;
        HIPCHK(hipStreamWaitEvent(ctx->side, done_event(round), 0), "hipStreamWaitEvent");
        waited = round;
        return GEMEL_OK;
    };
    for (Blob *b : loaded) {
        b->cache_off = at[b];
        b->w_dev = ctx->cache_base + b->cache_off;
        // the latest round that used any freed bytes this copy overwrites
        int last = 0;
        for (const auto &f : ctx->cache_freed)
            if (f.off < b->cache_off + sz(b) && b->cache_off < f.off + f.size) last = std::max(last, f.round);
        {
            const gemel_status ws = wait_for(std::max(last, R - 2));
            if (ws) return ws;
        }
        lb += sz(b);
        ctx->copies_issued++;
        if (ctx->opt.fail_copy_at && ctx->copies_issued == ctx->opt.fail_copy_at) {
            ctx->opt.fail_copy_at = 0;
            b->cache_off = -1;   // its copy never ran: not cached
            b->w_dev = nullptr;
            return fail(ctx, GEMEL_EDEVICE, "injected failure of a weight copy");
        }
        HIPCHK(hipMemcpyAsync(b->w_dev, b->w_pinned, b->w_bytes(), hipMemcpyHostToDevice, ctx->side),
               "hipMemcpyAsync (weight cache)");
        HIPCHK(hipEventRecord(b->ev_loaded, ctx->side), "hipEventRecord");
        b->loaded_round = ctx->cache_round;
    }
    // freed bytes now occupied by this round's blobs need no record; the
    // rest keep theirs (entries older than two rounds only ever ask for a
    // wait on a round the side stream has passed)
    std::vector<gemel_ctx::Freed> keep;
    for (const auto &f : ctx->cache_freed) {
        bool covered = false;
        for (Blob *b : loaded)
            if (b->cache_off <= f.off && f.off + f.size <= b->cache_off + sz(b)) covered = true;
        if (!covered && f.round >= R - 2) keep.push_back(f);
    }
    ctx->cache_freed.swap(keep);
    ctx->round_loaded = lb;
    ctx->round_evicted = eb;
    (void)st;
    return GEMEL_OK;
}

// Packs the plan's streamed chunks, in consumption order, into one pinned
// host image cut into copy segments of at most one staging slot: a round
// then copies each segment with one transfer instead of one per chunk.
static gemel_status stream_image(gemel_ctx *ctx, Plan &P) {
    const size_t cap = ctx->staging_slot_bytes;
    size_t total = 0, used = cap;   // forces a first segment
    P.chunk_seg.assign(P.chunks.size(), 0);
    P.chunk_off.assign(P.chunks.size(), 0);
    std::vector<Plan::CopySeg> segs;
    for (size_t c = 0; c < P.chunks.size(); ++c) {
        const size_t b = P.chunks[c].bytes();
        const size_t at = (size_t)round_up((int64_t)used, 256);
        if (at + b > cap) {
            segs.push_back({(size_t)round_up((int64_t)total, 256), 0});
            used = 0;
        } else {
            used = at;
        }
        Plan::CopySeg &sg = segs.back();
        P.chunk_seg[c] = (int)segs.size() - 1;
        P.chunk_off[c] = used;
        used += b;
        sg.bytes = used;
        total = sg.off + sg.bytes;
    }
    void *img = nullptr;
    if (alloc_pinned(ctx, &img, std::max<size_t>(total, 1)) != hipSuccess)
        return fail(ctx, GEMEL_ENOMEM, "pinned host allocation of the streamed-weight image failed");
    for (size_t c = 0; c < P.chunks.size(); ++c) {
        const Chunk &ch = P.chunks[c];
        std::memcpy((char *)img + segs[(size_t)P.chunk_seg[c]].off + P.chunk_off[c],
                    ch.blob->w_pinned + (size_t)(ch.row0 * ch.blob->k) * ch.blob->elem, ch.bytes());
    }
    std::vector<hipEvent_t> evs(P.chunks.size(), nullptr);
    for (auto &e : evs)
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
            e = nullptr;
            for (auto x : evs)
                if (x) (void)hipEventDestroy(x);
            (void)hipHostFree(img);
            return fail(ctx, GEMEL_EDEVICE, "event creation failed");
        }
    P.image = img;
    P.copy_segs = std::move(segs);
    P.ev_chunk = std::move(evs);
    return GEMEL_OK;
}

static gemel_status enqueue(gemel_ctx *ctx, Plan &P, const CallPtrs &cp, hipStream_t st) {
    const gemel_status s = enqueue_body(ctx, P, cp, st);
    if (s) join_partial_round(ctx, P, st);
    return s;
}

static gemel_status enqueue_body(gemel_ctx *ctx, Plan &P, const CallPtrs &cp, hipStream_t st) {
    if (ctx->cache_mode) {
        const gemel_status s = cache_round(ctx, P, st);
        if (s) return s;
    }
    const int nslots = ctx->staging_slots;
    const int nseg = (int)P.copy_segs.size();
    int next_copy = 0;
    auto slot_ptr = [&](int seg) { return (char *)ctx->staging + (size_t)(seg % nslots) * ctx->staging_slot_bytes; };
    // copies of segments [next_copy, upto]: each first waits for every
    // consumer of the segment that last used its slot (on any stream, in
    // this round or the previous one)
    auto issue_copies = [&](int upto) -> gemel_status {
        for (; next_copy < nseg && next_copy <= upto; ++next_copy) {
            const Plan::CopySeg &sg = P.copy_segs[(size_t)next_copy];
            const int slot = next_copy % nslots;
            ctx->copies_issued++;
            if (ctx->opt.fail_copy_at && ctx->copies_issued == ctx->opt.fail_copy_at) {
                ctx->opt.fail_copy_at = 0;
                return fail(ctx, GEMEL_EDEVICE, "injected failure of a weight copy");
            }
            for (auto &u : ctx->slot_users[(size_t)slot])
                HIPCHK(hipStreamWaitEvent(ctx->side, u.second, 0), "hipStreamWaitEvent");
            ctx->slot_users[(size_t)slot].clear();
            HIPCHK(hipMemcpyAsync(slot_ptr(next_copy), (char *)P.image + sg.off, sg.bytes, hipMemcpyHostToDevice,
                                  ctx->side),
                   "hipMemcpyAsync (weight swap-in)");
            HIPCHK(hipEventRecord(ctx->ev_copied[(size_t)slot], ctx->side), "hipEventRecord");
        }
        return GEMEL_OK;
    };
    if (nseg) {
        gemel_status s = issue_copies(nslots - 1);
        if (s) return s;
    }
    // per stream: the latest segment whose copy it has waited for (copies
    // complete in order on the copy stream, so later consumers of that or
    // an earlier segment on the stream need no wait of their own)
    std::vector<int> waited((size_t)std::max(P.n_streams, 1), -1);
    hipStream_t streams[8] = {st};
    for (int k = 1; k < P.n_streams; ++k) streams[k] = ctx->workers[(size_t)k - 1];
    for (size_t li = 0; li < P.launches.size(); ++li) {
        Launch &L = P.launches[li];
        if ((int)li == P.n_pack && P.n_streams > 1) {
            HIPCHK(hipEventRecord(P.ev_fork, st), "hipEventRecord");
            for (int k = 1; k < P.n_streams; ++k) HIPCHK(hipStreamWaitEvent(streams[k], P.ev_fork, 0), "hipStreamWaitEvent");
        }
        const hipStream_t ls = streams[L.stream];
        for (int ev : L.waits) HIPCHK(hipStreamWaitEvent(ls, P.events[(size_t)ev], 0), "hipStreamWaitEvent");
        void *wptr = nullptr;
        if (!L.wblobs.empty()) {
            // cached weights: wait for this round's copies of them, then
            // read them at their current cache addresses
            for (Blob *b : L.wblobs)
                if (b->loaded_round == ctx->cache_round)
                    HIPCHK(hipStreamWaitEvent(ls, b->ev_loaded, 0), "hipStreamWaitEvent");
            const bool fcl = L.type == L_FC_BF16 || L.type == L_FC_REDUCE;
            if (!fcl && L.conv.grouped)
                for (size_t i = 0; i < L.wblobs.size() && (int)i < L.conv.nseg; ++i) L.conv.seg[i].w = L.wblobs[i]->w_dev;
            if (fcl && L.fc.grouped)
                for (size_t i = 0; i < L.wblobs.size() && (int)i < L.fc.nseg; ++i) L.fc.seg[i].w = L.wblobs[i]->w_dev;
            wptr = L.wblobs[0]->w_dev;
        }
        if (L.chunk >= 0) {
            const int seg = P.chunk_seg[(size_t)L.chunk];
            gemel_status s = issue_copies(seg + nslots - 1);
            if (s) return s;
            if (seg > waited[(size_t)L.stream]) {
                HIPCHK(hipStreamWaitEvent(ls, ctx->ev_copied[(size_t)(seg % nslots)], 0), "hipStreamWaitEvent");
                waited[(size_t)L.stream] = seg;
            }
            wptr = slot_ptr(seg) + P.chunk_off[(size_t)L.chunk];
        }
        const int subset = L.kind == GEMEL_K_CONV_MFMA && L.merged ? GEMEL_K_CONV_MERGED : -1;
        Profile::Rec rec{nullptr, nullptr, L.kind, subset};
        if (ctx->opt.profile) {
            for (hipEvent_t *ev : {&rec.a, &rec.b}) {
                if (ctx->prof.pool.empty()) {
                    hipEvent_t e2;
                    HIPCHK(hipEventCreate(&e2), "hipEventCreate");
                    ctx->prof.pool.push_back(e2);
                }
                *ev = ctx->prof.pool.back();
                ctx->prof.pool.pop_back();
            }
            ctx->prof.pending.push_back(rec);
        }
        Sink sk;
        sk.stream = ls;
        // profiled: the events take the kernel's own start and end times
        sk.ev_start = rec.a;
        sk.ev_stop = rec.b;
        hipError_t e = launch_one(L, cp, P, wptr, sk);
        if (e != hipSuccess) return fail(ctx, GEMEL_EDEVICE, std::string("kernel launch: ") + hipGetErrorString(e));
        if (ctx->opt.profile) {
            for (int k : {L.kind, subset}) {
                if (k < 0) continue;
                ctx->prof.flops[k] += L.flops;
                ctx->prof.bytes[k] += L.bytes;
                ctx->prof.launches[k] += 1;
            }
        }
        if (L.chunk >= 0) {
            hipEvent_t e = P.ev_chunk[(size_t)L.chunk];
            HIPCHK(hipEventRecord(e, ls), "hipEventRecord");
            auto &users = ctx->slot_users[(size_t)(P.chunk_seg[(size_t)L.chunk] % nslots)];
            auto u = std::find_if(users.begin(), users.end(), [&](const auto &x) { return x.first == ls; });
            if (u != users.end())
                u->second = e;   // stream order: this consumer ends after the earlier one
            else
                users.push_back({ls, e});
        }
        if (L.record >= 0) HIPCHK(hipEventRecord(P.events[(size_t)L.record], ls), "hipEventRecord");
    }
    if ((int)P.launches.size() <= P.n_pack && P.n_streams > 1) {
        HIPCHK(hipEventRecord(P.ev_fork, st), "hipEventRecord");
        for (int k = 1; k < P.n_streams; ++k) HIPCHK(hipStreamWaitEvent(streams[k], P.ev_fork, 0), "hipStreamWaitEvent");
    }
    for (int k = 1; k < P.n_streams; ++k) {
        HIPCHK(hipEventRecord(P.ev_join[(size_t)k], streams[k]), "hipEventRecord");
        HIPCHK(hipStreamWaitEvent(st, P.ev_join[(size_t)k], 0), "hipStreamWaitEvent");
    }
    return GEMEL_OK;
}

// Edges of a graph over plan launches.
enum GraphEdges {
    EDGES_CHAIN = 0,    // each launch follows the previous one of the list
    EDGES_DATA = 1,     // each launch follows the launches whose results it reads
    EDGES_STREAMS = 2   // data edges plus the previous launch of its plan stream
};

// A HIP graph built node by node over the launches `idx` (in plan order),
// one kernel node per launch, with the given edges. Only plans without
// streamed weights are graphed.
static gemel_status build_graph(gemel_ctx *ctx, Plan &P, const CallPtrs &cp, const std::vector<int> &idx,
                                int edges, hipGraphExec_t *out) {
    hipGraph_t g = nullptr;
    HIPCHK(hipGraphCreate(&g, 0), "hipGraphCreate");
    // nodes that stand for launch i: its own node, or, when the launcher had
    // nothing to do, the nodes its dependencies stand for
    std::vector<std::vector<hipGraphNode_t>> done(P.launches.size());
    std::vector<hipGraphNode_t> deps;
    gemel_status st = GEMEL_OK;
    int prev = -1;
    std::vector<int> stream_last(8, -1);
    for (size_t k = 0; k < idx.size() && !st; ++k) {
        const int i = idx[k];
        const Launch &L = P.launches[(size_t)i];
        deps.clear();
        if (edges == EDGES_CHAIN) {
            if (prev >= 0) deps = done[(size_t)prev];
        } else {
            for (int d : L.deps) deps.insert(deps.end(), done[(size_t)d].begin(), done[(size_t)d].end());
            const int sp = stream_last[(size_t)L.stream];
            if (edges == EDGES_STREAMS && sp >= 0) deps.insert(deps.end(), done[(size_t)sp].begin(), done[(size_t)sp].end());
            std::sort(deps.begin(), deps.end());
            deps.erase(std::unique(deps.begin(), deps.end()), deps.end());
        }
        prev = i;
        stream_last[(size_t)L.stream] = i;
        hipGraphNode_t node = nullptr;
        Sink sk;
        sk.graph = g;
        sk.deps = deps.data();
        sk.ndeps = deps.size();
        sk.node = &node;
        const hipError_t e = launch_one(P.launches[(size_t)i], cp, P, nullptr, sk);
        if (e != hipSuccess)
            st = fail(ctx, GEMEL_EDEVICE, std::string("graph kernel node: ") + hipGetErrorString(e));
        else if (node)
            done[(size_t)i] = {node};
        else
            done[(size_t)i] = deps;
    }
    hipGraphExec_t ex = nullptr;
    if (!st) {
        const hipError_t e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
        if (e != hipSuccess) st = fail(ctx, GEMEL_EDEVICE, std::string("hipGraphInstantiate: ") + hipGetErrorString(e));
    }
    (void)hipGraphDestroy(g);
    if (!st) *out = ex;
    return st;
}

// Split the launches into segments (see Segment). With several streams the
// input packs form a segment of their own, so that the other streams fork
// right after them.
static void build_segments(Plan &P) {
    P.segs.clear();
    std::vector<int> open(8, -1);  // open segment of each stream
    for (size_t i = 0; i < P.launches.size(); ++i) {
        const Launch &L = P.launches[i];
        int &o = open[(size_t)L.stream];
        const bool fork = (int)i == P.n_pack && P.n_streams > 1;
        if (o < 0 || !L.waits.empty() || fork) {
            for (int &x : open)
                if (fork) x = -1;
            Segment sg;
            sg.stream = L.stream;
            sg.waits = L.waits;
            P.segs.push_back(sg);
            o = (int)P.segs.size() - 1;
        }
        P.segs[(size_t)o].launches.push_back((int)i);
        if (L.record >= 0) {
            P.segs[(size_t)o].record = L.record;
            o = -1;
        }
    }
}

// Execution modes of a round.
enum RoundMode { MODE_EAGER = 0, MODE_SEGMENTS = 1, MODE_DAG = 2, MODE_STREAMGRAPH = 3, MODE_SERIAL = 4 };

// One graph round of the per-stream segments, launched in plan order, each
// after its cross-stream waits, worker streams forked after the packs and
// joined at the end.
static gemel_status launch_segments_body(gemel_ctx *ctx, Plan &P, hipStream_t st);

static gemel_status launch_segments(gemel_ctx *ctx, Plan &P, hipStream_t st) {
    const gemel_status s = launch_segments_body(ctx, P, st);
    if (s) join_partial_round(ctx, P, st);
    return s;
}

static gemel_status launch_segments_body(gemel_ctx *ctx, Plan &P, hipStream_t st) {
    hipStream_t streams[8] = {st};
    for (int k = 1; k < P.n_streams; ++k) streams[k] = ctx->workers[(size_t)k - 1];
    bool forked = P.n_streams == 1;
    for (const Segment &sg : P.segs) {
        if (!forked && sg.launches.front() >= P.n_pack) {
            HIPCHK(hipEventRecord(P.ev_fork, st), "hipEventRecord");
            for (int k = 1; k < P.n_streams; ++k) HIPCHK(hipStreamWaitEvent(streams[k], P.ev_fork, 0), "hipStreamWaitEvent");
            forked = true;
        }
        const hipStream_t ss = streams[sg.stream];
        for (int ev : sg.waits) HIPCHK(hipStreamWaitEvent(ss, P.events[(size_t)ev], 0), "hipStreamWaitEvent");
        HIPCHK(hipGraphLaunch(sg.exec, ss), "hipGraphLaunch");
        if (sg.record >= 0) HIPCHK(hipEventRecord(P.events[(size_t)sg.record], ss), "hipEventRecord");
    }
    if (!forked) {
        HIPCHK(hipEventRecord(P.ev_fork, st), "hipEventRecord");
        for (int k = 1; k < P.n_streams; ++k) HIPCHK(hipStreamWaitEvent(streams[k], P.ev_fork, 0), "hipStreamWaitEvent");
    }
    for (int k = 1; k < P.n_streams; ++k) {
        HIPCHK(hipEventRecord(P.ev_join[(size_t)k], streams[k]), "hipEventRecord");
        HIPCHK(hipStreamWaitEvent(st, P.ev_join[(size_t)k], 0), "hipStreamWaitEvent");
    }
    return GEMEL_OK;
}

static void drop_graphs(Plan &P) {
    for (auto &g : P.graph) {
        if (g) (void)hipGraphExecDestroy(g);
        g = nullptr;
    }
    for (auto &sg : P.segs)
        if (sg.exec) (void)hipGraphExecDestroy(sg.exec);
    P.segs.clear();
}

gemel_status run(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models, const void *const *frames,
                 const int32_t *n_frames, void *const *outputs, hipStream_t stream) {
    // canonical slot order: active models sorted by id
    std::vector<std::pair<int, int>> act;  // (model id, caller index)
    std::vector<int> caller_out_base((size_t)n_models);
    for (int i = 0, ob = 0; i < n_models; ++i) {
        caller_out_base[(size_t)i] = ob;
        ob += (int)ctx->models[(size_t)model_ids[i]]->outputs.size();
        if (n_frames[i] > 0) act.push_back({model_ids[i], i});
    }
    if (act.empty()) return GEMEL_OK;
    std::sort(act.begin(), act.end());
    std::vector<int> ids, nfr, key;
    for (auto [id, ci] : act) {
        ids.push_back(id);
        nfr.push_back(n_frames[ci]);
        key.push_back(id);
        key.push_back(n_frames[ci]);
    }
    DeviceScope scope(ctx->device);
    // A round captured into the caller's graph may only enqueue work: the
    // weight placement and the plan (allocations, synchronous copies, tuning
    // runs) must come from an earlier round outside capture, and it runs on
    // the caller's stream alone.
    bool capturing = false;
    if (stream) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        HIPCHK(hipStreamIsCapturing(stream, &cs), "hipStreamIsCapturing");
        capturing = cs != hipStreamCaptureStatusNone;
    }
    if (capturing && !ctx->weights_ready)
        return fail(ctx, GEMEL_ESTATE, "weights are not placed yet: run one round outside stream capture first");
    gemel_status st = materialise(ctx);
    if (st) return st;
    // The null stream gets a single-stream plan (its implicit synchronisation
    // with other streams would serialise the worker streams anyway). So does
    // a round that streams weights through the staging slots: it is bound
    // by the copies, and one stream consumes the slots in copy order with
    // one wait per slot (measured 15% faster than three streams on the
    // 40%-budget workload)
    bool streams_weights = false;
    if (!ctx->cache_mode)
        for (auto [id, ci] : act)
            for (auto &l : ctx->models[(size_t)id]->layers)
                if (l.exec && !l.exec->w_dev) streams_weights = true;
    const bool will_graph = ctx->opt.use_graph && !ctx->opt.profile && stream != nullptr;
    const int nstreams = stream == nullptr || streams_weights ? 1 : ctx->opt.streams;
    key.push_back(nstreams);
    auto it = ctx->plans.find(key);
    if (it == ctx->plans.end()) {
        if (capturing)
            return fail(ctx, GEMEL_ESTATE,
                        "no plan for this model set and frame counts yet: run one round outside stream capture first");
        auto P = std::make_unique<Plan>();
        const int saved = ctx->opt.streams;
        ctx->opt.streams = nstreams;
        st = build_plan(ctx, ids, nfr, *P, true);
        ctx->opt.streams = saved;
        if (st) {
            if (!P->static_mem) {
                if (P->arena) (void)hipFree(P->arena);
                if (P->partial) (void)hipFree(P->partial);
                if (P->counters) (void)hipFree(P->counters);
            }
            for (auto ev : P->events)
                if (ev) (void)hipEventDestroy(ev);
            if (P->ev_fork) (void)hipEventDestroy(P->ev_fork);
            for (auto ev : P->ev_join)
                if (ev) (void)hipEventDestroy(ev);
            return st;
        }
        it = ctx->plans.emplace(key, std::move(P)).first;
    }
    Plan &P = *it->second;
    ctx->last_plan = &P;
    CallPtrs cp;
    for (auto [id, ci] : act) {
        cp.frames.push_back(frames[ci]);
        const int no = (int)ctx->models[(size_t)id]->outputs.size();
        for (int o = 0; o < no; ++o) cp.outputs.push_back(outputs[caller_out_base[(size_t)ci] + o]);
    }
    if (capturing) {
        if (!P.chunks.empty() || ctx->cache_mode)
            return fail(ctx, GEMEL_ESTATE, "a round that streams or caches weights cannot be captured");
        if (ctx->opt.profile) return fail(ctx, GEMEL_ESTATE, "a profiled round cannot be captured");
        ctx->last_mode = MODE_SERIAL;
        return enqueue_serial(ctx, P, cp, stream);
    }
    if (!P.chunks.empty() && !P.image) {
        st = stream_image(ctx, P);
        if (st) return st;
    }
    // rounds share the plan's arena and split-K regions and the staging
    // slots: a round on another stream than the previous one first waits
    // for the previous round's work
    if (ctx->round_seen && ctx->round_stream != stream)
        HIPCHK(hipStreamWaitEvent(stream, ctx->ev_round_done, 0), "hipStreamWaitEvent");
    auto round_done = [&]() -> gemel_status {
        HIPCHK(hipEventRecord(ctx->ev_round_done, stream), "hipEventRecord");
        ctx->round_stream = stream;
        ctx->round_seen = true;
        if (ctx->cache_mode) {
            const int slot = ctx->cache_round & 1;
            HIPCHK(hipEventRecord(ctx->ev_cache_done[slot], stream), "hipEventRecord");
            ctx->cache_done_round[slot] = ctx->cache_round;
        }
        return GEMEL_OK;
    };
    const bool graphable = will_graph && P.chunks.empty() && !ctx->cache_mode;
    ctx->tuning_left = 0;
    if (!graphable) {
        ctx->last_mode = MODE_EAGER;
        st = enqueue(ctx, P, cp, stream);
        if (!st && ctx->opt.profile) ctx->prof.rounds++;
        return st ? st : round_done();
    }
    // mode of this round: a single-stream plan is one chain graph; a
    // multi-stream plan uses the mode set by the options, or, with autotune,
    // one untimed round of each candidate mode, then kTimed timed rounds of
    // each with the modes interleaved (so that clock drift affects all
    // alike), and then the mode with the smallest median
    constexpr int kTimed = 4;
    constexpr int kNCand = 4;
    static const int kCand[kNCand] = {MODE_SEGMENTS, MODE_STREAMGRAPH, MODE_DAG, MODE_EAGER};
    int mode = ctx->opt.graph_dag ? MODE_DAG : MODE_SEGMENTS;
    bool timed = false, tuning = false;
    if (P.n_streams == 1) {
        mode = MODE_SEGMENTS;
    } else if (ctx->opt.autotune) {
        if (P.best_mode >= 0) {
            mode = P.best_mode;
        } else {
            mode = kCand[P.tune_round % kNCand];
            timed = P.tune_round >= kNCand;
            tuning = true;
            for (auto &ev : P.tune_ev)
                if (!ev) HIPCHK(hipEventCreate(&ev), "hipEventCreate");
        }
    }
    // graphs for this set of caller pointers (rebuilt when they change)
    if (P.graph_stream != stream || P.graph_frames != cp.frames || P.graph_outputs != cp.outputs) {
        drop_graphs(P);
        P.graph_stream = stream;
        P.graph_frames = cp.frames;
        P.graph_outputs = cp.outputs;
    }
    bool replay = true;
    if (mode == MODE_SEGMENTS && P.segs.empty()) {
        replay = false;
        build_segments(P);
        for (Segment &sg : P.segs) {
            st = build_graph(ctx, P, cp, sg.launches, EDGES_CHAIN, &sg.exec);
            if (st) {
                drop_graphs(P);
                return st;
            }
        }
    } else if ((mode == MODE_DAG || mode == MODE_STREAMGRAPH) && !P.graph[mode == MODE_DAG ? 0 : 1]) {
        replay = false;
        std::vector<int> all(P.launches.size());
        std::iota(all.begin(), all.end(), 0);
        st = build_graph(ctx, P, cp, all, mode == MODE_DAG ? EDGES_DATA : EDGES_STREAMS, &P.graph[mode == MODE_DAG ? 0 : 1]);
        if (st) return st;
    }
    ctx->last_mode = mode;
    if (timed) HIPCHK(hipEventRecord(P.tune_ev[0], stream), "hipEventRecord");
    if (mode == MODE_EAGER) {
        st = enqueue(ctx, P, cp, stream);
        if (st) return st;
    } else {
        if (replay) ctx->graph_replays++;
        if (mode == MODE_DAG || mode == MODE_STREAMGRAPH) {
            HIPCHK(hipGraphLaunch(P.graph[mode == MODE_DAG ? 0 : 1], stream), "hipGraphLaunch");
        } else {
            st = launch_segments(ctx, P, stream);
            if (st) return st;
        }
    }
    if (timed) {
        HIPCHK(hipEventRecord(P.tune_ev[1], stream), "hipEventRecord");
        HIPCHK(hipEventSynchronize(P.tune_ev[1]), "hipEventSynchronize");
        float ms = 0;
        HIPCHK(hipEventElapsedTime(&ms, P.tune_ev[0], P.tune_ev[1]), "hipEventElapsedTime");
        P.tune_ms[P.tune_round % kNCand][P.tune_round / kNCand - 1] = ms;
    }
    if (tuning) {
        if (++P.tune_round == kNCand * (1 + kTimed)) {
            static_assert(kTimed == 4, "median of four");
            int b = 0;
            double best = 0;
            for (int c = 0; c < kNCand; ++c) {
                double *t = P.tune_ms[c];
                std::sort(t, t + kTimed);
                const double med = 0.5 * (t[1] + t[2]);
                if (c == 0 || med < best) {
                    best = med;
                    b = c;
                }
            }
            P.best_mode = kCand[b];
        }
        ctx->tuning_left = P.best_mode >= 0 ? 0 : kNCand * (1 + kTimed) - P.tune_round;
    }
    return round_done();
}

// A round that allocates nothing (gemel_infer_noalloc): the weights must be
// placed already; the plan's arena, split-K partial sums and counters lie in
// the static scratch (one per device, shared by every call on it), and every
// launch runs in plan order on the caller's stream (no worker stream, event,
// graph or plan-time tuning).
gemel_status run_noalloc(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models, const void *const *frames,
                         const int32_t *n_frames, void *const *outputs, hipStream_t stream) {
    std::vector<std::pair<int, int>> act;  // (model id, caller index)
    std::vector<int> caller_out_base((size_t)n_models);
    for (int i = 0, ob = 0; i < n_models; ++i) {
        caller_out_base[(size_t)i] = ob;
        ob += (int)ctx->models[(size_t)model_ids[i]]->outputs.size();
        if (n_frames[i] > 0) act.push_back({model_ids[i], i});
    }
    if (act.empty()) return GEMEL_OK;
    if (!ctx->weights_ready)
        return fail(ctx, GEMEL_ESTATE, "weights are not placed yet: run one gemel_infer round first");
    if (ctx->opt.profile) return fail(ctx, GEMEL_ESTATE, "profiling is not available in allocation-free rounds");
    std::sort(act.begin(), act.end());
    std::vector<int> ids, nfr, key;
    for (auto [id, ci] : act) {
        ids.push_back(id);
        nfr.push_back(n_frames[ci]);
        key.push_back(id);
        key.push_back(n_frames[ci]);
    }
    key.push_back(-1);   // allocation-free plans: their own cache entries
    DeviceScope scope(ctx->device);
    bool capturing = false;
    if (stream) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        HIPCHK(hipStreamIsCapturing(stream, &cs), "hipStreamIsCapturing");
        capturing = cs != hipStreamCaptureStatusNone;
    }
    void *base = nullptr;
    HIPCHK(static_scratch(ctx->device, &base), "hipGetSymbolAddress (static scratch)");
    auto it = ctx->plans.find(key);
    if (it == ctx->plans.end()) {
        auto P = std::make_unique<Plan>();
        const int saved = ctx->opt.streams;
        ctx->opt.streams = 1;
        const gemel_status st = build_plan(ctx, ids, nfr, *P, false, base, GEMEL_STATIC_SCRATCH_BYTES);
        ctx->opt.streams = saved;
        if (st) {
            for (auto ev : P->events)
                if (ev) (void)hipEventDestroy(ev);
            return st;
        }
        it = ctx->plans.emplace(key, std::move(P)).first;
    }
    Plan &P = *it->second;
    if (!P.chunks.empty() || ctx->cache_mode) {
        ctx->last_plan = &P;
        return fail(ctx, GEMEL_ESTATE, "a round that streams or caches weights cannot run without allocation");
    }
    ctx->last_plan = &P;
    CallPtrs cp;
    for (auto [id, ci] : act) {
        cp.frames.push_back(frames[ci]);
        const int no = (int)ctx->models[(size_t)id]->outputs.size();
        for (int o = 0; o < no; ++o) cp.outputs.push_back(outputs[caller_out_base[(size_t)ci] + o]);
    }
    if (!capturing && ctx->round_seen && ctx->round_stream != stream)
        HIPCHK(hipStreamWaitEvent(stream, ctx->ev_round_done, 0), "hipStreamWaitEvent");
    Sink sk;
    sk.stream = stream;
    if (P.counters_n) {
        const hipError_t e = launch_fill_u32((uint32_t *)P.counters, P.counters_n, 0u, sk);
        if (e != hipSuccess) return fail(ctx, GEMEL_EDEVICE, std::string("clearing counters: ") + hipGetErrorString(e));
    }
    gemel_status st = enqueue_serial(ctx, P, cp, stream);
    if (st) return st;
    ctx->last_mode = MODE_SERIAL;
    if (!capturing) {
        HIPCHK(hipEventRecord(ctx->ev_round_done, stream), "hipEventRecord");
        ctx->round_stream = stream;
        ctx->round_seen = true;
    }
    return GEMEL_OK;
}

void profile_reset(gemel_ctx *ctx) {
    Profile &p = ctx->prof;
    if (!p.pending.empty() || !p.pool.empty()) {
        for (auto &r : p.pending) {
            (void)hipEventSynchronize(r.b);
            (void)hipEventDestroy(r.a);
            (void)hipEventDestroy(r.b);
        }
        for (auto e : p.pool) (void)hipEventDestroy(e);
    }
    const bool used = p.used;
    p = Profile();
    p.used = used;
}

gemel_status profile_read(gemel_ctx *ctx, gemel_kernel_stat *stats, int32_t *rounds) {
    Profile &p = ctx->prof;
    for (auto &r : p.pending) {
        float ms = 0.f;
        HIPCHK(hipEventSynchronize(r.b), "hipEventSynchronize");
        HIPCHK(hipEventElapsedTime(&ms, r.a, r.b), "hipEventElapsedTime");
        p.ms[r.kind] += ms;
        if (r.subset >= 0) p.ms[r.subset] += ms;
        p.pool.push_back(r.a);
        p.pool.push_back(r.b);
    }
    p.pending.clear();
    const double n = p.rounds ? (double)p.rounds : 1.0;
    for (int k = 0; k < GEMEL_K_COUNT; ++k) {
        stats[k].kind = k;
        stats[k].launches = (int32_t)((double)p.launches[k] / n + 0.5);
        stats[k].flops = p.flops[k] / n;
        stats[k].bytes = p.bytes[k] / n;
        stats[k].ms = p.ms[k] / n;
    }
    *rounds = p.rounds;
    return GEMEL_OK;
}

}  // namespace gemel
