// Per-model batch sizes of a round-robin schedule under a per-frame
// deadline (Section 3.2: the time-sharing scheduler's offline profiling
// picks the global list of per-model batch sizes that maximises the minimum
// per-model throughput within the SLA; Section 5.4: merging changes the
// swap delays that profiling accounts for; Section 6.1: a 100 ms SLA).
//
// gemel_profile_batches measures the cost table on the device;
// gemel_sla_batches chooses the batches from it. The cycle, latency and
// throughput rules are stated with gemel_sla_batches in the header.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <set>
#include <vector>

#include "internal.h"
#include "kernels.h"

using namespace gemel;

namespace {

struct Sched {
    int n, nb;
    const double *cost;   // [n][nb]
    const double *swap;   // [n] or null
    bool pipe;
    double sla, fps;

    double c(int m, int b) const { return cost[(size_t)m * nb + (b - 1)]; }
    double s(int m) const { return swap ? swap[m] : 0.0; }
    double cycle(const std::vector<int> &b) const {
        double t = 0;
        for (int i = 0; i < n; ++i)
            t += pipe ? std::max(c(i, b[(size_t)i]), s((i + 1) % n)) : s(i) + c(i, b[(size_t)i]);
        return t;
    }
    bool meets_sla(const std::vector<int> &b) const {
        const double t = cycle(b);
        for (int m = 0; m < n; ++m)
            if (t + c(m, b[(size_t)m]) > sla) return false;
        return true;
    }
    double value(const std::vector<int> &b) const {
        const double t = cycle(b) / 1000.0;
        double v = fps;
        for (int m = 0; m < n; ++m) v = std::min(v, b[(size_t)m] / t);
        return v;
    }
    // Smallest batch list with b_m >= theta * T(b) for every model: the
    // least fixed point of b -> max(1, ceil(theta * T(b))), reached by
    // iterating from all ones (T grows with b, so the map is monotone).
    // False when it needs more than nb frames for some model.
    bool least(double theta, std::vector<int> &b) const {
        b.assign((size_t)n, 1);
        for (;;) {
            const double per = theta * cycle(b) / 1000.0 * (1.0 - 1e-12);
            bool changed = false;
            for (int m = 0; m < n; ++m) {
                const double need = std::ceil(per);
                if (need > nb) return false;
                if ((int)need > b[(size_t)m]) {
                    b[(size_t)m] = (int)need;
                    changed = true;
                }
            }
            if (!changed) return true;
        }
    }
    bool ok(double theta, std::vector<int> &b) const { return least(theta, b) && meets_sla(b); }
};

}  // namespace

extern "C" gemel_status gemel_sla_batches(int32_t n_models, int32_t max_batch, const double *cost_ms,
                                          const double *swap_ms, int32_t pipelined, double sla_ms, double fps,
                                          int32_t *batch, double *min_fps, double *cycle_ms) {
    if (n_models <= 0 || max_batch <= 0 || !cost_ms || !batch) return GEMEL_EINVAL;
    if (!(sla_ms > 0) || !(fps > 0) || !std::isfinite(sla_ms) || !std::isfinite(fps)) return GEMEL_EINVAL;
    if ((int64_t)n_models * max_batch > (int64_t)1 << 24) return GEMEL_EINVAL;
    for (int m = 0; m < n_models; ++m) {
        for (int b = 0; b < max_batch; ++b) {
            const double c = cost_ms[(size_t)m * max_batch + b];
            if (!std::isfinite(c) || c < 0) return GEMEL_EINVAL;
            if (b > 0 && c < cost_ms[(size_t)m * max_batch + b - 1]) return GEMEL_EINVAL;
        }
        if (swap_ms && (!std::isfinite(swap_ms[m]) || swap_ms[m] < 0)) return GEMEL_EINVAL;
    }
    Sched S{n_models, max_batch, cost_ms, swap_ms, pipelined != 0, sla_ms, fps};
    std::vector<int> b, cand;
    // batches of one frame are the cheapest list: if they miss the SLA,
    // every list does
    b.assign((size_t)n_models, 1);
    if (!S.meets_sla(b)) return GEMEL_EBUDGET;
    // feasibility is monotone in the target throughput theta (a smaller
    // target has a componentwise smaller least list): bisect for the
    // largest feasible theta, then settle on the least list at the value
    // that list achieves
    double lo = S.value(b), hi = fps;
    if (S.ok(hi, cand)) {
        lo = hi;
    } else {
        for (int it = 0; it < 200 && hi - lo > lo * 1e-15; ++it) {
            const double mid = 0.5 * (lo + hi);
            if (S.ok(mid, cand))
                lo = mid;
            else
                hi = mid;
        }
    }
    if (!S.ok(lo, b)) return GEMEL_EBUDGET;   // not reached: lo is feasible
    // b meets its own value v, so the least list at v is componentwise no
    // larger, meets the SLA, and achieves at least v: move to it until the
    // value stops rising (the least list at the optimum is the optimum with
    // the shortest cycle and the smallest batches)
    for (int guard = 0; guard < 64; ++guard) {
        const double v = S.value(b);
        if (!S.ok(v, cand)) break;
        const bool rose = S.value(cand) > v;
        b = cand;
        if (!rose) break;
    }
    for (int m = 0; m < n_models; ++m) batch[m] = b[(size_t)m];
    if (min_fps) *min_fps = S.value(b);
    if (cycle_ms) *cycle_ms = S.cycle(b);
    return GEMEL_OK;
}

extern "C" gemel_status gemel_profile_batches(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                                              int32_t max_batch, int32_t reps, void *hip_stream, double *cost_ms) {
    if (!ctx) return GEMEL_EINVAL;
    if (!model_ids || n_models <= 0 || !cost_ms) return fail(ctx, GEMEL_EINVAL, "null argument or no models");
    if (max_batch <= 0 || max_batch > 4096) return fail(ctx, GEMEL_EINVAL, "max_batch must be in 1..4096");
    if (reps <= 0 || reps > 1000) return fail(ctx, GEMEL_EINVAL, "reps must be in 1..1000");
    std::set<int> seen;
    for (int i = 0; i < n_models; ++i) {
        if (model_ids[i] < 0 || model_ids[i] >= (int)ctx->models.size())
            return fail(ctx, GEMEL_EINVAL, "unknown model id " + std::to_string(model_ids[i]));
        if (!seen.insert(model_ids[i]).second) return fail(ctx, GEMEL_EINVAL, "model id listed twice");
    }
    const hipStream_t st = (hipStream_t)hip_stream;
    const gemel_status placed = materialise(ctx);   // the device, its streams and the weights
    if (placed) return placed;
    int prev_dev = -1;
    if (hipGetDevice(&prev_dev) != hipSuccess) prev_dev = -1;
    if (hipSetDevice(ctx->device) != hipSuccess) return fail(ctx, GEMEL_EDEVICE, "hipSetDevice");
    {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
            if (prev_dev >= 0) (void)hipSetDevice(prev_dev);
            return fail(ctx, GEMEL_ESTATE, "profiling cannot run while the stream is captured");
        }
    }
    std::vector<void *> bufs;
    std::vector<hipEvent_t> evs;
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(st);
        for (void *p : bufs) (void)hipFree(p);
        for (hipEvent_t e : evs)
            if (e) (void)hipEventDestroy(e);
        // the n_models * max_batch plans built here hold activation arenas
        drop_plans(ctx);
        if (prev_dev >= 0) (void)hipSetDevice(prev_dev);
    };
    auto dev_buf = [&](size_t bytes, void **p) -> gemel_status {
        if (alloc_device(ctx, p, bytes) != hipSuccess) {
            *p = nullptr;
            return fail(ctx, GEMEL_ENOMEM, "profiling buffers");
        }
        bufs.push_back(*p);
        Sink sk;
        sk.stream = st;
        if (launch_fill_u32((uint32_t *)*p, bytes / 4, 0u, sk) != hipSuccess)
            return fail(ctx, GEMEL_EDEVICE, "zero-filling a profiling buffer");
        return GEMEL_OK;
    };
    gemel_status status = GEMEL_OK;
    evs.assign((size_t)2 * reps, nullptr);
    for (auto &e : evs)
        if (hipEventCreate(&e) != hipSuccess) {
            e = nullptr;
            status = fail(ctx, GEMEL_EDEVICE, "hipEventCreate");
        }
    for (int i = 0; i < n_models && !status; ++i) {
        const int id = model_ids[i];
        const Model &m = *ctx->models[(size_t)id];
        void *frames = nullptr;
        status = dev_buf((size_t)max_batch * m.in_c * m.in_h * m.in_w * 4, &frames);
        std::vector<void *> outs;
        for (size_t o = 0; o < m.outputs.size() && !status; ++o) {
            const Layer &l = m.layers[(size_t)m.outputs[o]];
            void *p = nullptr;
            status = dev_buf((size_t)max_batch * l.out_c * l.out_h * l.out_w * 4, &p);
            outs.push_back(p);
        }
        double prev = 0;
        for (int b = 1; b <= max_batch && !status; ++b) {
            const void *fr = frames;
            // untimed rounds: plan build and plan-time tuning, then until
            // the round-mode tuner has settled
            for (int w = 0; w < 200 && !status; ++w) {
                status = run(ctx, &id, 1, &fr, &b, outs.data(), st);
                if (w > 0 && ctx->tuning_left == 0) break;
            }
            std::vector<float> ms((size_t)reps, 0.f);
            for (int r = 0; r < reps && !status; ++r) {
                if (hipEventRecord(evs[(size_t)2 * r], st) != hipSuccess) status = fail(ctx, GEMEL_EDEVICE, "hipEventRecord");
                if (!status) status = run(ctx, &id, 1, &fr, &b, outs.data(), st);
                if (!status && hipEventRecord(evs[(size_t)2 * r + 1], st) != hipSuccess)
                    status = fail(ctx, GEMEL_EDEVICE, "hipEventRecord");
            }
            if (status) break;
            if (hipStreamSynchronize(st) != hipSuccess) {
                status = fail(ctx, GEMEL_EDEVICE, "hipStreamSynchronize");
                break;
            }
            for (int r = 0; r < reps; ++r)
                if (hipEventElapsedTime(&ms[(size_t)r], evs[(size_t)2 * r], evs[(size_t)2 * r + 1]) != hipSuccess)
                    status = fail(ctx, GEMEL_EDEVICE, "hipEventElapsedTime");
            if (status) break;
            std::sort(ms.begin(), ms.end());
            const double med = reps % 2 ? ms[(size_t)reps / 2] : 0.5 * (ms[(size_t)reps / 2 - 1] + ms[(size_t)reps / 2]);
            prev = std::max(prev, med);
            cost_ms[(size_t)i * max_batch + (b - 1)] = prev;
        }
    }
    cleanup();
    return status;
}
