// C ABI entry points and the host-side registry: model registration
// (validation, shape inference, conversion of weights to kernel layout),
// merging (architectural-identity check, one copy per group), byte
// accounting and options. Nothing here calls the HIP runtime except
// gemel_infer (through run()) and gemel_destroy.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <map>
#include <new>
#include <set>
#include <tuple>

#include "internal.h"

using namespace gemel;

static thread_local std::string g_create_err;

namespace gemel {

gemel_status fail(gemel_ctx *ctx, gemel_status code, const std::string &msg) {
    if (ctx)
        ctx->err = msg;
    else
        g_create_err = msg;
    return code;
}

size_t unmerged_bytes(const gemel_ctx *ctx) {
    size_t b = 0;
    for (auto &m : ctx->models)
        for (auto &l : m->layers)
            if (l.own) b += l.own->bytes();
    return b;
}

size_t merged_bytes(const gemel_ctx *ctx) {
    std::set<const Blob *> seen;
    size_t b = 0;
    for (auto &m : ctx->models)
        for (auto &l : m->layers)
            if (l.eff && seen.insert(l.eff.get()).second) b += l.eff->bytes();
    return b;
}

}  // namespace gemel

static uint16_t host_f2bf(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Build the kernel-layout parameter blob of a conv or FC layer.
static std::shared_ptr<Blob> make_blob(const gemel_layer_desc &d, const Layer &l, int dtype) {
    auto b = std::make_shared<Blob>();
    b->elem = dtype == GEMEL_BF16 ? 2 : 4;
    b->rows = l.out_cp;
    if (l.op == GEMEL_OP_CONV)
        b->k = (int64_t)l.kh * l.kw * l.in_cp;
    else
        b->k = (int64_t)l.in_h * l.in_w * l.in_cp;
    b->w.assign((size_t)(b->rows * b->k) * b->elem, 0);
    auto put = [&](int64_t row, int64_t col, float v) {
        const size_t i = (size_t)(row * b->k + col);
        if (b->elem == 2) {
            const uint16_t h = host_f2bf(v);
            std::memcpy(&b->w[2 * i], &h, 2);
        } else {
            std::memcpy(&b->w[4 * i], &v, 4);
        }
    };
    if (l.op == GEMEL_OP_CONV) {
        // OIHW -> [o][r][s][c_p]
        for (int o = 0; o < l.cout; ++o)
            for (int c = 0; c < l.cin; ++c)
                for (int r = 0; r < l.kh; ++r)
                    for (int s = 0; s < l.kw; ++s)
                        put(o, ((int64_t)r * l.kw + s) * l.in_cp + c,
                            d.weight[(((int64_t)o * l.cin + c) * l.kh + r) * l.kw + s]);
    } else {
        // [o][c*H*W + h*W + w] (NCHW flatten) -> [o][(h*W + w)*C_p + c]
        const int64_t hw = (int64_t)l.in_h * l.in_w;
        for (int o = 0; o < l.cout; ++o)
            for (int c = 0; c < l.in_c; ++c)
                for (int64_t p = 0; p < hw; ++p)
                    put(o, p * l.in_cp + c, d.weight[(int64_t)o * l.cin + c * hw + p]);
    }
    b->scale.assign((size_t)b->rows, 0.f);
    b->shift.assign((size_t)b->rows, 0.f);
    for (int o = 0; o < l.cout; ++o) {
        const double bias = d.bias ? (double)d.bias[o] : 0.0;
        if (d.bn_gamma) {
            const double sc = (double)d.bn_gamma[o] / std::sqrt((double)d.bn_var[o] + (double)d.bn_eps);
            b->scale[o] = (float)sc;
            b->shift[o] = (float)(sc * (bias - (double)d.bn_mean[o]) + (double)d.bn_beta[o]);
        } else {
            b->scale[o] = 1.f;
            b->shift[o] = (float)bias;
        }
    }
    return b;
}

static gemel_status validate_and_build(gemel_ctx *ctx, const gemel_layer_desc *L, int32_t n,
                                       int32_t in_c, int32_t in_h, int32_t in_w, Model &m) {
    m.in_c = in_c;
    m.in_h = in_h;
    m.in_w = in_w;
    m.in_cp = (int)round_up(in_c, 8);
    m.layers.resize((size_t)n);
    for (int i = 0; i < n; ++i) {
        const gemel_layer_desc &d = L[i];
        Layer &l = m.layers[(size_t)i];
        auto bad = [&](gemel_status code, const std::string &why) {
            return fail(ctx, code, "layer " + std::to_string(i) + ": " + why);
        };
        if (d.op < GEMEL_OP_CONV || d.op > GEMEL_OP_CONCAT) return bad(GEMEL_EINVAL, "unknown op");
        if (d.src0 < -1 || d.src0 >= i) return bad(GEMEL_EINVAL, "src0 must be -1 or an earlier layer");
        if (d.act < GEMEL_ACT_NONE || d.act > GEMEL_ACT_LEAKY) return bad(GEMEL_EINVAL, "unknown activation");
        if (d.res_mode != GEMEL_RES_ADD_THEN_ACT && d.res_mode != GEMEL_RES_ACT_THEN_ADD)
            return bad(GEMEL_EINVAL, "unknown residual mode");
        const bool conv = d.op == GEMEL_OP_CONV, fc = d.op == GEMEL_OP_FC;
        if (d.op != GEMEL_OP_CONCAT && d.src1 != -1) return bad(GEMEL_EINVAL, "src1 is for concat only");
        if (!conv && d.res_src != -1) return bad(GEMEL_EINVAL, "residual is for conv only");
        if (!conv && !fc && d.act != GEMEL_ACT_NONE) return bad(GEMEL_EINVAL, "activation on a layer without weights");
        if (!conv && !fc && (d.weight || d.bias)) return bad(GEMEL_EINVAL, "weights on a layer without weights");
        const bool any_bn = d.bn_gamma || d.bn_beta || d.bn_mean || d.bn_var;
        const bool all_bn = d.bn_gamma && d.bn_beta && d.bn_mean && d.bn_var;
        if (any_bn && !all_bn) return bad(GEMEL_EINVAL, "batch norm needs gamma, beta, mean and var");
        if (any_bn && !conv) return bad(GEMEL_EINVAL, "batch norm is for conv only");
        if (any_bn && !(d.bn_eps >= 0.f)) return bad(GEMEL_EINVAL, "bad batch-norm eps");
        if ((conv || fc) && !d.weight) return bad(GEMEL_EINVAL, "missing weights");
        if (d.act == GEMEL_ACT_LEAKY && !std::isfinite(d.act_slope)) return bad(GEMEL_EINVAL, "bad leaky slope");

        l.op = d.op; l.src0 = d.src0; l.src1 = d.src1; l.cin = d.cin; l.cout = d.cout;
        l.kh = d.kh; l.kw = d.kw; l.stride = d.stride; l.pad = d.pad; l.act = d.act;
        l.slope = d.act == GEMEL_ACT_LEAKY ? d.act_slope : 0.f;
        l.res = d.res_src; l.res_mode = d.res_mode; l.is_output = d.is_output ? 1 : 0;
        l.has_bias = d.bias != nullptr; l.has_bn = all_bn;
        if (d.src0 < 0) {
            l.in_c = in_c; l.in_h = in_h; l.in_w = in_w;
        } else {
            const Layer &p = m.layers[(size_t)d.src0];
            l.in_c = p.out_c; l.in_h = p.out_h; l.in_w = p.out_w;
        }
        l.in_cp = (int)round_up(l.in_c, 8);
        switch (d.op) {
        case GEMEL_OP_CONV:
        case GEMEL_OP_MAXPOOL: {
            if (d.kh <= 0 || d.kw != d.kh || d.stride <= 0 || d.pad < 0)
                return bad(GEMEL_EINVAL, "window needs kh == kw > 0, stride > 0, pad >= 0");
            if (d.op == GEMEL_OP_MAXPOOL && d.pad >= d.kh) return bad(GEMEL_EINVAL, "maxpool pad must be < k");
            if (d.cin != l.in_c) return bad(GEMEL_ESHAPE, "cin does not match the producer");
            if (d.op == GEMEL_OP_MAXPOOL && d.cout != d.cin) return bad(GEMEL_ESHAPE, "maxpool cout != cin");
            if (d.cout <= 0) return bad(GEMEL_ESHAPE, "cout must be positive");
            const int64_t ho = ((int64_t)l.in_h + 2 * d.pad - d.kh) / d.stride + 1;
            const int64_t wo = ((int64_t)l.in_w + 2 * d.pad - d.kw) / d.stride + 1;
            if (l.in_h + 2 * d.pad < d.kh || l.in_w + 2 * d.pad < d.kw || ho <= 0 || wo <= 0)
                return bad(GEMEL_ESHAPE, "window larger than the padded input");
            l.out_c = d.cout; l.out_h = (int)ho; l.out_w = (int)wo;
            break;
        }
        case GEMEL_OP_FC:
            if ((int64_t)d.cin != (int64_t)l.in_c * l.in_h * l.in_w)
                return bad(GEMEL_ESHAPE, "fc cin must equal C*H*W of the producer");
            if (d.cout <= 0) return bad(GEMEL_ESHAPE, "cout must be positive");
            l.out_c = d.cout; l.out_h = 1; l.out_w = 1;
            break;
        case GEMEL_OP_AVGPOOL:
        case GEMEL_OP_UPSAMPLE2X: {
            if (d.cin != l.in_c || d.cout != d.cin) return bad(GEMEL_ESHAPE, "channels must match the producer");
            const int f = d.op == GEMEL_OP_UPSAMPLE2X ? 2 : 0;
            l.out_c = d.cout;
            l.out_h = f ? 2 * l.in_h : 1;
            l.out_w = f ? 2 * l.in_w : 1;
            break;
        }
        case GEMEL_OP_CONCAT: {
            if (d.src1 < -1 || d.src1 >= i) return bad(GEMEL_EINVAL, "src1 must be -1 or an earlier layer");
            int c1, h1, w1;
            if (d.src1 < 0) {
                c1 = in_c; h1 = in_h; w1 = in_w;
            } else {
                const Layer &p = m.layers[(size_t)d.src1];
                c1 = p.out_c; h1 = p.out_h; w1 = p.out_w;
            }
            if (h1 != l.in_h || w1 != l.in_w) return bad(GEMEL_ESHAPE, "concat inputs differ in H x W");
            if (l.in_c % 8 || c1 % 8) return bad(GEMEL_ESHAPE, "concat inputs need channels divisible by 8");
            if (d.cin != l.in_c || d.cout != l.in_c + c1) return bad(GEMEL_ESHAPE, "concat channels mismatch");
            l.src1_cp = c1;
            l.out_c = d.cout; l.out_h = l.in_h; l.out_w = l.in_w;
            break;
        }
        }
        l.out_cp = (int)round_up(l.out_c, 8);
        if (d.res_src >= 0) {
            if (d.res_src >= i) return bad(GEMEL_EINVAL, "res_src must be an earlier layer");
            const Layer &r = m.layers[(size_t)d.res_src];
            if (r.out_c != l.out_c || r.out_h != l.out_h || r.out_w != l.out_w)
                return bad(GEMEL_ESHAPE, "residual shape differs from the output");
        }
        if (l.is_output) {
            l.out_index = (int)m.outputs.size();
            m.outputs.push_back(i);
        }
    }
    for (int i = 0; i < n; ++i) {
        const Layer &l = m.layers[(size_t)i];
        for (int p : {l.src0, l.src1, l.res})
            if (p >= 0) m.layers[(size_t)p].consumers++;
    }
    if (m.outputs.empty()) return fail(ctx, GEMEL_EINVAL, "model has no output layer");
    return GEMEL_OK;
}

extern "C" {

gemel_status gemel_create(gemel_ctx **out, int32_t device, int32_t dtype, uint64_t budget) {
    if (!out) return fail(nullptr, GEMEL_EINVAL, "out is null");
    *out = nullptr;
    if (device < 0) return fail(nullptr, GEMEL_EINVAL, "negative device");
    if (dtype != GEMEL_F32 && dtype != GEMEL_BF16) return fail(nullptr, GEMEL_EINVAL, "unknown dtype");
    gemel_ctx *c = new (std::nothrow) gemel_ctx();
    if (!c) return fail(nullptr, GEMEL_ENOMEM, "out of host memory");
    c->device = device;
    c->dtype = dtype;
    c->budget = budget;
    *out = c;
    return GEMEL_OK;
}

gemel_status gemel_register_model(gemel_ctx *ctx, const gemel_layer_desc *layers, int32_t n_layers,
                                  int32_t in_c, int32_t in_h, int32_t in_w, int32_t *out_model_id) {
    if (!ctx) return GEMEL_EINVAL;
    if (!layers || n_layers <= 0 || !out_model_id) return fail(ctx, GEMEL_EINVAL, "null layers/out id or no layers");
    if (in_c <= 0 || in_h <= 0 || in_w <= 0) return fail(ctx, GEMEL_EINVAL, "frame shape must be positive");
    try {
        auto m = std::make_unique<Model>();
        gemel_status st = validate_and_build(ctx, layers, n_layers, in_c, in_h, in_w, *m);
        if (st != GEMEL_OK) return st;
        for (int i = 0; i < n_layers; ++i) {
            Layer &l = m->layers[(size_t)i];
            if (l.op == GEMEL_OP_CONV || l.op == GEMEL_OP_FC) {
                l.own = make_blob(layers[i], l, ctx->dtype);
                l.eff = l.own;
            }
        }
        m->id = (int)ctx->models.size();
        *out_model_id = m->id;
        ctx->models.push_back(std::move(m));
        ctx->weights_ready = false;
        drop_plans(ctx);
        return GEMEL_OK;
    } catch (const std::bad_alloc &) {
        return fail(ctx, GEMEL_ENOMEM, "out of host memory while copying weights");
    }
}

gemel_status gemel_merge(gemel_ctx *ctx, const gemel_group *groups, int32_t n_groups) {
    if (!ctx) return GEMEL_EINVAL;
    if (n_groups < 0 || (n_groups > 0 && !groups)) return fail(ctx, GEMEL_EINVAL, "bad group array");
    std::set<std::pair<int, int>> seen;
    for (int g = 0; g < n_groups; ++g) {
        const gemel_group &gr = groups[g];
        const std::string tag = "group " + std::to_string(g) + ": ";
        if (gr.n_members < 1 || !gr.members) return fail(ctx, GEMEL_EINVAL, tag + "needs members");
        for (int j = 0; j < gr.n_members; ++j) {
            const gemel_member &mb = gr.members[j];
            if (mb.model_id < 0 || mb.model_id >= (int)ctx->models.size())
                return fail(ctx, GEMEL_EINVAL, tag + "unknown model id " + std::to_string(mb.model_id));
            const Model &m = *ctx->models[(size_t)mb.model_id];
            if (mb.layer < 0 || mb.layer >= (int)m.layers.size())
                return fail(ctx, GEMEL_EINVAL, tag + "layer index out of range");
            if (!seen.insert({mb.model_id, mb.layer}).second)
                return fail(ctx, GEMEL_EINVAL, tag + "a layer appears in two groups or twice");
        }
        const Layer &s = ctx->models[(size_t)gr.members[0].model_id]->layers[(size_t)gr.members[0].layer];
        for (int j = 1; j < gr.n_members; ++j) {
            const gemel_member &mb = gr.members[j];
            const Layer &l = ctx->models[(size_t)mb.model_id]->layers[(size_t)mb.layer];
            // Section 4.1: same layer type and same type-specific properties
            const bool same = l.op == s.op && l.cin == s.cin && l.cout == s.cout && l.kh == s.kh &&
                              l.kw == s.kw && l.stride == s.stride && l.pad == s.pad &&
                              l.has_bias == s.has_bias && l.has_bn == s.has_bn;
            if (!same)
                return fail(ctx, GEMEL_ENOTMERGEABLE,
                            tag + "member " + std::to_string(j) + " is not architecturally identical to member 0");
            // an FC's stored column order follows its producer's C x H x W
            if (l.op == GEMEL_OP_FC && (l.in_c != s.in_c || l.in_h != s.in_h || l.in_w != s.in_w))
                return fail(ctx, GEMEL_ENOTMERGEABLE, tag + "fc producers differ in C x H x W");
            if (l.op == GEMEL_OP_CONCAT && l.src1_cp != s.src1_cp)
                return fail(ctx, GEMEL_ENOTMERGEABLE, tag + "concat inputs differ");
        }
    }
    // commit: every member uses the source's parameter copy
    for (auto &m : ctx->models)
        for (auto &l : m->layers) {
            l.eff = l.own;
            l.group = -1;
        }
    ctx->groups.clear();
    for (int g = 0; g < n_groups; ++g) {
        const gemel_group &gr = groups[g];
        std::vector<gemel_member> mem(gr.members, gr.members + gr.n_members);
        Layer &s = ctx->models[(size_t)mem[0].model_id]->layers[(size_t)mem[0].layer];
        for (auto &mb : mem) {
            Layer &l = ctx->models[(size_t)mb.model_id]->layers[(size_t)mb.layer];
            l.eff = s.own;
            l.group = (int)ctx->groups.size();
        }
        ctx->groups.push_back(std::move(mem));
    }
    ctx->weights_ready = false;
    drop_plans(ctx);
    return GEMEL_OK;
}

gemel_status gemel_enumerate_groups(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                                    gemel_group *groups, int32_t groups_cap, gemel_member *members,
                                    int32_t members_cap, int64_t *group_bytes, int32_t *n_groups,
                                    int32_t *n_members) {
    if (!ctx) return GEMEL_EINVAL;
    if (!n_groups || !n_members) return fail(ctx, GEMEL_EINVAL, "null count pointer");
    *n_groups = 0;
    *n_members = 0;
    if (n_models <= 0 || !model_ids) return fail(ctx, GEMEL_EINVAL, "no models");
    std::set<int> ids;
    for (int i = 0; i < n_models; ++i) {
        if (model_ids[i] < 0 || model_ids[i] >= (int)ctx->models.size())
            return fail(ctx, GEMEL_EINVAL, "unknown model id " + std::to_string(model_ids[i]));
        if (!ids.insert(model_ids[i]).second) return fail(ctx, GEMEL_EINVAL, "a model id appears twice");
    }
    try {
        // one candidate per architectural identity (the properties gemel_merge
        // compares), its appearances in model-position then layer order
        struct Cand {
            std::vector<gemel_member> mem;
            int64_t bytes = 0;
            int first_pos = 0, first_layer = 0;
        };
        const int64_t elem = ctx->dtype == GEMEL_BF16 ? 2 : 4;
        std::map<std::vector<int64_t>, size_t> index;
        std::vector<Cand> cands;
        for (int p = 0; p < n_models; ++p) {
            const Model &m = *ctx->models[(size_t)model_ids[p]];
            for (int l = 0; l < (int)m.layers.size(); ++l) {
                const Layer &L = m.layers[(size_t)l];
                if (L.op != GEMEL_OP_CONV && L.op != GEMEL_OP_FC) continue;
                const bool fc = L.op == GEMEL_OP_FC;
                const std::vector<int64_t> key = {L.op,      L.cin,      L.cout,         L.kh,
                                                  L.kw,      L.stride,   L.pad,          L.has_bias,
                                                  L.has_bn,  fc ? L.in_c : 0, fc ? L.in_h : 0, fc ? L.in_w : 0};
                const int64_t params = (int64_t)L.cout * L.cin * (fc ? 1 : (int64_t)L.kh * L.kw) +
                                       (L.has_bias ? L.cout : 0) + (L.has_bn ? 4 * (int64_t)L.cout : 0);
                auto it = index.find(key);
                if (it == index.end()) {
                    it = index.emplace(key, cands.size()).first;
                    cands.push_back(Cand{{}, 0, p, l});
                }
                Cand &c = cands[it->second];
                c.mem.push_back(gemel_member{model_ids[p], l});
                c.bytes += params * elem;
            }
        }
        std::vector<size_t> order;
        int64_t total = 0;
        for (size_t i = 0; i < cands.size(); ++i)
            if (cands[i].mem.size() >= 2) {
                order.push_back(i);
                total += (int64_t)cands[i].mem.size();
            }
        // most memory first; ties in order of first appearance
        std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) {
            const Cand &x = cands[a], &y = cands[b];
            if (x.bytes != y.bytes) return x.bytes > y.bytes;
            if (x.first_pos != y.first_pos) return x.first_pos < y.first_pos;
            return x.first_layer < y.first_layer;
        });
        if (total > INT32_MAX) return fail(ctx, GEMEL_EINVAL, "too many appearances");
        *n_groups = (int32_t)order.size();
        *n_members = (int32_t)total;
        if (!groups && !members) return GEMEL_OK;
        if (!groups || !members || groups_cap < *n_groups || members_cap < *n_members)
            return fail(ctx, GEMEL_EINVAL, "group or member array smaller than the counts");
        int32_t at = 0;
        for (size_t g = 0; g < order.size(); ++g) {
            const Cand &c = cands[order[g]];
            groups[g].n_members = (int32_t)c.mem.size();
            groups[g].members = members + at;
            for (const gemel_member &mb : c.mem) members[at++] = mb;
            if (group_bytes) group_bytes[g] = c.bytes;
        }
        return GEMEL_OK;
    } catch (const std::bad_alloc &) {
        return fail(ctx, GEMEL_ENOMEM, "out of host memory");
    }
}

// Argument checks shared by gemel_infer and gemel_infer_noalloc.
static gemel_status check_infer_args(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                                     const void *const *frames, const int32_t *n_frames, void *const *outputs) {
    if (n_models <= 0 || !model_ids || !frames || !n_frames || !outputs)
        return fail(ctx, GEMEL_EINVAL, "null argument array or no models");
    if (n_models > (int)ctx->models.size()) return fail(ctx, GEMEL_EINVAL, "more models than registered");
    std::set<int> ids;
    int out_slot = 0;
    for (int i = 0; i < n_models; ++i) {
        if (model_ids[i] < 0 || model_ids[i] >= (int)ctx->models.size())
            return fail(ctx, GEMEL_EINVAL, "unknown model id " + std::to_string(model_ids[i]));
        if (!ids.insert(model_ids[i]).second) return fail(ctx, GEMEL_EINVAL, "model id listed twice");
        if (n_frames[i] < 0) return fail(ctx, GEMEL_EINVAL, "negative frame count");
        const Model &m = *ctx->models[(size_t)model_ids[i]];
        if (n_frames[i] > 0) {
            if (!frames[i]) return fail(ctx, GEMEL_EINVAL, "null frames pointer");
            if ((int64_t)n_frames[i] * m.in_h * m.in_w * m.in_cp > (int64_t)1 << 31)
                return fail(ctx, GEMEL_ESHAPE, "too many frames for one call");
            for (size_t o = 0; o < m.outputs.size(); ++o)
                if (!outputs[out_slot + o]) return fail(ctx, GEMEL_EINVAL, "null output pointer");
        }
        out_slot += (int)m.outputs.size();
    }
    return GEMEL_OK;
}

gemel_status gemel_infer(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                         const void *const *frames, const int32_t *n_frames, void *const *outputs,
                         void *hip_stream) {
    if (!ctx) return GEMEL_EINVAL;
    const gemel_status st = check_infer_args(ctx, model_ids, n_models, frames, n_frames, outputs);
    if (st) return st;
    try {
        return run(ctx, model_ids, n_models, frames, n_frames, outputs, (hipStream_t)hip_stream);
    } catch (const std::bad_alloc &) {
        return fail(ctx, GEMEL_ENOMEM, "out of host memory");
    }
}

gemel_status gemel_infer_noalloc(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models,
                                 const void *const *frames, const int32_t *n_frames, void *const *outputs,
                                 void *hip_stream) {
    if (!ctx) return GEMEL_EINVAL;
    const gemel_status st = check_infer_args(ctx, model_ids, n_models, frames, n_frames, outputs);
    if (st) return st;
    try {
        return run_noalloc(ctx, model_ids, n_models, frames, n_frames, outputs, (hipStream_t)hip_stream);
    } catch (const std::bad_alloc &) {
        return fail(ctx, GEMEL_ENOMEM, "out of host memory");
    }
}

gemel_status gemel_set_next_round(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models) {
    if (!ctx) return GEMEL_EINVAL;
    if (n_models < 0 || (n_models > 0 && !model_ids)) return fail(ctx, GEMEL_EINVAL, "bad model list");
    std::vector<int> next;
    for (int i = 0; i < n_models; ++i) {
        if (model_ids[i] < 0 || model_ids[i] >= (int)ctx->models.size())
            return fail(ctx, GEMEL_EINVAL, "unknown model id " + std::to_string(model_ids[i]));
        next.push_back(model_ids[i]);
    }
    ctx->next_models = next;
    return GEMEL_OK;
}

// Bytes of the stored parameter copies two models both use.
static int64_t shared_param_bytes(const Model &a, const Model &b) {
    std::set<const Blob *> in_a;
    for (auto &l : a.layers)
        if (l.eff) in_a.insert(l.eff.get());
    std::set<const Blob *> seen;
    int64_t s = 0;
    for (auto &l : b.layers)
        if (l.eff && in_a.count(l.eff.get()) && seen.insert(l.eff.get()).second)
            s += round_up((int64_t)l.eff->w_bytes(), 256);
    return s;
}

gemel_status gemel_load_order(gemel_ctx *ctx, const int32_t *model_ids, int32_t n_models, int32_t *order) {
    if (!ctx) return GEMEL_EINVAL;
    if (n_models <= 0 || !model_ids || !order) return fail(ctx, GEMEL_EINVAL, "null argument or no models");
    std::set<int> ids;
    for (int i = 0; i < n_models; ++i) {
        if (model_ids[i] < 0 || model_ids[i] >= (int)ctx->models.size())
            return fail(ctx, GEMEL_EINVAL, "unknown model id " + std::to_string(model_ids[i]));
        if (!ids.insert(model_ids[i]).second) return fail(ctx, GEMEL_EINVAL, "model id listed twice");
    }
    std::map<int, int64_t> total;
    for (int id : ids) {
        std::set<const Blob *> seen;
        int64_t t = 0;
        for (auto &l : ctx->models[(size_t)id]->layers)
            if (l.eff && seen.insert(l.eff.get()).second) t += round_up((int64_t)l.eff->w_bytes(), 256);
        total[id] = t;
    }
    std::vector<int> left(ids.begin(), ids.end()), seq;
    // the model of the most bytes first (lower id on ties)
    int first = left[0];
    for (int m : left)
        if (total[m] > total[first]) first = m;
    seq.push_back(first);
    left.erase(std::find(left.begin(), left.end(), first));
    while (!left.empty()) {
        // the remaining model that shares the most bytes with either end,
        // placed at that end (ties: more bytes, lower id, the back end)
        std::tuple<int64_t, int64_t, int, int> best{-1, -1, 0, 0};
        bool have = false;
        for (int m : left)
            for (int end : {0, 1}) {
                const int e = end == 0 ? seq.back() : seq.front();
                const auto key = std::make_tuple(
                    shared_param_bytes(*ctx->models[(size_t)e], *ctx->models[(size_t)m]), total[m], -m, -end);
                if (!have || key > best) {
                    best = key;
                    have = true;
                }
            }
        const int m = -std::get<2>(best);
        if (std::get<3>(best) == 0)
            seq.push_back(m);
        else
            seq.insert(seq.begin(), m);
        left.erase(std::find(left.begin(), left.end(), m));
    }
    for (int i = 0; i < n_models; ++i) order[i] = seq[(size_t)i];
    return GEMEL_OK;
}

gemel_status gemel_model_outputs(gemel_ctx *ctx, int32_t model_id, int32_t *n_outputs) {
    if (!ctx) return GEMEL_EINVAL;
    if (!n_outputs || model_id < 0 || model_id >= (int)ctx->models.size())
        return fail(ctx, GEMEL_EINVAL, "bad model id or null pointer");
    *n_outputs = (int32_t)ctx->models[(size_t)model_id]->outputs.size();
    return GEMEL_OK;
}

gemel_status gemel_output_shape(gemel_ctx *ctx, int32_t model_id, int32_t output_idx, int32_t n_frames,
                                int64_t dims[4]) {
    if (!ctx) return GEMEL_EINVAL;
    if (!dims || model_id < 0 || model_id >= (int)ctx->models.size() || n_frames < 0)
        return fail(ctx, GEMEL_EINVAL, "bad model id, frame count or null dims");
    const Model &m = *ctx->models[(size_t)model_id];
    if (output_idx < 0 || output_idx >= (int)m.outputs.size()) return fail(ctx, GEMEL_EINVAL, "bad output index");
    const Layer &l = m.layers[(size_t)m.outputs[(size_t)output_idx]];
    dims[0] = n_frames;
    dims[1] = l.out_c;
    dims[2] = l.out_h;
    dims[3] = l.out_w;
    return GEMEL_OK;
}

gemel_status gemel_query(gemel_ctx *ctx, int32_t key, int64_t *val) {
    if (!ctx) return GEMEL_EINVAL;
    if (!val) return fail(ctx, GEMEL_EINVAL, "null val");
    switch (key) {
    case GEMEL_Q_UNMERGED_BYTES: *val = (int64_t)unmerged_bytes(ctx); break;
    case GEMEL_Q_MERGED_BYTES: *val = (int64_t)merged_bytes(ctx); break;
    case GEMEL_Q_RESIDENT_BYTES: *val = (int64_t)ctx->resident_bytes; break;
    case GEMEL_Q_PEAK_BYTES: *val = (int64_t)ctx->peak_bytes; break;
    case GEMEL_Q_STREAMED_BYTES: *val = ctx->last_plan ? (int64_t)ctx->last_plan->streamed_bytes : 0; break;
    case GEMEL_Q_ACTIVATION_BYTES: *val = ctx->last_plan ? (int64_t)ctx->last_plan->arena_bytes : 0; break;
    case GEMEL_Q_LAUNCHES: *val = ctx->last_plan ? (int64_t)ctx->last_plan->launches.size() : 0; break;
    case GEMEL_Q_N_MODELS: *val = (int64_t)ctx->models.size(); break;
    case GEMEL_Q_GRAPH_REPLAYS: *val = ctx->graph_replays; break;
    case GEMEL_Q_STREAMS: *val = ctx->opt.streams; break;
    case GEMEL_Q_ROUND_MODE: *val = ctx->last_mode; break;
    case GEMEL_Q_ROUND_TUNING: *val = ctx->tuning_left; break;
    case GEMEL_Q_ROUND_LOADED_BYTES: *val = ctx->round_loaded; break;
    case GEMEL_Q_ROUND_EVICTED_BYTES: *val = ctx->round_evicted; break;
    case GEMEL_Q_CACHED_BYTES: {
        int64_t c = 0;
        for (auto &b : ctx->placed)
            if (b->cache_off >= 0) c += round_up((int64_t)b->w_bytes(), 256);
        *val = c;
        break;
    }
    case GEMEL_Q_CACHE_CAPACITY: *val = (int64_t)ctx->cache_cap; break;
    case GEMEL_Q_PREFETCHES: {
        int64_t n = 0;
        if (ctx->last_plan)
            for (const Launch &L : ctx->last_plan->launches) n += L.type == L_CONV_BF16 && L.conv.pf ? 1 : 0;
        *val = n;
        break;
    }
    default: return fail(ctx, GEMEL_EINVAL, "unknown query key");
    }
    return GEMEL_OK;
}

gemel_status gemel_set_option(gemel_ctx *ctx, int32_t key, int64_t value) {
    if (!ctx) return GEMEL_EINVAL;
    switch (key) {
    case GEMEL_OPT_USE_GRAPH:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "use_graph is 0 or 1");
        ctx->opt.use_graph = (int)value;
        break;
    case GEMEL_OPT_SWAP_SLOT_BYTES:
        if (value < (1 << 16) || value > (1ll << 34)) return fail(ctx, GEMEL_EINVAL, "slot size out of range");
        ctx->opt.slot_bytes = round_up(value, 256);
        ctx->weights_ready = false;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_SWAP_SLOTS:
        if (value < 2 || value > 64) return fail(ctx, GEMEL_EINVAL, "slots must be 2..64");
        ctx->opt.slots = (int)value;
        ctx->weights_ready = false;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_FAIL_COPY_AT:
        if (value < 0) return fail(ctx, GEMEL_EINVAL, "fail_copy_at must be >= 0");
        ctx->opt.fail_copy_at = value ? ctx->copies_issued + value : 0;
        break;
    case GEMEL_OPT_SWAP_CACHE:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "swap_cache is 0 or 1");
        if (ctx->opt.swap_cache != (int)value) {
            ctx->opt.swap_cache = (int)value;
            ctx->weights_ready = false;
            drop_plans(ctx);
        }
        break;
    case GEMEL_OPT_GROUP_UNMERGED:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "group_unmerged is 0 or 1");
        ctx->opt.group_unmerged = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_FAIL_ALLOC_AT:
        if (value < 0) return fail(ctx, GEMEL_EINVAL, "fail_alloc_at must be >= 0");
        ctx->opt.fail_alloc_at = value ? ctx->allocs_issued + value : 0;
        break;
    case GEMEL_OPT_SPLIT_MERGED:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "split_merged is 0 or 1");
        ctx->opt.split_merged = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_CONV_TILE:
        if (value < -1 || value >= TILE_COUNT)
            return fail(ctx, GEMEL_EINVAL, "conv tile is -1.." + std::to_string(TILE_COUNT - 1));
        ctx->opt.conv_tile = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_CONV_SPLITS:
        if (value < 0 || value > 64) return fail(ctx, GEMEL_EINVAL, "conv splits is 0..64");
        ctx->opt.conv_splits = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_STREAMS:
        if (value < 1 || value > 8) return fail(ctx, GEMEL_EINVAL, "streams is 1..8");
        ctx->opt.streams = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_AUTOTUNE:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "autotune is 0 or 1");
        ctx->opt.autotune = (int)value;
        break;
    case GEMEL_OPT_TUNE:
        if (value < 0 || value > 16) return fail(ctx, GEMEL_EINVAL, "tune is 0..16");
        ctx->opt.tune = value > 0;
        if (value > 1) ctx->opt.tune_candidates = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_MIXED_SIZES:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "mixed_sizes is 0 or 1");
        ctx->opt.mixed_sizes = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_FUSE_POOL:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "fuse_pool is 0 or 1");
        ctx->opt.fuse_pool = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_PAIRED_ACTS:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "paired_acts is 0 or 1");
        if (ctx->opt.paired_acts != (int)value) {
            ctx->opt.paired_acts = (int)value;
            ctx->weights_ready = false;
            drop_plans(ctx);
        }
        break;
    case GEMEL_OPT_PREFETCH:
        if (value < 0 || value > 2) return fail(ctx, GEMEL_EINVAL, "prefetch is 0, 1 or 2");
        ctx->opt.prefetch = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_SPLITK_FUSED:
        if (value < 0 || value > 2) return fail(ctx, GEMEL_EINVAL, "splitk_fused is 0, 1 or 2");
        ctx->opt.splitk_fused = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_FORK_US:
        if (value < 0 || value > 1000000) return fail(ctx, GEMEL_EINVAL, "fork_us is 0..1e6");
        ctx->opt.fork_us = (int)value;
        drop_plans(ctx);
        break;
    case GEMEL_OPT_GRAPH_DAG:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "graph_dag is 0 or 1");
        ctx->opt.graph_dag = (int)value;
        break;
    case GEMEL_OPT_PROFILE:
        if (value != 0 && value != 1) return fail(ctx, GEMEL_EINVAL, "profile is 0 or 1");
        profile_reset(ctx);
        ctx->opt.profile = (int)value;
        if (value) ctx->prof.used = true;
        break;
    case GEMEL_OPT_WEIGHT_BUDGET:
        if (value < 0) return fail(ctx, GEMEL_EINVAL, "budget must be >= 0");
        ctx->budget = (uint64_t)value;
        ctx->weights_ready = false;
        drop_plans(ctx);
        break;
    default: return fail(ctx, GEMEL_EINVAL, "unknown option");
    }
    return GEMEL_OK;
}

gemel_status gemel_profile(gemel_ctx *ctx, gemel_kernel_stat *stats, int32_t *rounds) {
    if (!ctx) return GEMEL_EINVAL;
    if (!stats || !rounds) return fail(ctx, GEMEL_EINVAL, "null stats or rounds");
    if (!ctx->prof.used) return fail(ctx, GEMEL_ESTATE, "profiling was never enabled");
    return profile_read(ctx, stats, rounds);
}

const char *gemel_last_error(const gemel_ctx *ctx) {
    return ctx ? ctx->err.c_str() : g_create_err.c_str();
}

gemel_status gemel_destroy(gemel_ctx *ctx) {
    if (!ctx) return GEMEL_OK;
    gemel_status st = GEMEL_OK;
    profile_reset(ctx);
    if (ctx->dev_ready) {
        int prev = 0;
        (void)hipGetDevice(&prev);
        if (hipSetDevice(ctx->device) != hipSuccess || hipDeviceSynchronize() != hipSuccess) st = GEMEL_EDEVICE;
        release_device(ctx);
        (void)hipSetDevice(prev);
    }
    delete ctx;
    return st;
}

}  // extern "C"
