// CPU stand-in for the HIP runtime and for libgemel's kernel launchers.
//
// Compiled together with the library's host sources (registry.cpp,
// plan.cpp) into a CPU-only shared library, it lets the tests drive the
// real planner and round executor without a GPU: device allocations are
// host allocations recorded in a registry, and every "kernel launch"
// checks that each pointer range the kernel would read or write lies
// inside one live allocation (and that the argument block is
// self-consistent). Any violation is printed and counted.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <string>

#include "hip/hip_runtime.h"
#include "kargs.h"
#include "kernels.h"

namespace {
std::mutex mu;
std::map<uintptr_t, size_t> live;     // base -> bytes
long violations = 0, launches = 0;
std::set<void *> events_recorded;
std::string last;

bool inside(const void *p, size_t bytes) {
    const uintptr_t a = (uintptr_t)p;
    auto it = live.upper_bound(a);
    if (it == live.begin()) return false;
    --it;
    return a >= it->first && a + bytes <= it->first + it->second;
}

bool chk(const void *p, long long bytes, const char *what, const char *kern) {
    if (bytes <= 0) return true;
    if (!p || !inside(p, (size_t)bytes)) {
        char buf[256];
        std::snprintf(buf, sizeof buf, "%s: %s [%p, +%lld) outside any live allocation", kern, what, p, bytes);
        last = buf;
        std::fprintf(stderr, "hoststub violation: %s\n", buf);
        ++violations;
        return false;
    }
    return true;
}

hipError_t verdict(bool ok) { return ok ? hipSuccess : hipErrorInvalidValue; }
}  // namespace

extern "C" {
long hoststub_violations() { return violations; }
long hoststub_launches() { return launches; }
const char *hoststub_last() { return last.c_str(); }
long hoststub_live_bytes() {
    size_t b = 0;
    for (auto &kv : live) b += kv.second;
    return (long)b;
}

hipError_t hipGetDevice(int *d) { *d = 0; return hipSuccess; }
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipGetDeviceCount(int *n) { *n = 1; return hipSuccess; }
hipError_t hipGetDeviceProperties(hipDeviceProp_t *p, int) {
    std::strcpy(p->gcnArchName, "gfx950:sramecc+:xnack-");
    return hipSuccess;
}
hipError_t hipStreamCreateWithFlags(hipStream_t *s, unsigned) { *s = (hipStream_t)std::malloc(16); return hipSuccess; }
hipError_t hipStreamDestroy(hipStream_t s) { std::free(s); return hipSuccess; }
hipError_t hipEventCreate(hipEvent_t *e) { *e = (hipEvent_t)std::malloc(16); return hipSuccess; }
hipError_t hipEventCreateWithFlags(hipEvent_t *e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) { events_recorded.erase(e); std::free(e); return hipSuccess; }
hipError_t hipEventRecord(hipEvent_t e, hipStream_t) { events_recorded.insert(e); return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipEventElapsedTime(float *ms, hipEvent_t, hipEvent_t) { *ms = 0.001f; return hipSuccess; }
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned) { return (s && e) ? hipSuccess : hipErrorInvalidValue; }
hipError_t hipMalloc(void **p, size_t n) {
    *p = std::malloc(n ? n : 1);
    if (!*p) return hipErrorOutOfMemory;
    std::lock_guard<std::mutex> g(mu);
    live[(uintptr_t)*p] = n;
    return hipSuccess;
}
hipError_t hipFree(void *p) {
    if (!p) return hipSuccess;
    std::lock_guard<std::mutex> g(mu);
    auto it = live.find((uintptr_t)p);
    if (it == live.end()) {
        ++violations;
        last = "hipFree of an unknown pointer";
        return hipErrorInvalidValue;
    }
    live.erase(it);
    std::free(p);
    return hipSuccess;
}
hipError_t hipHostMalloc(void **p, size_t n, unsigned) { return hipMalloc(p, n); }
hipError_t hipHostFree(void *p) { return hipFree(p); }
hipError_t hipMemcpy(void *d, const void *s, size_t n, hipMemcpyKind) {
    bool ok = chk(d, (long long)n, "memcpy dst", "hipMemcpy");
    if (ok) std::memcpy(d, s, n);
    return verdict(ok);
}
hipError_t hipMemcpyAsync(void *d, const void *s, size_t n, hipMemcpyKind k, hipStream_t) {
    bool ok = chk(d, (long long)n, "copy dst", "hipMemcpyAsync") & chk(s, (long long)n, "copy src", "hipMemcpyAsync");
    if (ok) std::memcpy(d, s, n);
    (void)k;
    return verdict(ok);
}
hipError_t hipDeviceSynchronize() { return hipSuccess; }
hipError_t hipGetLastError() { return hipSuccess; }
const char *hipGetErrorString(hipError_t e) { return e == hipSuccess ? "success" : "stub error"; }
hipError_t hipStreamBeginCapture(hipStream_t, hipStreamCaptureMode) { return hipSuccess; }
hipError_t hipStreamEndCapture(hipStream_t, hipGraph_t *g) { *g = (hipGraph_t)std::malloc(16); return hipSuccess; }
hipError_t hipGraphInstantiate(hipGraphExec_t *e, hipGraph_t, hipGraphNode_t *, char *, size_t) {
    *e = (hipGraphExec_t)std::malloc(16);
    return hipSuccess;
}
hipError_t hipGraphDestroy(hipGraph_t g) { std::free(g); return hipSuccess; }
hipError_t hipGraphExecDestroy(hipGraphExec_t e) { std::free(e); return hipSuccess; }
hipError_t hipGraphLaunch(hipGraphExec_t, hipStream_t) { return hipSuccess; }
}  // extern "C"

namespace gemel {

static const int kBm[TILE_COUNT] = {128, 128, 64, 256, 256, 256, 64, 128, 64, 256, 256, 128, 128};
static const int kBn[TILE_COUNT] = {128, 64, 64, 256, 128, 64, 64, 64, 128, 256, 128, 128, 64};
int conv_tile_bm(int t) { return t >= 0 && t < TILE_COUNT ? kBm[t] : 0; }
int conv_tile_bn(int t) { return t >= 0 && t < TILE_COUNT ? kBn[t] : 0; }
int conv_tile_threads(int t) { return (t == TILE_256x256 || t == TILE_256x128) ? 512 : 256; }

template <typename Seg>
static long long seg_rows(const Seg *seg, int nseg, int i, int M) {
    return (long long)((i + 1 < nseg ? seg[i + 1].m_start : M) - seg[i].m_start);
}

static hipError_t conv_common(const ConvArgs &a, int esz, const char *kern, bool need_zero) {
    ++launches;
    bool ok = a.M > 0 && a.N > 0 && a.N % 8 == 0 && a.K == a.kh * a.kw * a.Cin && a.Cin % 8 == 0 &&
              a.nseg >= 1 && a.nseg <= GEMEL_MAX_SEG && a.seg[0].m_start == 0 && a.out_cs >= a.N;
    if (!ok) {
        ++violations;
        last = std::string(kern) + ": inconsistent argument block";
        return hipErrorInvalidValue;
    }
    const long long hwo = (long long)a.Ho * a.Wo;
    ok &= chk(a.w, (long long)a.N * a.K * esz, "weights", kern);
    if (need_zero) ok &= chk(a.zero, 16, "zero page", kern);
    for (int i = 0; i < a.nseg; ++i) {
        const ConvSeg &s = a.seg[i];
        const long long rows = seg_rows(a.seg, a.nseg, i, a.M);
        if (rows <= 0 || rows % hwo || s.m_start != (long long)s.f_start * hwo) {
            ++violations;
            last = std::string(kern) + ": segment rows do not match frames";
            return hipErrorInvalidValue;
        }
        const long long frames = rows / hwo;
        ok &= chk(s.in, frames * a.H * a.W * a.in_cs * esz, "input", kern);
        ok &= chk(s.scale, (long long)a.N * 4, "scale", kern) & chk(s.shift, (long long)a.N * 4, "shift", kern);
        if (a.has_res) ok &= chk(s.res, ((rows - 1) * a.out_cs + a.N) * esz, "residual", kern);
        if (a.k_splits <= 1) {
            if (a.out_mode == OUT_NHWC)
                ok &= chk(s.out, ((rows - 1) * a.out_cs + a.N) * esz, "output", kern);
            else
                ok &= chk(s.out, frames * a.cout * hwo * 4, "output nchw", kern);
        }
    }
    if (a.k_splits > 1) ok &= chk(a.partial, (long long)a.k_splits * a.M * a.N * 4, "partial", kern);
    return verdict(ok);
}

bool conv_dma_supported(const ConvArgs &a) {
    return a.Cin % 32 == 0 && a.in_cs % 8 == 0 && a.K % 32 == 0 && a.k_per_split % 32 == 0 && a.zero &&
           a.uni_affine;
}
hipError_t launch_conv_dma(const ConvArgs &a, int tile, hipStream_t s) { return launch_conv_bf16(a, tile, s); }
hipError_t launch_conv_bf16(const ConvArgs &a, int tile, hipStream_t) {
    if (tile < 0 || tile >= TILE_COUNT) return hipErrorInvalidValue;
    if (tile_is_dma(tile) && !conv_dma_supported(a)) {
        ++violations;
        last = "dma tile on an unsupported conv";
        return hipErrorInvalidValue;
    }
    return conv_common(a, 2, "conv_bf16", true);
}
hipError_t launch_conv_f32(const ConvArgs &a, hipStream_t) { return conv_common(a, 4, "conv_f32", false); }

hipError_t launch_conv_reduce(const ReduceArgs &a, bool bf16, hipStream_t) {
    ++launches;
    const int esz = bf16 ? 2 : 4;
    bool ok = chk(a.partial, (long long)a.splits * a.M * a.N * 4, "partial", "conv_reduce");
    for (int i = 0; i < a.nseg; ++i) {
        const ConvSeg &s = a.seg[i];
        const long long rows = seg_rows(a.seg, a.nseg, i, a.M);
        if (a.out_mode == OUT_NHWC)
            ok &= chk(s.out, ((rows - 1) * a.out_cs + a.N) * esz, "output", "conv_reduce");
        else
            ok &= chk(s.out, rows * a.cout * 4, "output nchw", "conv_reduce");
        if (a.has_res) ok &= chk(s.res, ((rows - 1) * a.out_cs + a.N) * esz, "residual", "conv_reduce");
        ok &= chk(s.scale, (long long)a.N * 4, "scale", "conv_reduce");
    }
    return verdict(ok);
}

static hipError_t fc_common(const FcArgs &a, int esz, const char *kern, bool reads_w) {
    ++launches;
    bool ok = a.M > 0 && a.N > 0 && a.N % 8 == 0 && a.K % 8 == 0 && a.nseg >= 1 && a.seg[0].f_start == 0;
    if (!ok) {
        ++violations;
        last = std::string(kern) + ": inconsistent argument block";
        return hipErrorInvalidValue;
    }
    if (reads_w) ok &= chk(a.w, (long long)a.N * a.K * esz, "weights", kern);
    for (int i = 0; i < a.nseg; ++i) {
        const FcSeg &s = a.seg[i];
        const long long frames = (i + 1 < a.nseg ? a.seg[i + 1].f_start : a.M) - s.f_start;
        if (reads_w) ok &= chk(s.in, frames * a.K * esz, "input", kern);
        if (a.out_mode == OUT_NHWC)
            ok &= chk(s.out, ((frames - 1) * a.out_cs + a.N) * esz, "output", kern);
        else
            ok &= chk(s.out, frames * a.cout * 4, "output final", kern);
        ok &= chk(s.scale, (long long)a.N * 4, "scale", kern);
    }
    if (a.k_splits > 1) ok &= chk(a.partial, (long long)a.k_splits * a.M * a.N * 4, "partial", kern);
    return verdict(ok);
}
hipError_t launch_fc_bf16(const FcArgs &a, hipStream_t) { return fc_common(a, 2, "fc_bf16", true); }
hipError_t launch_fc_f32(const FcArgs &a, hipStream_t) { return fc_common(a, 4, "fc_f32", true); }
hipError_t launch_fc_reduce(const FcArgs &a, bool bf16, hipStream_t) {
    return fc_common(a, bf16 ? 2 : 4, "fc_reduce", false);
}

static hipError_t ew(const EwArgs &a, const char *kern, long long in0, long long in1, long long out,
                     int in_esz, int out_esz) {
    ++launches;
    bool ok = a.nseg >= 1 && a.nseg <= GEMEL_MAX_SEG;
    for (int i = 0; ok && i < a.nseg; ++i) {
        const long long f = a.seg[i].frames;
        ok &= chk(a.seg[i].in0, f * in0 * in_esz, "in0", kern);
        if (in1) ok &= chk(a.seg[i].in1, f * in1 * in_esz, "in1", kern);
        ok &= chk(a.seg[i].out, f * out * out_esz, "out", kern);
    }
    return verdict(ok);
}
hipError_t launch_pack(const EwArgs &a, bool bf16, hipStream_t) {
    return ew(a, "pack", (long long)a.c_logical * a.H * a.W, 0, (long long)a.H * a.W * a.Co, 4, bf16 ? 2 : 4);
}
hipError_t launch_maxpool(const EwArgs &a, bool bf16, hipStream_t) {
    const int e = bf16 ? 2 : 4;
    return ew(a, "maxpool", (long long)a.H * a.W * a.C, 0, (long long)a.Ho * a.Wo * a.C, e, e);
}
hipError_t launch_avgpool(const EwArgs &a, bool bf16, hipStream_t) {
    const int e = bf16 ? 2 : 4;
    return ew(a, "avgpool", (long long)a.H * a.W * a.C, 0, a.C, e, e);
}
hipError_t launch_upsample2x(const EwArgs &a, bool bf16, hipStream_t) {
    const int e = bf16 ? 2 : 4;
    return ew(a, "upsample", (long long)a.H * a.W * a.C, 0, (long long)a.Ho * a.Wo * a.C, e, e);
}
hipError_t launch_concat(const EwArgs &a, bool bf16, hipStream_t) {
    const int e = bf16 ? 2 : 4;
    return ew(a, "concat", (long long)a.H * a.W * a.C, (long long)a.H * a.W * a.C1, (long long)a.H * a.W * a.Co, e, e);
}
hipError_t launch_export(const EwArgs &a, bool bf16, hipStream_t) {
    ++launches;
    bool ok = true;
    for (int i = 0; i < a.nseg; ++i) {
        const long long f = a.seg[i].frames;
        ok &= chk(a.seg[i].in0, f * a.H * a.W * a.C * (bf16 ? 2 : 4), "in0", "export");
        ok &= chk(a.seg[i].out, f * a.c_logical * a.H * a.W * 4, "out", "export");
    }
    return verdict(ok);
}

}  // namespace gemel
