// api.hip -- host side of libconvcrf: the C ABI of include/convcrf.h.
//
// Validation happens before any HIP call.  The context owns a workspace
// that grows on demand: one [B][C][H][W] buffer for the ping-pong of Q
// (the other half of the ping-pong is the caller's q_out), the kernel matrix
// for the materialised variant, pooled buffers for the blur path, and a
// small device block holding the compatibility matrix.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <mutex>
#include <string>
#include <vector>

#include "convcrf.h"
#include "crf_internal.h"

using namespace convcrf;

// Scratch memory of the allocation-free entry point (see scratch_address):
// 64 MiB per device, zero at load, held until the process ends.
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr double kLog2eD = 1.4426950408889634073599;
constexpr size_t kLdsLimit = 160 * 1024;  // gfx950 LDS per work-group
// Most class groups the adjoint message splits its classes into (at least 4
// classes per group).
constexpr int kBwdClassGroups = 3;
constexpr int kBwdMinGroups = 8;     // adjoint-message work-groups per CU sought on small grids

const char* const kKernelNames[] = {"fused_iter",   "softmax",      "build_kernel",
                                    "materialised_iter", "blur_pool", "blur_message",
                                    "blur_update",  "fused_resident", "sync_reset",
                                    "bwd_point", "bwd_message", "bwd_reduce", "feature_iter",
                                    "bwd_blur_transpose", "fused_first", "blur_iteration"};
enum KernelId {
    kFused = 0, kSoftmax, kBuild, kMatIter, kPool, kBlurMsg, kBlurUpd, kResident, kSyncReset,
    kBwdPoint, kBwdMsg, kBwdReduce, kFeatIter, kBwdBlurT, kFusedFirst, kBlurIter, kNumKernels
};

struct DevBuf {
    void* p = nullptr;
    size_t bytes = 0;
};

struct ProfRec {
    int kernel;
    hipEvent_t start, stop;
};

thread_local std::string g_last_error = "no error";

}  // namespace

struct convcrf_ctx {
    int device = 0;
    int num_cus = 256;
    bool coop = false;              // cooperative launches supported
    std::string err = "no error";
    DevBuf q_ws, q_ws2, kmat, pool_q, pool_m, pool_f, mu, sync;
    // reverse mode: Q^0..Q^T, dL/dQ ping-pong, dL/dM, -dL/dZ, per-tile sums,
    // dL/dF when not requested, the pooled derivatives (blur)
    DevBuf b_q, b_dq, b_dm, b_dp, b_gpart, b_kpart, b_df, b_pd, b_dfp;
    std::vector<float> mu_last;   // host copy of the uploaded compatibility
    float* mu_pinned = nullptr;   // pinned staging for the upload
    size_t mu_pinned_cap = 0;
    hipEvent_t mu_copied = nullptr;
    // the resident variant's bounded neighbour waits: sync.p[0] is a sticky
    // device flag that a wait past its bound sets; a copy of it is read back
    // without blocking (flag_event) and reported by the next call or by
    // convcrf_synchronize
    unsigned int* flag_host = nullptr;
    hipEvent_t flag_event = nullptr;
    bool flag_pending = false;
    void* scratch_ptr = nullptr;    // device address of this device's scratch array
    bool profiling = false;
    bool no_events = false;         // set during an allocation-free call
    std::vector<ProfRec> prof;
    std::vector<hipEvent_t> free_events;
};

namespace {

convcrf_status fail(convcrf_ctx* ctx, convcrf_status s, const std::string& msg) {
    if (ctx) ctx->err = msg;
    else g_last_error = msg;
    return s;
}

convcrf_status hip_fail(convcrf_ctx* ctx, hipError_t e, const char* what) {
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    return fail(ctx, CONVCRF_E_HIP, m);
}

bool finite_pos(float v) { return std::isfinite(v) && v > 0.f; }

convcrf_status validate(convcrf_ctx* ctx, int B, int C, int H, int W, const convcrf_params* p,
                        int iters) {
    if (!p) return fail(ctx, CONVCRF_E_INVALID_ARG, "params is NULL");
    if (B < 0 || H < 0 || W < 0) return fail(ctx, CONVCRF_E_INVALID_ARG, "negative B, H or W");
    if (C < 1) return fail(ctx, CONVCRF_E_INVALID_ARG, "C must be >= 1");
    if (iters < 0) return fail(ctx, CONVCRF_E_INVALID_ARG, "iters must be >= 0");
    const int k = p->filter_size;
    if (k < 1 || (k & 1) == 0) return fail(ctx, CONVCRF_E_INVALID_ARG, "filter_size must be odd and >= 1");
    if (k > kMaxK) return fail(ctx, CONVCRF_E_UNSUPPORTED, "filter_size > 15 is not built");
    if (C > kMaxC) return fail(ctx, CONVCRF_E_UNSUPPORTED, "more than 24 classes is not built");
    if (p->include_center != 0 && p->include_center != 1)
        return fail(ctx, CONVCRF_E_INVALID_ARG, "include_center must be 0 or 1");
    if (p->variant != CONVCRF_VARIANT_FUSED && p->variant != CONVCRF_VARIANT_MATERIALISED &&
        p->variant != CONVCRF_VARIANT_RESIDENT)
        return fail(ctx, CONVCRF_E_INVALID_ARG, "unknown variant");
    // w_smooth may take either sign (the smoothness term is added to the
    // weight); w_app is folded into an exponent as log2(w_app)
    if (!std::isfinite(p->w_app) || !std::isfinite(p->w_smooth))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "kernel weights must be finite");
    if (p->w_app < 0.f)
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "a negative appearance weight is not built");
    if (!finite_pos(p->theta_alpha) || !finite_pos(p->theta_beta) || !finite_pos(p->theta_gamma))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "theta parameters must be finite and > 0");
    const int s = p->blur;
    if (s != 1 && s != 2 && s != 4 && s != 8)
        return fail(ctx, CONVCRF_E_INVALID_ARG, "blur must be 1, 2, 4 or 8");
    if (s > 1 && p->variant == CONVCRF_VARIANT_MATERIALISED)
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "blur is not built for the materialised variant");
    if (s > 1 && (H % s != 0 || W % s != 0))
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "H and W must be multiples of the blur factor");
    if (s > 1 && (H / s > 65535 || B > 65535))
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "blur grid: H / blur and B must be at most 65535");
    if (p->features) {
        if (p->feature_dim < 1 || p->feature_dim > kMaxFeat)
            return fail(ctx, CONVCRF_E_INVALID_ARG, "feature_dim must be 1 .. 4 with features");
        // with blur the features are pooled and staged by the pooled message
        if (s == 1 ? feat_lds_bytes(k, C, p->feature_dim) > kLdsLimit
                   : pmsg_lds_bytes(k, p->feature_dim) > kLdsLimit)
            return fail(ctx, CONVCRF_E_UNSUPPORTED, "window, classes and features exceed LDS");
    }
    const long long npix = (long long)B * H * W;
    if (npix * (long long)C > (1LL << 40))
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "tensor too large");
    if ((long long)H * W > (1LL << 31) - 1)
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "image plane larger than 2^31 pixels");
    return CONVCRF_OK;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = static_cast<const char*>(a);
    const char* pb = static_cast<const char*>(b);
    return pa < pb + nb && pb < pa + na;
}

convcrf_status ensure(convcrf_ctx* ctx, DevBuf& buf, size_t bytes) {
    if (buf.bytes >= bytes) return CONVCRF_OK;
    if (buf.p) {
        hipError_t e = hipDeviceSynchronize();
        if (e != hipSuccess) return hip_fail(ctx, e, "hipDeviceSynchronize");
        (void)hipFree(buf.p);
        buf.p = nullptr;
        buf.bytes = 0;
    }
    hipError_t e = hipMalloc(&buf.p, bytes);
    if (e != hipSuccess) {
        buf.p = nullptr;
        (void)hipGetLastError();
        return fail(ctx, CONVCRF_E_OOM, std::string("workspace allocation failed: ") + hipGetErrorString(e));
    }
    buf.bytes = bytes;
    return CONVCRF_OK;
}

// Per-offset constants of Eq. 4, indexed by n = dx^2 + dy^2 on a grid whose
// step is `step` full-resolution pixels (1, or the blur factor on the pooled
// grid).
void fill_taps(const convcrf_params& p, int step, TapTable& t) {
    const double ta2 = 2.0 * (double)p.theta_alpha * p.theta_alpha;
    const double tg2 = 2.0 * (double)p.theta_gamma * p.theta_gamma;
    const double lw = p.w_app > 0 ? std::log2((double)p.w_app) : -INFINITY;
    for (int n = 0; n <= kMaxN; ++n) {
        const double d2 = (double)step * step * n;
        t.app_log2[n] = p.w_app > 0 ? (float)(lw - d2 * kLog2eD / ta2) : -INFINITY;
        t.smooth[n] = (float)(p.w_smooth * std::exp(-d2 / tg2));
    }
}

hipEvent_t take_event(convcrf_ctx* ctx) {
    if (!ctx->free_events.empty()) {
        hipEvent_t e = ctx->free_events.back();
        ctx->free_events.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Launch wrapper: records an event pair around the launch when profiling.
template <typename F>
convcrf_status launch(convcrf_ctx* ctx, int kernel, hipStream_t stream, const char* what, F&& fn) {
    ProfRec rec{kernel, nullptr, nullptr};
    const bool record = ctx->profiling && !ctx->no_events;
    if (record) {
        rec.start = take_event(ctx);
        rec.stop = take_event(ctx);
        if (rec.start) (void)hipEventRecord(rec.start, stream);
    }
    hipError_t e = fn();
    if (record && rec.start && rec.stop) {
        (void)hipEventRecord(rec.stop, stream);
        ctx->prof.push_back(rec);
    }
    if (e != hipSuccess) return hip_fail(ctx, e, what);
    return CONVCRF_OK;
}

hipError_t launch_iter(const IterArgs& a, int k, bool mat, TileConfig t, size_t lds,
                       hipStream_t s) {
    switch (k) {
        case 1: return launch_iter_k1(a, mat, t, lds, s);
        case 3: return launch_iter_k3(a, mat, t, lds, s);
        case 5: return launch_iter_k5(a, mat, t, lds, s);
        case 7: return launch_iter_k7(a, mat, t, lds, s);
        case 9: return launch_iter_k9(a, mat, t, lds, s);
        case 11: return launch_iter_k11(a, mat, t, lds, s);
        case 13: return launch_iter_k13(a, mat, t, lds, s);
        case 15: return launch_iter_k15(a, mat, t, lds, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_pmsg(const IterArgs& a, int k, int nchunks, size_t lds, hipStream_t s) {
    switch (k) {
        case 1: return launch_pmsg_k1(a, nchunks, lds, s);
        case 3: return launch_pmsg_k3(a, nchunks, lds, s);
        case 5: return launch_pmsg_k5(a, nchunks, lds, s);
        case 7: return launch_pmsg_k7(a, nchunks, lds, s);
        case 9: return launch_pmsg_k9(a, nchunks, lds, s);
        case 11: return launch_pmsg_k11(a, nchunks, lds, s);
        case 13: return launch_pmsg_k13(a, nchunks, lds, s);
        case 15: return launch_pmsg_k15(a, nchunks, lds, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t convcrf::launch_blur_iter(const BlurIterArgs& a, int k, hipStream_t s) {
    switch (k) {
        case 3: return launch_blur_iter_k3(a, s);
        case 5: return launch_blur_iter_k5(a, s);
        case 7: return launch_blur_iter_k7(a, s);
        case 9: return launch_blur_iter_k9(a, s);
        case 11: return launch_blur_iter_k11(a, s);
        case 13: return launch_blur_iter_k13(a, s);
        case 15: return launch_blur_iter_k15(a, s);
        default: return hipErrorNotSupported;
    }
}

namespace {

hipError_t launch_rstream(const IterArgs& a, int k, size_t lds, int num_cus, hipStream_t s,
                          bool probe) {
    switch (k) {
        case 3: return launch_rstream_k3(a, lds, num_cus, s, probe);
        case 5: return launch_rstream_k5(a, lds, num_cus, s, probe);
        case 7: return launch_rstream_k7(a, lds, num_cus, s, probe);
        default: return hipErrorNotSupported;
    }
}

hipError_t launch_stream(const IterArgs& a, int k, size_t lds, hipStream_t s) {
    switch (k) {
        case 3: return launch_stream_k3(a, lds, s);
        case 5: return launch_stream_k5(a, lds, s);
        case 7: {
            // the first round, Potts without a centre tap: the quad form
            const hipError_t e = a.first ? launch_quad_first_k7(a, s) : hipErrorNotSupported;
            return e == hipErrorNotSupported ? launch_stream_k7(a, lds, s) : e;
        }
        default: return hipErrorNotSupported;
    }
}

hipError_t launch_ring(const IterArgs& a, int k, hipStream_t s) {
    switch (k) {
        case 3: return launch_ring_k3(a, s);
        case 5: return launch_ring_k5(a, s);
        case 7: {
            // Potts without a centre tap or features: the quad form
            const hipError_t e = launch_quad_k7(a, s);
            return e == hipErrorNotSupported ? launch_ring_k7(a, s) : e;
        }
        default: return hipErrorNotSupported;
    }
}

hipError_t launch_resident(const IterArgs& a, int k, TileConfig t, size_t lds, int num_cus,
                           hipStream_t s, bool probe) {
    switch (k) {
        case 1: return launch_resident_k1(a, t, lds, num_cus, s, probe);
        case 3: return launch_resident_k3(a, t, lds, num_cus, s, probe);
        case 5: return launch_resident_k5(a, t, lds, num_cus, s, probe);
        case 7: return launch_resident_k7(a, t, lds, num_cus, s, probe);
        default: return hipErrorNotSupported;
    }
}

// Tile of iter_kernel: the first candidate whose LDS fits one work-group
// (rows = 0 if none does).  32 columns; up to k = 7 two pixels per thread
// (512 threads on 32 rows, two waves per SIMD), wider windows four pixels
// per thread; fewer rows when the classes and the halo outgrow the LDS.
TileConfig pick_tile(int k, int C, bool colour, bool compat) {
    const TileConfig narrow[] = {{32, 2, 32}, {16, 2, 32}, {8, 2, 32}};
    const TileConfig wide[] = {{32, 4, 32}, {16, 4, 32}, {8, 4, 32}};
    const TileConfig* cand = k <= 7 ? narrow : wide;
    for (int i = 0; i < 3; ++i)
        if (iter_lds_bytes(k, C, cand[i], colour, compat) <= kLdsLimit) return cand[i];
    return TileConfig{0, 4, 32};
}

// Tiling of the unpooled iterations over B x C x H x W.  `a` already holds
// the parameters (compatibility, centre, taps); this sets its sizes and
// tiles, and `as`, the copy with the tiling of the streamed kernel.
// `bufs` are the Q buffers the launches read or write besides the unary.
// streamed: whether the streamed kernel runs the iterations (k = 3..7,
// C = 19 or 21, whole float2 rows, unary rows in 16-byte pieces, buffers
// under 2 GB, the LDS within bounds).
void plan_unpooled(IterArgs& a, IterArgs& as, IterArgs& ar, bool& streamed, bool& ring,
                   size_t& lds_s, TileConfig tile, bool mat, int k, int B, int C, int H, int W,
                   const float* unary, const float* image, const float* kmat,
                   std::initializer_list<const void*> bufs) {
    a.C = C;
    a.planes = C;
    a.H = H;
    a.W = W;
    a.unary = unary;
    a.feat = image;
    a.kmat = kmat;
    a.tiles_x = (W + tile.width - 1) / tile.width;
    a.tiles_per_img = a.tiles_x * ((H + tile.rows - 1) / tile.rows);
    a.ntiles = a.tiles_per_img * B;
    a.mode = kModeUpdate;
    const uintptr_t va = 4u * tile.pix;
    bool aligned = reinterpret_cast<uintptr_t>(unary) % va == 0;
    for (const void* b : bufs) aligned = aligned && reinterpret_cast<uintptr_t>(b) % va == 0;
    a.vec = (W % tile.pix == 0) && aligned;
    lds_s = stream_lds_bytes(k, C, a.mu != nullptr);
    streamed = !mat && k >= 3 && k <= 7 && (C == 19 || C == 21) && a.vec && W % 4 == 0 &&
               reinterpret_cast<uintptr_t>(unary) % 16 == 0 && lds_s <= kLdsLimit &&
               (size_t)C * H * W * 4 < (1ull << 31);
    as = a;
    as.tiles_x = (W + kStreamTW - 1) / kStreamTW;
    as.tiles_per_img = as.tiles_x * ((H + kStreamRows - 1) / kStreamRows);
    as.ntiles = as.tiles_per_img * B;
    // the later streamed iterations on half-height tiles, two work-groups
    // per CU (the first one stages all classes at once and keeps stream_kernel)
    ar = as;
    ar.tiles_per_img = as.tiles_x * ((H + kRingRows - 1) / kRingRows);
    ar.ntiles = ar.tiles_per_img * B;
    ring = streamed && ring_lds_bytes(k, C, C == 19 ? 4 : 3, a.mu != nullptr) <= kLdsLimit;
}

// Ring launches for the learnable-feature iterations (Sec. 4.2, "+T") over
// B x C x H x W: true and `ar` set when the shapes allow them (k = 3..7,
// C = 19 or 21, 1..kMaxFeat feature planes, whole float2 rows with W a
// multiple of 4, the unary 16-byte aligned, buffers under 2 GB, the LDS
// within bounds); every iteration then reads Q_t (no first-iteration form).
bool plan_feature_ring(IterArgs& ar, const convcrf_params& p, const float* unary,
                       const float* image, const float* mu_dev, int B, int C, int H, int W,
                       std::initializer_list<const void*> bufs) {
    const int k = p.filter_size, D = p.feature_dim;
    if (k < 3 || k > 7 || D < 1 || D > kMaxFeat || (size_t)D * H * W * 4 >= (1ull << 31))
        return false;
    IterArgs a{}, as{};
    a.mu = mu_dev;
    a.include_center = p.include_center;
    a.neg_beta = (float)(-kLog2eD / (2.0 * (double)p.theta_beta * p.theta_beta));
    a.center_w = (float)((double)p.w_app + (double)p.w_smooth);
    fill_taps(p, 1, a.taps);
    bool streamed = false, ring = false;
    size_t lds_s = 0;
    plan_unpooled(a, as, ar, streamed, ring, lds_s, TileConfig{32, 2, 32}, false, k, B, C, H, W,
                  unary, image, nullptr, bufs);
    if (!ring || ring_lds_bytes(k, C, C == 19 ? 4 : 3, mu_dev != nullptr, D) > kLdsLimit)
        return false;
    ar.sfeat = p.features;
    ar.D = D;
    ar.neg_gamma = (float)(-kLog2eD / (2.0 * (double)p.theta_gamma * p.theta_gamma));
    ar.w_smooth = p.w_smooth;
    ar.first = 0;
    return true;
}

// Arguments of the learnable-feature update over B x C x H x W.
FeatArgs feat_args(const convcrf_params& p, const float* unary, const float* image,
                   const float* mu_dev, int B, int C, int H, int W) {
    FeatArgs f{};
    f.unary = unary;
    f.image = image;
    f.feat = p.features;
    f.mu = mu_dev;
    f.C = C;
    f.H = H;
    f.W = W;
    f.D = p.feature_dim;
    f.tiles_x = (W + kFeatTW - 1) / kFeatTW;
    f.tiles_per_img = f.tiles_x * ((H + kFeatTH - 1) / kFeatTH);
    f.ntiles = f.tiles_per_img * B;
    f.include_center = p.include_center;
    // 16-byte staging: whole vectors per row, every plane 16-byte aligned
    f.vec4 = p.filter_size <= 7 && W % 4 == 0 && reinterpret_cast<uintptr_t>(image) % 16 == 0 &&
             reinterpret_cast<uintptr_t>(p.features) % 16 == 0 &&
             feat_lds_bytes(p.filter_size, C, p.feature_dim, true) <= kLdsLimit;
    f.neg_beta = (float)(-kLog2eD / (2.0 * (double)p.theta_beta * p.theta_beta));
    f.neg_gamma = (float)(-kLog2eD / (2.0 * (double)p.theta_gamma * p.theta_gamma));
    f.w_app = p.w_app;
    f.w_smooth = p.w_smooth;
    for (int n = 0; n <= kMaxN; ++n)
        f.a_log2[n] = (float)(-(double)n * kLog2eD /
                              (2.0 * (double)p.theta_alpha * p.theta_alpha));
    return f;
}

// Upload mu (C*C floats) if it differs from what the device holds.
convcrf_status upload_mu(convcrf_ctx* ctx, const float* mu, int C, hipStream_t stream) {
    const size_t n = (size_t)C * C;
    if (ctx->mu_last.size() == n && std::memcmp(ctx->mu_last.data(), mu, n * sizeof(float)) == 0)
        return CONVCRF_OK;
    convcrf_status st = ensure(ctx, ctx->mu, n * sizeof(float));
    if (st != CONVCRF_OK) return st;
    hipError_t e;
    if (ctx->mu_pinned_cap < n) {
        if (ctx->mu_pinned) {
            if (ctx->mu_copied) (void)hipEventSynchronize(ctx->mu_copied);
            (void)hipHostFree(ctx->mu_pinned);
            ctx->mu_pinned = nullptr;
        }
        e = hipHostMalloc(reinterpret_cast<void**>(&ctx->mu_pinned), kMaxC * kMaxC * sizeof(float), 0);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipHostMalloc");
        ctx->mu_pinned_cap = kMaxC * kMaxC;
    }
    if (!ctx->mu_copied) {
        e = hipEventCreateWithFlags(&ctx->mu_copied, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventCreate");
    } else {
        e = hipEventSynchronize(ctx->mu_copied);  // previous upload has left the staging
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventSynchronize");
    }
    std::memcpy(ctx->mu_pinned, mu, n * sizeof(float));
    e = hipMemcpyAsync(ctx->mu.p, ctx->mu_pinned, n * sizeof(float), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipMemcpyAsync(compat)");
    e = hipEventRecord(ctx->mu_copied, stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipEventRecord");
    ctx->mu_last.assign(mu, mu + n);
    return CONVCRF_OK;
}

// Report a wait overrun of an earlier resident call: the sticky flag
// sync[0] is copied to pinned host memory after each resident launch (when
// no copy is outstanding).  Non-blocking: a copy not yet landed is left for
// a later check.
convcrf_status poll_overrun(convcrf_ctx* ctx) {
    if (!ctx->flag_pending) return CONVCRF_OK;
    const hipError_t e = hipEventQuery(ctx->flag_event);
    if (e == hipErrorNotReady) {
        (void)hipGetLastError();
        return CONVCRF_OK;
    }
    ctx->flag_pending = false;
    if (e != hipSuccess) return hip_fail(ctx, e, "hipEventQuery(resident flag)");
    if (*ctx->flag_host == 0) return CONVCRF_OK;
    *ctx->flag_host = 0;
    // clear the device flag (ordered after the copy that saw it)
    const hipError_t z = launch_zero_u32(static_cast<unsigned int*>(ctx->sync.p), 1, nullptr);
    if (z != hipSuccess) return hip_fail(ctx, z, "clearing the resident flag");
    return fail(ctx, CONVCRF_E_HIP,
                "an earlier CONVCRF_VARIANT_RESIDENT call passed the bound of a neighbour wait; "
                "the Q it wrote is not valid");
}

// Blocking form: wait for the device and read the flag itself.
convcrf_status check_overrun(convcrf_ctx* ctx) {
    if (!ctx->sync.p) return CONVCRF_OK;
    ctx->flag_pending = false;
    unsigned int v = 0;
    hipError_t e = hipMemcpy(&v, ctx->sync.p, sizeof(v), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(ctx, e, "reading the resident flag");
    if (v == 0) return CONVCRF_OK;
    e = launch_zero_u32(static_cast<unsigned int*>(ctx->sync.p), 1, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(ctx, e, "clearing the resident flag");
    return fail(ctx, CONVCRF_E_HIP,
                "a CONVCRF_VARIANT_RESIDENT call passed the bound of a neighbour wait; the Q it "
                "wrote is not valid");
}

// The flag words of a resident launch over `ntiles` tiles: sync[0] (sticky,
// checked before the buffer is replaced) and one counter per tile.
convcrf_status ensure_sync(convcrf_ctx* ctx, size_t ntiles, hipStream_t stream) {
    const size_t bytes = (1 + ntiles) * sizeof(unsigned int);
    if (ctx->sync.bytes >= bytes) return CONVCRF_OK;
    convcrf_status st = check_overrun(ctx);
    if (st != CONVCRF_OK) return st;
    if ((st = ensure(ctx, ctx->sync, bytes)) != CONVCRF_OK) return st;
    const hipError_t e = launch_zero_u32(static_cast<unsigned int*>(ctx->sync.p), 1, stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "clearing the resident flag");
    return CONVCRF_OK;
}

// After a resident launch: copy the sticky flag back (one copy outstanding
// at a time; a flag set meanwhile stays set for the next copy).
convcrf_status queue_overrun_check(convcrf_ctx* ctx, hipStream_t stream) {
    if (ctx->flag_pending) return CONVCRF_OK;
    hipError_t e;
    if (!ctx->flag_host) {
        e = hipHostMalloc(reinterpret_cast<void**>(&ctx->flag_host), sizeof(unsigned int), 0);
        if (e != hipSuccess) {
            ctx->flag_host = nullptr;
            return hip_fail(ctx, e, "hipHostMalloc(resident flag)");
        }
        *ctx->flag_host = 0;
    }
    if (!ctx->flag_event) {
        e = hipEventCreateWithFlags(&ctx->flag_event, hipEventDisableTiming);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventCreate(resident flag)");
    }
    e = hipMemcpyAsync(ctx->flag_host, ctx->sync.p, sizeof(unsigned int), hipMemcpyDeviceToHost,
                       stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipMemcpyAsync(resident flag)");
    e = hipEventRecord(ctx->flag_event, stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipEventRecord(resident flag)");
    ctx->flag_pending = true;
    return CONVCRF_OK;
}

// ---- the allocation-free entry point's scratch memory
// One array per device, for callers that cannot allocate (graph capture,
// serving loops): the Q ping-pong buffer, the pooled buffers of the blur
// path and the compatibility matrix of a convcrf_meanfield_noalloc call are
// carved from it.  Its name is a host-side stand-in: host code uses only the
// device address hipGetSymbolAddress returns for it, taken once per device
// (with that device current) by convcrf_init.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on `device` (current on entry), taken on
// the first call for that device.
hipError_t scratch_address(int device, void** out) {
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    if (!g_scratch_ptr[device]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[device] = ptr;
    }
    *out = g_scratch_ptr[device];
    return hipSuccess;
}

// Where a call's workspace comes from: the context's growable buffers, or
// consecutive 256-byte aligned slices of the scratch array (no allocation;
// sizes beyond it are refused).
struct Workspace {
    char* base = nullptr;     // scratch address, or null: the context's buffers
    size_t used = 0;
    size_t need = 0;          // bytes the call asked of the scratch array
};

convcrf_status take(convcrf_ctx* ctx, Workspace& w, DevBuf& buf, size_t bytes, void** out) {
    if (!w.base) {
        convcrf_status st = ensure(ctx, buf, bytes);
        if (st != CONVCRF_OK) return st;
        *out = buf.p;
        return CONVCRF_OK;
    }
    const size_t at = (w.used + 255) / 256 * 256;
    w.need = at + bytes;
    if (w.need > kNoAllocScratchBytes)
        return fail(ctx, CONVCRF_E_UNSUPPORTED,
                    "convcrf_meanfield_noalloc: this call needs " + std::to_string(w.need) +
                        " bytes of workspace, more than its " +
                        std::to_string(kNoAllocScratchBytes) + "-byte scratch array");
    w.used = at + bytes;
    *out = w.base + at;
    return CONVCRF_OK;
}

// The compatibility matrix for an allocation-free call: copied into the
// scratch slice by a kernel that takes the C x C values as its argument, so
// that no pinned staging buffer is needed.
convcrf_status upload_mu_noalloc(convcrf_ctx* ctx, Workspace& w, const float* mu, int C,
                                 hipStream_t stream, const float** out) {
    void* dst = nullptr;
    DevBuf unused;
    convcrf_status st = take(ctx, w, unused, sizeof(float) * (size_t)C * C, &dst);
    if (st != CONVCRF_OK) return st;
    CompatBlock blk{};
    std::memcpy(blk.v, mu, sizeof(float) * (size_t)C * C);
    const hipError_t e = launch_copy_compat(blk, C * C, static_cast<float*>(dst), stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "copying the compatibility matrix");
    *out = static_cast<const float*>(dst);
    return CONVCRF_OK;
}

}  // namespace

extern "C" {

const char* convcrf_status_string(convcrf_status s) {
    switch (s) {
        case CONVCRF_OK: return "CONVCRF_OK";
        case CONVCRF_E_INVALID_ARG: return "CONVCRF_E_INVALID_ARG";
        case CONVCRF_E_UNSUPPORTED: return "CONVCRF_E_UNSUPPORTED";
        case CONVCRF_E_NO_DEVICE: return "CONVCRF_E_NO_DEVICE";
        case CONVCRF_E_HIP: return "CONVCRF_E_HIP";
        case CONVCRF_E_OOM: return "CONVCRF_E_OOM";
    }
    return "CONVCRF_E_UNKNOWN";
}

const char* convcrf_last_error(const convcrf_ctx* ctx) {
    return ctx ? ctx->err.c_str() : g_last_error.c_str();
}

const char* convcrf_strerror(const convcrf_ctx* ctx, convcrf_status status) {
    thread_local std::string text;
    if (status == CONVCRF_OK) return convcrf_status_string(status);
    text = std::string(convcrf_status_string(status)) + ": " + convcrf_last_error(ctx);
    return text.c_str();
}

convcrf_status convcrf_synchronize(convcrf_ctx* ctx, void* stream) {
    if (!ctx) return fail(nullptr, CONVCRF_E_INVALID_ARG, "ctx is NULL");
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    return check_overrun(ctx);
}

convcrf_status convcrf_default_params(convcrf_params* p) {
    if (!p) return fail(nullptr, CONVCRF_E_INVALID_ARG, "params is NULL");
    p->filter_size = 7;
    p->blur = 1;
    p->include_center = 0;
    p->variant = CONVCRF_VARIANT_FUSED;
    p->w_app = 10.f;
    p->theta_alpha = 80.f;
    p->theta_beta = 13.f;
    p->w_smooth = 3.f;
    p->theta_gamma = 3.f;
    p->compat = nullptr;
    p->features = nullptr;
    p->feature_dim = 0;
    return CONVCRF_OK;
}

convcrf_status convcrf_validate(int B, int C, int H, int W, const convcrf_params* params,
                                int iters) {
    return validate(nullptr, B, C, H, W, params, iters);
}

convcrf_status convcrf_init(convcrf_ctx** out, int device) {
    if (!out) return fail(nullptr, CONVCRF_E_INVALID_ARG, "out is NULL");
    *out = nullptr;
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        return fail(nullptr, CONVCRF_E_NO_DEVICE, "no HIP device is visible");
    }
    if (device < 0 || device >= n) return fail(nullptr, CONVCRF_E_NO_DEVICE, "device index out of range");
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return fail(nullptr, CONVCRF_E_NO_DEVICE, hipGetErrorString(e));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(nullptr, CONVCRF_E_NO_DEVICE,
                    std::string("device is ") + prop.gcnArchName + ", library is built for gfx950");
    convcrf_ctx* ctx = new (std::nothrow) convcrf_ctx();
    if (!ctx) return fail(nullptr, CONVCRF_E_OOM, "context allocation failed");
    ctx->device = device;
    ctx->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
    {
        // the scratch array's address on this device, with the device current
        int prev = 0;
        (void)hipGetDevice(&prev);
        void* ptr = nullptr;
        e = hipSetDevice(device);
        if (e == hipSuccess) e = scratch_address(device, &ptr);
        // the allocation-free entry point's one kernel of its own is launched
        // once here (copying nothing), so that whatever the runtime sets up
        // on a kernel's first launch happens at set-up, not inside that call
        if (e == hipSuccess) e = launch_copy_compat(CompatBlock{}, 0, static_cast<float*>(ptr), nullptr);
        if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
        (void)hipSetDevice(prev);
        if (e != hipSuccess) {
            delete ctx;
            (void)hipGetLastError();
            return fail(nullptr, CONVCRF_E_HIP,
                        std::string("scratch array address: ") + hipGetErrorString(e));
        }
        ctx->scratch_ptr = ptr;
    }
    int coop = 0;
    if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, device) == hipSuccess)
        ctx->coop = coop != 0;
    (void)hipGetLastError();
    *out = ctx;
    return CONVCRF_OK;
}

void convcrf_destroy(convcrf_ctx* ctx) {
    if (!ctx) return;
    int prev = 0;
    (void)hipGetDevice(&prev);
    (void)hipSetDevice(ctx->device);
    (void)hipDeviceSynchronize();
    for (DevBuf* b : {&ctx->q_ws, &ctx->q_ws2, &ctx->kmat, &ctx->pool_q, &ctx->pool_m,
                      &ctx->pool_f, &ctx->mu, &ctx->sync, &ctx->b_q, &ctx->b_dq, &ctx->b_dm,
                      &ctx->b_dp, &ctx->b_gpart, &ctx->b_kpart, &ctx->b_df,
                      &ctx->b_pd, &ctx->b_dfp})
        if (b->p) (void)hipFree(b->p);
    if (ctx->mu_pinned) (void)hipHostFree(ctx->mu_pinned);
    if (ctx->mu_copied) (void)hipEventDestroy(ctx->mu_copied);
    if (ctx->flag_host) (void)hipHostFree(ctx->flag_host);
    if (ctx->flag_event) (void)hipEventDestroy(ctx->flag_event);
    for (auto& r : ctx->prof) {
        (void)hipEventDestroy(r.start);
        (void)hipEventDestroy(r.stop);
    }
    for (hipEvent_t e : ctx->free_events) (void)hipEventDestroy(e);
    (void)hipSetDevice(prev);
    delete ctx;
}

convcrf_status convcrf_profile_enable(convcrf_ctx* ctx, int enable) {
    if (!ctx) return fail(nullptr, CONVCRF_E_INVALID_ARG, "ctx is NULL");
    if (enable) {
        for (auto& r : ctx->prof) {
            (void)hipEventSynchronize(r.stop);
            ctx->free_events.push_back(r.start);
            ctx->free_events.push_back(r.stop);
        }
        ctx->prof.clear();
    }
    ctx->profiling = enable != 0;
    return CONVCRF_OK;
}

convcrf_status convcrf_profile_read(convcrf_ctx* ctx, const char* name, double* total_ms,
                                    int64_t* launches) {
    if (!ctx || !name || !total_ms || !launches)
        return fail(ctx, CONVCRF_E_INVALID_ARG, "NULL argument");
    int id = -1;
    for (int i = 0; i < kNumKernels; ++i)
        if (std::strcmp(name, kKernelNames[i]) == 0) id = i;
    double tot = 0.0;
    int64_t cnt = 0;
    for (auto& r : ctx->prof) {
        if (r.kernel != id) continue;
        hipError_t e = hipEventSynchronize(r.stop);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventSynchronize");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, r.start, r.stop);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipEventElapsedTime");
        tot += ms;
        ++cnt;
    }
    *total_ms = tot;
    *launches = cnt;
    return CONVCRF_OK;
}

}  // extern "C"

namespace {

// convcrf_meanfield, with its workspace from w (the context's buffers when
// w.base is null, else the scratch array: no allocation, no events, the
// materialised variant refused and the resident one run as fused).
convcrf_status meanfield_impl(convcrf_ctx* ctx, const float* unary, const float* image, int B,
                              int C, int H, int W, const convcrf_params* params, int iters,
                              float* q_out, void* stream_ptr, Workspace& w) {
    if (!ctx) return fail(nullptr, CONVCRF_E_INVALID_ARG, "ctx is NULL");
    convcrf_status st = validate(ctx, B, C, H, W, params, iters);
    if (st != CONVCRF_OK) return st;
    const long long npix = (long long)B * H * W;
    if (npix == 0) return CONVCRF_OK;  // empty input: nothing to compute
    if (!unary || !image || !q_out) return fail(ctx, CONVCRF_E_INVALID_ARG, "NULL tensor pointer");
    const size_t qbytes = sizeof(float) * (size_t)npix * C;
    const size_t ibytes = sizeof(float) * (size_t)npix * 3;
    if (overlaps(q_out, qbytes, unary, qbytes) || overlaps(q_out, qbytes, image, ibytes))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "q_out overlaps unary or image");
    if (params->features &&
        overlaps(q_out, qbytes, params->features, sizeof(float) * (size_t)npix * params->feature_dim))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "q_out overlaps the features");

    const convcrf_params p = *params;
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    if ((st = poll_overrun(ctx)) != CONVCRF_OK) return st;

    if (iters == 0)
        return launch(ctx, kSoftmax, stream, "softmax",
                      [&] { return launch_softmax(unary, q_out, B, C, H * W, stream); });

    const int k = p.filter_size;
    const int s = p.blur;
    const bool mat = p.variant == CONVCRF_VARIANT_MATERIALISED;
    const bool noalloc = w.base != nullptr;
    if (noalloc && mat)
        return fail(ctx, CONVCRF_E_UNSUPPORTED,
                    "convcrf_meanfield_noalloc: the materialised variant needs its kernel matrix "
                    "allocated; use convcrf_meanfield");
    const float* mu_dev = nullptr;
    if (p.compat) {
        if (noalloc) {
            st = upload_mu_noalloc(ctx, w, p.compat, C, stream, &mu_dev);
            if (st != CONVCRF_OK) return st;
        } else {
            st = upload_mu(ctx, p.compat, C, stream);
            if (st != CONVCRF_OK) return st;
            mu_dev = static_cast<const float*>(ctx->mu.p);
        }
    }

    if (p.features && s == 1) {
        // learnable smoothness features: Q0 = softmax(U), then one update
        // launch per iteration, the last one into q_out
        void* wsp = nullptr;
        if ((st = take(ctx, w, ctx->q_ws, qbytes, &wsp)) != CONVCRF_OK) return st;
        float* ws = static_cast<float*>(wsp);
        FeatArgs f = feat_args(p, unary, image, mu_dev, B, C, H, W);
        // the staged Q planes live in q_out and the workspace
        f.vec4 = f.vec4 && reinterpret_cast<uintptr_t>(q_out) % 16 == 0 &&
                 reinterpret_cast<uintptr_t>(ws) % 16 == 0;
        IterArgs ar{};
        const bool ring = plan_feature_ring(ar, p, unary, image, mu_dev, B, C, H, W, {q_out, ws});
        float* q0 = iters % 2 == 0 ? q_out : ws;
        st = launch(ctx, kSoftmax, stream, "softmax",
                    [&] { return launch_softmax(unary, q0, B, C, H * W, stream); });
        if (st != CONVCRF_OK) return st;
        const float* cur = q0;
        for (int t = 0; t < iters; ++t) {
            f.src = ar.src = cur;
            f.dst = ar.dst = ((iters - 1 - t) % 2 == 0) ? q_out : ws;
            st = launch(ctx, kFeatIter, stream, "feature_iter", [&] {
                return ring ? launch_ring(ar, k, stream) : launch_feat_update(f, k, stream);
            });
            if (st != CONVCRF_OK) return st;
            cur = f.dst;
        }
        return CONVCRF_OK;
    }

    IterArgs a{};
    a.mu = mu_dev;
    a.include_center = p.include_center;
    a.neg_beta = (float)(-kLog2eD / (2.0 * (double)p.theta_beta * p.theta_beta));
    a.center_w = (float)((double)p.w_app + (double)p.w_smooth);
    fill_taps(p, s, a.taps);

    if (s == 1) {
        const TileConfig tile = pick_tile(k, C, !mat, mu_dev != nullptr);
        if (tile.rows == 0) return fail(ctx, CONVCRF_E_UNSUPPORTED, "window and classes exceed LDS");
        const size_t lds = iter_lds_bytes(k, C, tile, !mat, mu_dev != nullptr);
        void* wsp = nullptr;
        if (iters > 1) {
            st = take(ctx, w, ctx->q_ws, qbytes, &wsp);
            if (st != CONVCRF_OK) return st;
        }
        if (mat) {
            st = ensure(ctx, ctx->kmat, sizeof(float) * (size_t)npix * (k * k - 1));
            if (st != CONVCRF_OK) return st;
            if (k > 1) {
                st = launch(ctx, kBuild, stream, "build_kernel", [&] {
                    return launch_build_kernel(image, static_cast<float*>(ctx->kmat.p), B, H, W, k,
                                               a.neg_beta, a.taps, stream);
                });
                if (st != CONVCRF_OK) return st;
            }
        }
        IterArgs as, ar;                      // the streamed and ring launches' tilings
        bool streamed = false, ring = false;
        size_t lds_s = 0;
        plan_unpooled(a, as, ar, streamed, ring, lds_s, tile, mat, k, B, C, H, W, unary, image,
                      static_cast<const float*>(ctx->kmat.p), {q_out, wsp});
        // Resident variant: all iterations in one launch when every tile's
        // work-group fits on the device at once (Potts): the tile stays in
        // LDS and only border rings cross memory.  On the streamed tiles the
        // weights and the unary also stay in registers for the whole call.
        if (p.variant == CONVCRF_VARIANT_RESIDENT && !noalloc && !mu_dev && iters >= 2 &&
            ctx->coop && streamed && as.ntiles <= 4 * ctx->num_cus) {
            if ((st = ensure(ctx, ctx->q_ws2, qbytes)) != CONVCRF_OK) return st;
            if ((st = ensure_sync(ctx, (size_t)as.ntiles, stream)) != CONVCRF_OK) return st;
            IterArgs r = as;
            r.src = unary;
            r.dst = q_out;
            r.first = 1;
            r.iters = iters;
            r.ring[0] = static_cast<float*>(ctx->q_ws.p);
            r.ring[1] = static_cast<float*>(ctx->q_ws2.p);
            r.sync = static_cast<unsigned int*>(ctx->sync.p);
            const hipError_t fits = launch_rstream(r, k, lds_s, ctx->num_cus, stream, true);
            if (fits == hipSuccess) {
                st = launch(ctx, kSyncReset, stream, "sync_reset",
                            [&] { return launch_zero_u32(r.sync + 1, as.ntiles, stream); });
                if (st != CONVCRF_OK) return st;
                st = launch(ctx, kResident, stream, "fused_resident", [&] {
                    return launch_rstream(r, k, lds_s, ctx->num_cus, stream, false);
                });
                if (st != CONVCRF_OK) return st;
                return queue_overrun_check(ctx, stream);
            }
            (void)hipGetLastError();  // refused: one launch per iteration below
            ctx->err = std::string("resident launch refused (") + hipGetErrorString(fits) +
                       "); ran one launch per iteration";
        } else if (p.variant == CONVCRF_VARIANT_RESIDENT && !noalloc && !mu_dev && iters >= 2 &&
                   ctx->coop && tile.pix == 2 && tile.width == 32 && k <= 7 &&
                   a.ntiles <= 4 * ctx->num_cus) {
            if ((st = ensure(ctx, ctx->q_ws2, qbytes)) != CONVCRF_OK) return st;
            if ((st = ensure_sync(ctx, (size_t)a.ntiles, stream)) != CONVCRF_OK) return st;
            IterArgs r = a;
            r.src = unary;
            r.dst = q_out;
            r.first = 1;
            r.iters = iters;
            r.ring[0] = static_cast<float*>(ctx->q_ws.p);
            r.ring[1] = static_cast<float*>(ctx->q_ws2.p);
            r.sync = static_cast<unsigned int*>(ctx->sync.p);
            const hipError_t fits = launch_resident(r, k, tile, lds, ctx->num_cus, stream, true);
            if (fits == hipSuccess) {
                st = launch(ctx, kSyncReset, stream, "sync_reset",
                            [&] { return launch_zero_u32(r.sync + 1, a.ntiles, stream); });
                if (st != CONVCRF_OK) return st;
                st = launch(ctx, kResident, stream, "fused_resident", [&] {
                    return launch_resident(r, k, tile, lds, ctx->num_cus, stream, false);
                });
                if (st != CONVCRF_OK) return st;
                return queue_overrun_check(ctx, stream);
            }
            (void)hipGetLastError();  // refused: one launch per iteration below
            ctx->err = std::string("resident launch refused (") + hipGetErrorString(fits) +
                       "); ran one launch per iteration";
        }
        float* ws = static_cast<float*>(wsp);
        // the last iteration writes q_out; earlier ones alternate so that
        // source and destination always differ
        const float* cur = unary;
        for (int t = 0; t < iters; ++t) {
            float* dst = ((iters - 1 - t) % 2 == 0) ? q_out : ws;
            a.src = as.src = ar.src = cur;
            a.dst = as.dst = ar.dst = dst;
            a.first = as.first = ar.first = t == 0;
            st = launch(ctx, mat ? kMatIter : (t == 0 ? kFusedFirst : kFused), stream,
                        mat ? "materialised_iter" : "fused_iter", [&] {
                            if (ring && t > 0) return launch_ring(ar, k, stream);
                            return streamed ? launch_stream(as, k, lds_s, stream)
                                            : launch_iter(a, k, mat, tile, lds, stream);
                        });
            if (st != CONVCRF_OK) return st;
            cur = dst;
        }
        return CONVCRF_OK;
    }

    // ---- blur: message on the s x s pooled grid (Sec. 4.2)
    const int Hp = H / s, Wp = W / s;
    const size_t pbytes = sizeof(float) * (size_t)B * Hp * Wp;
    void *qpv = nullptr, *mpv = nullptr, *fpv = nullptr;
    if ((st = take(ctx, w, ctx->pool_q, pbytes * C, &qpv)) != CONVCRF_OK) return st;
    if ((st = take(ctx, w, ctx->pool_m, pbytes * C, &mpv)) != CONVCRF_OK) return st;
    // pooled colours, then (learnable features) the pooled features
    const int D = p.features ? p.feature_dim : 0;
    const size_t fcol = ((size_t)B * 3 * Hp * Wp + 63) / 64 * 64;   // floats, whole 256 B
    if ((st = take(ctx, w, ctx->pool_f, sizeof(float) * fcol + pbytes * D, &fpv)) != CONVCRF_OK)
        return st;
    float* qp = static_cast<float*>(qpv);
    float* mp = static_cast<float*>(mpv);
    float* fp = static_cast<float*>(fpv);
    float* sfp = D > 0 ? fp + fcol : nullptr;
    // 4 x 4 pooling: one launch initialises (softmax(U), the image and the
    // learnable features, pooled), then one fused launch per iteration (pooled
    // message of each work-group's cells and the full-resolution update of its
    // pixels), the pooled Q ping-ponging between qp and mp; the last one
    // writes q_out.  Other poolings take the general form below.
    const auto al8 = [](const void* ptr) { return reinterpret_cast<uintptr_t>(ptr) % 8 == 0; };
    if (s == kFusedBlurFactor && k >= 3 && B <= 65535 && D <= kMaxFeat && al8(unary) &&
        al8(q_out) && al8(image) && (D == 0 || al8(p.features)) &&
        (Hp + kBlurInitTY - 1) / kBlurInitTY <= 65535 &&
        blur_iter_lds_bytes(k, C == 19 || C == 21 ? C : (C <= 8 ? 8 : 24), mu_dev != nullptr,
                            D > 0 ? kMaxFeat : 0) <= kLdsLimit) {
        BlurInitArgs bin{};
        bin.unary = unary;
        bin.image = image;
        bin.qbar = qp;
        bin.pcol = fp;
        bin.B = B;
        bin.C = C;
        bin.H = H;
        bin.W = W;
        bin.Hp = Hp;
        bin.Wp = Wp;
        bin.feat = D > 0 ? p.features : nullptr;
        bin.pfeat = D > 0 ? sfp : nullptr;
        bin.D = D;
        st = launch(ctx, kPool, stream, "blur_pool", [&] { return launch_blur_init(bin, stream); });
        if (st != CONVCRF_OK) return st;
        BlurIterArgs bi{};
        bi.pcol = fp;
        bi.unary = unary;
        bi.mu = mu_dev;
        bi.B = B;
        bi.C = C;
        bi.H = H;
        bi.W = W;
        bi.Hp = Hp;
        bi.Wp = Wp;
        bi.include_center = p.include_center;
        bi.center_w = a.center_w;
        bi.neg_beta = a.neg_beta;
        bi.taps = a.taps;
        bi.sfeat = D > 0 ? sfp : nullptr;
        bi.D = D;
        bi.w_smooth = p.w_smooth;
        bi.neg_gamma = (float)(-kLog2eD / (2.0 * (double)p.theta_gamma * p.theta_gamma));
        float* cur = qp;
        float* nxt = mp;
        for (int t = 0; t < iters; ++t) {
            const bool last = t == iters - 1;
            bi.qbar = cur;
            bi.qbar_out = last ? nullptr : nxt;
            bi.q_full = last ? q_out : nullptr;
            st = launch(ctx, kBlurIter, stream, "blur_iteration",
                        [&] { return launch_blur_iter(bi, k, stream); });
            if (st != CONVCRF_OK) return st;
            std::swap(cur, nxt);
        }
        return CONVCRF_OK;
    }

    // pooled message: 16 x 8 cell tiles, one wavefront per window row, the
    // classes in chunks of at most kPmsgClasses (the message does not mix
    // classes; each chunk recomputes the weights)
    const int nchunks = (C + kPmsgClasses - 1) / kPmsgClasses;
    const int chunk = (C + nchunks - 1) / nchunks;
    const size_t lds = pmsg_lds_bytes(k, D);
    if (lds > kLdsLimit) return fail(ctx, CONVCRF_E_UNSUPPORTED, "window exceeds LDS");
    st = launch(ctx, kPool, stream, "blur_pool",
                [&] { return launch_pool(image, fp, B, 3, H, W, s, 0, stream); });
    if (st != CONVCRF_OK) return st;
    if (D > 0) {
        st = launch(ctx, kPool, stream, "blur_pool",
                    [&] { return launch_pool(p.features, sfp, B, D, H, W, s, 0, stream); });
        if (st != CONVCRF_OK) return st;
    }
    st = launch(ctx, kPool, stream, "blur_pool",
                [&] { return launch_pool(unary, qp, B, C, H, W, s, 1, stream); });
    if (st != CONVCRF_OK) return st;

    a.C = chunk;
    a.planes = C;
    a.H = Hp;
    a.W = Wp;
    a.unary = nullptr;
    a.feat = fp;
    a.kmat = nullptr;
    a.src = qp;
    a.dst = mp;
    a.first = 0;
    a.mode = kModeMessage;
    a.tiles_x = (Wp + kPmsgTW - 1) / kPmsgTW;
    a.tiles_per_img = a.tiles_x * ((Hp + kPmsgTH - 1) / kPmsgTH);
    a.ntiles = a.tiles_per_img * B;
    a.vec = 0;
    a.sfeat = sfp;
    a.D = D;
    a.w_smooth = p.w_smooth;
    a.neg_gamma = (float)(-kLog2eD / (2.0 * (double)p.theta_gamma * p.theta_gamma));
    for (int t = 0; t < iters; ++t) {
        st = launch(ctx, kBlurMsg, stream, "blur_message",
                    [&] { return launch_pmsg(a, k, nchunks, lds, stream); });
        if (st != CONVCRF_OK) return st;
        const bool last = t == iters - 1;
        st = launch(ctx, kBlurUpd, stream, "blur_update", [&] {
            return launch_blur_update(mp, unary, mu_dev, last ? q_out : nullptr, last ? nullptr : qp,
                                      B, C, H, W, s, stream);
        });
        if (st != CONVCRF_OK) return st;
    }
    return CONVCRF_OK;
}

}  // namespace

extern "C" {

convcrf_status convcrf_meanfield(convcrf_ctx* ctx, const float* unary, const float* image, int B,
                                 int C, int H, int W, const convcrf_params* params, int iters,
                                 float* q_out, void* stream_ptr) {
    Workspace w;
    return meanfield_impl(ctx, unary, image, B, C, H, W, params, iters, q_out, stream_ptr, w);
}

convcrf_status convcrf_meanfield_noalloc(convcrf_ctx* ctx, const float* unary, const float* image,
                                         int B, int C, int H, int W,
                                         const convcrf_params* params, int iters, float* q_out,
                                         void* stream_ptr) {
    if (!ctx) return fail(nullptr, CONVCRF_E_INVALID_ARG, "ctx is NULL");
    if (!ctx->scratch_ptr) return fail(ctx, CONVCRF_E_HIP, "no scratch address for this device");
    Workspace w;
    w.base = static_cast<char*>(ctx->scratch_ptr);
    ctx->no_events = true;
    const convcrf_status st =
        meanfield_impl(ctx, unary, image, B, C, H, W, params, iters, q_out, stream_ptr, w);
    ctx->no_events = false;
    return st;
}

convcrf_status convcrf_meanfield_backward(convcrf_ctx* ctx, const float* unary,
                                          const float* image, int B, int C, int H, int W,
                                          const convcrf_params* params, int iters,
                                          const float* grad_q, float* grad_unary,
                                          float* grad_compat, float* grad_kernel,
                                          float* grad_features, void* stream_ptr) {
    if (!ctx) return fail(nullptr, CONVCRF_E_INVALID_ARG, "ctx is NULL");
    convcrf_status st = validate(ctx, B, C, H, W, params, iters);
    if (st != CONVCRF_OK) return st;
    const convcrf_params p = *params;
    const int k = p.filter_size;
    const int D = p.features ? p.feature_dim : 0;
    // the adjoint message runs on the grid of the message: the image, or
    // with blur s the s x s pooled grid (offsets of s pixels)
    const int s = p.blur;
    const int Hg = H / s, Wg = W / s;
    // staging with buffer loads into LDS needs each image's planes under 2 GB;
    // it pads every plane to whole 64-float rows, and is used only where that
    // keeps the tile height (measured: 8-row tiles cost more than the
    // scalar staging saves)
    // class groups of the adjoint message (grid dim y): every work-group
    // stages and sums its group's classes only, which leaves room for more
    // work-groups per CU and, on small grids, more work-groups.  dL/dF is
    // linear in the per-class sums, so with learnable features each group
    // stores its part and a sum adds the parts in group order
    int groups = std::max(1, std::min(kBwdClassGroups, C / 4));
    if (groups > 1) {
        // small grids (the pooled grid of the blur variant): more groups,
        // down to three classes each, until the launch has kBwdMinGroups
        // work-groups per CU (the tiles of groups of at most 8 classes)
        const long long t8 = (long long)((Wg + bwd_tile_w(k) - 1) / bwd_tile_w(k)) *
                             ((Hg + 7) / 8) * B;
        const long long want = (long long)kBwdMinGroups * ctx->num_cus;
        if (t8 > 0 && t8 * groups < want)
            groups = (int)std::max<long long>(groups, std::min<long long>(C / 3, (want + t8 - 1) / t8));
    }
    const int cgsize = (C + groups - 1) / groups;
    groups = (C + cgsize - 1) / cgsize;
    const long long hw_ll = (long long)Hg * Wg;
    const bool dma = (long long)std::max(std::max(3, C), D) * hw_ll * 4 < (1LL << 31) &&
                     bwd_tile_h(k, C, D, true, cgsize) == bwd_tile_h(k, C, D, false, cgsize);
    if (bwd_lds_need(k, C, D, dma, cgsize) > kBwdLdsLimit)
        return fail(ctx, CONVCRF_E_UNSUPPORTED, "window and classes exceed LDS");
    const long long npix = (long long)B * H * W;
    const size_t qbytes = sizeof(float) * (size_t)npix * C;
    const size_t ibytes = sizeof(float) * (size_t)npix * 3;
    if (npix > 0 && (!unary || !image || !grad_q || !grad_unary))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "NULL tensor pointer");
    if (npix > 0 && (overlaps(grad_unary, qbytes, unary, qbytes) ||
                     overlaps(grad_unary, qbytes, image, ibytes) ||
                     overlaps(grad_unary, qbytes, grad_q, qbytes)))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "grad_unary overlaps unary, image or grad_q");
    if (npix > 0 && D > 0) {
        const size_t fbytes = sizeof(float) * (size_t)npix * D;
        if (overlaps(grad_unary, qbytes, p.features, fbytes))
            return fail(ctx, CONVCRF_E_INVALID_ARG, "grad_unary overlaps the features");
        if (grad_features && (overlaps(grad_features, fbytes, p.features, fbytes) ||
                              overlaps(grad_features, fbytes, unary, qbytes) ||
                              overlaps(grad_features, fbytes, image, ibytes) ||
                              overlaps(grad_features, fbytes, grad_q, qbytes) ||
                              overlaps(grad_features, fbytes, grad_unary, qbytes)))
            return fail(ctx, CONVCRF_E_INVALID_ARG,
                        "grad_features overlaps the features or another tensor");
    }
    hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    if ((st = poll_overrun(ctx)) != CONVCRF_OK) return st;

    const double ta = p.theta_alpha, tb = p.theta_beta, tg = p.theta_gamma;
    // the kernel sums grid offsets n = dx^2 + dy^2; the squared distance in
    // pixels is s^2 n.  With learnable features the smoothness sum is taken
    // on the feature distance itself, which needs no such scale.
    const double s2 = (double)s * s;
    const double s2g = D > 0 ? 1.0 : s2;
    const float scale[5] = {1.f, (float)(s2 * p.w_app / (ta * ta * ta)),
                            (float)(p.w_app / (tb * tb * tb)), 1.f,
                            (float)(s2g * p.w_smooth / (tg * tg * tg))};
    const int tw = bwd_tile_w(k), th = bwd_tile_h(k, C, D, dma, cgsize);
    const long long ntiles_ll = (long long)((Wg + tw - 1) / tw) * ((Hg + th - 1) / th) * B;
    if (ntiles_ll > 0x7fffffffLL) return fail(ctx, CONVCRF_E_UNSUPPORTED, "too many tiles");
    const int ntiles = (int)ntiles_ll;
    const bool run = npix > 0 && iters > 0;
    const long long npg = (long long)B * Hg * Wg;   // pixels of the message grid
    if (p.features && grad_features && npix > 0 &&
        overlaps(grad_features, sizeof(float) * (size_t)npix * D, p.features,
                 sizeof(float) * (size_t)npix * D))
        return fail(ctx, CONVCRF_E_INVALID_ARG, "grad_features overlaps the features");
    if (npix == 0) {
        if (grad_compat || grad_kernel)   // nothing to sum: zeros
            return launch(ctx, kBwdReduce, stream, "bwd_reduce", [&] {
                return launch_bwd_reduce(nullptr, 0, C, grad_compat, nullptr, 0, scale,
                                         grad_kernel, stream);
            });
        return CONVCRF_OK;
    }

    const float* mu_dev = nullptr;
    if (p.compat) {
        if ((st = upload_mu(ctx, p.compat, C, stream)) != CONVCRF_OK) return st;
        mu_dev = static_cast<const float*>(ctx->mu.p);
    }
    const bool potts_dz = mu_dev == nullptr && C > 1;
    // workspace: Q^0 .. Q^T in 256-byte aligned slices
    const size_t slice = (qbytes + 255) / 256 * 256;
    if ((st = ensure(ctx, ctx->b_q, slice * (iters + 1))) != CONVCRF_OK) return st;
    if (run) {
        // dL/dQ^t ping-pong at full resolution (with blur it stays pooled)
        if (s == 1 && (st = ensure(ctx, ctx->b_dq, slice * 2)) != CONVCRF_OK) return st;
        if ((st = ensure(ctx, ctx->b_dm, slice)) != CONVCRF_OK) return st;
        if (grad_compat && !potts_dz)
            if ((st = ensure(ctx, ctx->b_dp, slice)) != CONVCRF_OK) return st;
        if (grad_compat)
            if ((st = ensure(ctx, ctx->b_gpart, sizeof(float) * (size_t)ntiles * C * C)) !=
                CONVCRF_OK)
                return st;
        if ((st = ensure(ctx, ctx->b_kpart, sizeof(float) * (size_t)ntiles * groups * 5)) !=
            CONVCRF_OK)
            return st;
        // dL/dF on the grid of the message (with blur, of the pooled features:
        // always a workspace buffer, the pooling's transpose writes grad_features)
        if (p.features && (!grad_features || s > 1) &&
            (st = ensure(ctx, ctx->b_df, sizeof(float) * (size_t)npg * D)) != CONVCRF_OK)
            return st;
        if (p.features && groups > 1 &&
            (st = ensure(ctx, ctx->b_dfp, sizeof(float) * (size_t)npg * D * groups)) !=
                CONVCRF_OK)
            return st;
        if (s > 1) {
            // pooled image, pooled Q^t for every round, pooled message, and
            // the pooled dL/dM, -dL/dZ and dL/dQ
            const size_t pb = sizeof(float) * (size_t)B * Hg * Wg;
            const size_t fcol = ((size_t)B * 3 * Hg * Wg + 63) / 64 * 64;
            if ((st = ensure(ctx, ctx->pool_f, sizeof(float) * fcol + pb * D)) != CONVCRF_OK)
                return st;
            if ((st = ensure(ctx, ctx->pool_q, pb * C * std::max(iters, 1))) != CONVCRF_OK)
                return st;
            if ((st = ensure(ctx, ctx->pool_m, pb * C)) != CONVCRF_OK) return st;
            if ((st = ensure(ctx, ctx->b_pd, pb * C * 3)) != CONVCRF_OK) return st;
        }
    }
    char* qbase = static_cast<char*>(ctx->b_q.p);
    auto qs = [&](int t) { return reinterpret_cast<float*>(qbase + slice * t); };

    float* pf = static_cast<float*>(ctx->pool_f.p);
    // blur with learnable features: the pooled features follow the pooled colours
    float* psf = s > 1 && D > 0 ? pf + ((size_t)B * 3 * Hg * Wg + 63) / 64 * 64 : nullptr;
    // pooled Q^t of round t (blur)
    auto pqs = [&](int t) {
        return static_cast<float*>(ctx->pool_q.p) + (size_t)t * B * C * Hg * Wg;
    };
    float* pm = static_cast<float*>(ctx->pool_m.p);
    // 4 x 4 pooling: the recompute takes the fused form of convcrf_meanfield
    // (one initialisation launch, then one fused round per iteration, each
    // writing Q^{t+1} and its pooled form)
    const auto al8 = [](const void* ptr) { return reinterpret_cast<uintptr_t>(ptr) % 8 == 0; };
    const bool fused_blur =
        run && s == kFusedBlurFactor && k >= 3 && B <= 65535 && D <= kMaxFeat && al8(unary) &&
        al8(image) && (D == 0 || al8(p.features)) && al8(qs(0)) &&
        (Hg + kBlurInitTY - 1) / kBlurInitTY <= 65535 &&
        blur_iter_lds_bytes(k, C == 19 || C == 21 ? C : (C <= 8 ? 8 : 24), mu_dev != nullptr,
                            D > 0 ? kMaxFeat : 0) <= kLdsLimit;

    // forward: Q^0 = softmax(U), then the rounds, keeping every Q^t
    if (fused_blur) {
        BlurInitArgs bin{};
        bin.unary = unary;
        bin.image = image;
        bin.q_full = qs(0);
        bin.qbar = pqs(0);
        bin.pcol = pf;
        bin.B = B;
        bin.C = C;
        bin.H = H;
        bin.W = W;
        bin.Hp = Hg;
        bin.Wp = Wg;
        bin.feat = D > 0 ? p.features : nullptr;
        bin.pfeat = psf;
        bin.D = D;
        st = launch(ctx, kPool, stream, "blur_pool", [&] { return launch_blur_init(bin, stream); });
    } else {
        st = launch(ctx, kSoftmax, stream, "softmax",
                    [&] { return launch_softmax(unary, qs(0), B, C, H * W, stream); });
    }
    if (st != CONVCRF_OK) return st;
    if (run && s > 1) {
        // the pooled message of Sec. 4.2 (as convcrf_meanfield), with every
        // Q^t kept at full resolution
        IterArgs a{};
        a.mu = mu_dev;
        a.include_center = p.include_center;
        a.neg_beta = (float)(-kLog2eD / (2.0 * tb * tb));
        a.center_w = (float)((double)p.w_app + (double)p.w_smooth);
        fill_taps(p, s, a.taps);
        const int nchunks = (C + kPmsgClasses - 1) / kPmsgClasses;
        const size_t lds = pmsg_lds_bytes(k, D);
        if (lds > kLdsLimit) return fail(ctx, CONVCRF_E_UNSUPPORTED, "window exceeds LDS");
        a.sfeat = psf;
        a.D = D;
        a.w_smooth = p.w_smooth;
        a.neg_gamma = (float)(-kLog2eD / (2.0 * tg * tg));
        a.C = (C + nchunks - 1) / nchunks;
        a.planes = C;
        a.H = Hg;
        a.W = Wg;
        a.feat = pf;
        a.dst = pm;
        a.mode = kModeMessage;
        a.tiles_x = (Wg + kPmsgTW - 1) / kPmsgTW;
        a.tiles_per_img = a.tiles_x * ((Hg + kPmsgTH - 1) / kPmsgTH);
        a.ntiles = a.tiles_per_img * B;
        if (!fused_blur) {
            st = launch(ctx, kPool, stream, "blur_pool",
                        [&] { return launch_pool(image, pf, B, 3, H, W, s, 0, stream); });
            if (st != CONVCRF_OK) return st;
            if (D > 0) {
                st = launch(ctx, kPool, stream, "blur_pool", [&] {
                    return launch_pool(p.features, psf, B, D, H, W, s, 0, stream);
                });
                if (st != CONVCRF_OK) return st;
            }
            // Q^0 pooled here; every update also writes its pooled Q^{t+1},
            // kept for the reverse rounds
            st = launch(ctx, kPool, stream, "blur_pool",
                        [&] { return launch_pool(qs(0), pqs(0), B, C, H, W, s, 0, stream); });
            if (st != CONVCRF_OK) return st;
        }
        if (fused_blur) {
            BlurIterArgs bi{};
            bi.pcol = pf;
            bi.unary = unary;
            bi.mu = mu_dev;
            bi.B = B;
            bi.C = C;
            bi.H = H;
            bi.W = W;
            bi.Hp = Hg;
            bi.Wp = Wg;
            bi.include_center = p.include_center;
            bi.center_w = a.center_w;
            bi.neg_beta = a.neg_beta;
            bi.taps = a.taps;
            bi.sfeat = psf;
            bi.D = D;
            bi.w_smooth = p.w_smooth;
            bi.neg_gamma = a.neg_gamma;
            for (int t = 0; t < iters; ++t) {
                bi.qbar = pqs(t);
                bi.q_full = qs(t + 1);
                bi.qbar_out = t + 1 < iters ? pqs(t + 1) : nullptr;
                st = launch(ctx, kBlurIter, stream, "blur_iteration",
                            [&] { return launch_blur_iter(bi, k, stream); });
                if (st != CONVCRF_OK) return st;
            }
        } else {
            for (int t = 0; t < iters; ++t) {
                a.src = pqs(t);
                st = launch(ctx, kBlurMsg, stream, "blur_message",
                            [&] { return launch_pmsg(a, k, nchunks, lds, stream); });
                if (st != CONVCRF_OK) return st;
                st = launch(ctx, kBlurUpd, stream, "blur_update", [&] {
                    return launch_blur_update(pm, unary, mu_dev, qs(t + 1),
                                              t + 1 < iters ? pqs(t + 1) : nullptr, B, C, H, W,
                                              s, stream);
                });
                if (st != CONVCRF_OK) return st;
            }
        }
    } else if (run && p.features) {
        FeatArgs f = feat_args(p, unary, image, mu_dev, B, C, H, W);
        IterArgs ar{};
        const bool ring = plan_feature_ring(ar, p, unary, image, mu_dev, B, C, H, W, {qbase});
        for (int t = 0; t < iters; ++t) {
            f.src = ar.src = qs(t);
            f.dst = ar.dst = qs(t + 1);
            st = launch(ctx, kFeatIter, stream, "feature_iter", [&] {
                return ring ? launch_ring(ar, k, stream) : launch_feat_update(f, k, stream);
            });
            if (st != CONVCRF_OK) return st;
        }
    } else if (run) {
        IterArgs a{};
        a.mu = mu_dev;
        a.include_center = p.include_center;
        a.neg_beta = (float)(-kLog2eD / (2.0 * tb * tb));
        a.center_w = (float)((double)p.w_app + (double)p.w_smooth);
        fill_taps(p, 1, a.taps);
        const TileConfig tile = pick_tile(k, C, true, mu_dev != nullptr);
        if (tile.rows == 0) return fail(ctx, CONVCRF_E_UNSUPPORTED, "window and classes exceed LDS");
        const size_t lds = iter_lds_bytes(k, C, tile, true, mu_dev != nullptr);
        IterArgs as, ar;
        bool streamed = false, ring = false;
        size_t lds_s = 0;
        plan_unpooled(a, as, ar, streamed, ring, lds_s, tile, false, k, B, C, H, W, unary, image,
                      nullptr, {qbase});
        for (int t = 0; t < iters; ++t) {
            a.src = as.src = ar.src = t == 0 ? unary : qs(t);
            a.dst = as.dst = ar.dst = qs(t + 1);
            a.first = as.first = ar.first = t == 0;
            st = launch(ctx, t == 0 ? kFusedFirst : kFused, stream, "fused_iter", [&] {
                if (ring && t > 0) return launch_ring(ar, k, stream);
                return streamed ? launch_stream(as, k, lds_s, stream)
                                : launch_iter(a, k, false, tile, lds, stream);
            });
            if (st != CONVCRF_OK) return st;
        }
    }

    // reverse rounds
    BwdArgs ba{};
    ba.feat = s > 1 ? pf : image;
    ba.C = C;
    ba.H = Hg;
    ba.W = Wg;
    ba.tiles_x = (Wg + tw - 1) / tw;
    ba.tiles_per_img = ba.tiles_x * ((Hg + th - 1) / th);
    ba.ntiles = ntiles;
    ba.include_center = p.include_center;
    ba.cgroups = groups;
    ba.cgsize = cgsize;
    ba.dma = dma;
    ba.neg_beta = (float)(-kLog2eD / (2.0 * tb * tb));
    ba.w_app = p.w_app;
    ba.w_smooth = p.w_smooth;
    for (int n = 0; n <= kMaxN; ++n) {
        ba.a_log2[n] = (float)(-s2 * n * kLog2eD / (2.0 * ta * ta));
        ba.smooth[n] = (float)std::exp(-s2 * n / (2.0 * tg * tg));
    }
    ba.dm = static_cast<const float*>(ctx->b_dm.p);
    ba.kpart = static_cast<float*>(ctx->b_kpart.p);
    // dL/dF lands on the message's grid: grad_features itself without blur,
    // the pooled derivative in the workspace with it
    float* const df_grid = grad_features && s == 1 ? grad_features : static_cast<float*>(ctx->b_df.p);
    if (p.features) {
        ba.sfeat = s > 1 ? psf : p.features;
        ba.dfeat = df_grid;
        if (groups > 1) {
            // each class group stores its part of dL/dF; a sum adds them
            ba.dfeat = static_cast<float*>(ctx->b_dfp.p);
            ba.dfeat_gstride = npg * D;
        }
        ba.D = D;
        ba.neg_gamma = (float)(-kLog2eD / (2.0 * tg * tg));
        ba.inv_gamma2 = (float)(1.0 / (tg * tg));
    }
    // Potts (C > 1): the compatibility derivative takes -dL/dZ from dL/dM,
    // so dL/dZ is neither written nor upsampled
    float* dp = grad_compat && !potts_dz ? static_cast<float*>(ctx->b_dp.p) : nullptr;
    ba.dm_sum_scale = grad_compat && potts_dz ? (float)(1.0 / (1.0 - (double)C)) : 0.f;
    ba.gpart = grad_compat ? static_cast<float*>(ctx->b_gpart.p) : nullptr;
    float* dm = static_cast<float*>(ctx->b_dm.p);
    // blur: the pooled dL/dM, -dL/dZ and dL/dQ
    const size_t pn = (size_t)B * C * Hg * Wg;
    float* pdm = static_cast<float*>(ctx->b_pd.p);
    float* pdp = pdm ? pdm + pn : nullptr;
    float* pdq = pdm ? pdm + 2 * pn : nullptr;
    ba.dp = s > 1 ? (dp ? pdp : nullptr) : dp;
    // dL/dQ^{t+1}: grad_q for the last round; with blur, the pooled adjoint of
    // the round after (dq_s = s), read in place through the pooling's transpose
    const float* dq = grad_q;
    int dq_s = 1;
    for (int t = iters - 1; t >= 0; --t) {
        const int acc = t != iters - 1;
        st = launch(ctx, kBwdPoint, stream, "bwd_point", [&] {
            return launch_bwd_point(qs(t + 1), dq, mu_dev, grad_unary, dm, dp, B, C,
                                    (long long)H * W, acc, stream, W, dq_s);
        });
        if (st != CONVCRF_OK) return st;
        float* dq_next = nullptr;
        ba.accumulate = acc;
        if (s == 1) {
            dq_next = reinterpret_cast<float*>(static_cast<char*>(ctx->b_dq.p) + slice * (t & 1));
            ba.q = qs(t);
            ba.dq_out = dq_next;
            st = launch(ctx, kBwdMsg, stream, "bwd_message",
                        [&] { return launch_bwd_message(ba, k, stream); });
            if (st != CONVCRF_OK) return st;
            if (ba.dfeat_gstride > 0) {
                st = launch(ctx, kBwdReduce, stream, "bwd_reduce", [&] {
                    return launch_group_sum(ba.dfeat, groups, npg * D, df_grid, acc, stream);
                });
                if (st != CONVCRF_OK) return st;
            }
        } else {
            // M = upsample(pooled message of avgpool(Q^t)): the transpose of
            // the upsampling (for dL/dM and, for dL/dmu, -dL/dZ), then the
            // pooled adjoint message; the pooling's transpose is applied by
            // the next bwd_point as it reads dL/dQ^t
            st = launch(ctx, kBwdBlurT, stream, "bwd_blur_transpose", [&] {
                return launch_upsample_t(dm, pdm, B, C, Hg, Wg, s, stream);
            });
            if (st != CONVCRF_OK) return st;
            if (dp) {
                st = launch(ctx, kBwdBlurT, stream, "bwd_blur_transpose", [&] {
                    return launch_upsample_t(dp, pdp, B, C, Hg, Wg, s, stream);
                });
                if (st != CONVCRF_OK) return st;
            }
            ba.q = pqs(t);
            ba.dm = pdm;
            ba.dq_out = pdq;
            st = launch(ctx, kBwdMsg, stream, "bwd_message",
                        [&] { return launch_bwd_message(ba, k, stream); });
            if (st != CONVCRF_OK) return st;
            if (ba.dfeat_gstride > 0) {
                st = launch(ctx, kBwdReduce, stream, "bwd_reduce", [&] {
                    return launch_group_sum(ba.dfeat, groups, npg * D, df_grid, acc, stream);
                });
                if (st != CONVCRF_OK) return st;
            }
            dq_next = pdq;
            dq_s = s;
        }
        dq = dq_next;
    }
    if (p.features && grad_features && run && s > 1) {
        // dL/dF: the transpose of the features' pooling (each pixel gets its
        // cell's derivative / s^2)
        st = launch(ctx, kBwdBlurT, stream, "bwd_blur_transpose", [&] {
            return launch_pool_t(df_grid, grad_features, B, D, Hg, Wg, s, stream);
        });
        if (st != CONVCRF_OK) return st;
    }
    if (p.features && grad_features && !run) {
        // T = 0: Q = softmax(U) does not depend on the features
        for (long long off = 0; off < npix * D; off += 1LL << 30) {
            const int n = (int)std::min<long long>(1LL << 30, npix * D - off);
            st = launch(ctx, kSyncReset, stream, "sync_reset", [&] {
                return launch_zero_u32(reinterpret_cast<unsigned int*>(grad_features + off), n,
                                       stream);
            });
            if (st != CONVCRF_OK) return st;
        }
    }
    // Q^0 = softmax(U)
    st = launch(ctx, kBwdPoint, stream, "bwd_point", [&] {
        return launch_bwd_point(qs(0), dq, nullptr, grad_unary, nullptr, nullptr, B, C,
                                (long long)H * W, iters > 0, stream, W, dq_s);
    });
    if (st != CONVCRF_OK) return st;
    if (grad_compat || grad_kernel)
        return launch(ctx, kBwdReduce, stream, "bwd_reduce", [&] {
            return launch_bwd_reduce(static_cast<const float*>(ctx->b_gpart.p), run ? ntiles : 0,
                                     C, grad_compat, static_cast<const float*>(ctx->b_kpart.p),
                                     run ? ntiles * groups : 0, scale, grad_kernel, stream);
        });
    return CONVCRF_OK;
}

}  // extern "C"
