// crf_internal.h -- launch structures and launcher declarations shared by the
// HIP translation units of libconvcrf.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>
#include <utility>

namespace convcrf {

// Largest window side k and class count the kernels are built for.
constexpr int kMaxK = 15;
constexpr int kMaxC = 24;

// Output tile: `width` (32, or 16 for small grids) columns by `rows` rows;
// each thread owns `pix` (2 or 4) horizontally adjacent pixels of one row.
struct TileConfig {
    int rows;       // output rows per work-group
    int pix;        // pixels per thread: 2 or 4
    int width = 32; // output columns per work-group
    int threads() const { return (width / pix) * rows; }
};

// The Eq. 4 kernel split into its per-offset and its per-pixel parts.  Both
// Gaussians depend on the offset d = (dx, dy) only through n = dx^2 + dy^2
// (grid units; a grid step is `step` full-resolution pixels, so
// |d|^2 = step^2 n), which takes few distinct values in a window:
//   app_log2[n] = log2(w_app) - step^2 n log2(e) / (2 theta_alpha^2)
//   smooth[n]   = w_smooth exp(-step^2 n / (2 theta_gamma^2))
// so that K(p, p + d) = exp2(app_log2[n] + neg_beta |I_p - I_{p+d}|^2)
//                       + smooth[n],  neg_beta = -log2(e) / (2 theta_beta^2).
constexpr int kMaxN = 2 * ((kMaxK - 1) / 2) * ((kMaxK - 1) / 2);
struct TapTable {
    float app_log2[kMaxN + 1];
    float smooth[kMaxN + 1];
};

enum IterMode : int {
    kModeUpdate = 0,   // message -> compatibility -> + unary -> softmax -> Q
    kModeMessage = 1,  // message only -> M (pooled message of the blur path)
};

// Arguments of one message-passing launch over a grid of H x W cells.
struct IterArgs {
    const float* src;     // Q_t [B][C][H][W], or U when `first` (softmax
                          // applied while staging)
    const float* unary;   // U [B][C][H][W] (update mode)
    const float* feat;    // colour planes [B][3][H][W] of the same grid
    const float* kmat;    // materialised weights [B][k*k-1][H][W] or null
    const float* mu;      // device C x C row-major compatibility, null = Potts
    float* dst;           // Q_{t+1} (update) or M (message), [B][C][H][W]
    int C, H, W;          // C: classes this launch computes (a chunk of the
                          // image's classes in message mode, grid dim y)
    int planes;           // class planes per image in src / dst / unary
    int tiles_x, tiles_per_img, ntiles;
    int first;            // stage softmax(src) instead of src
    // resident launch (all iterations in one launch, every tile's work-group
    // co-resident): iterations to run, the two exchange buffers [B][C][H][W]
    // for the tiles' border rings, and the synchronisation words
    int iters;
    float* ring[2];
    unsigned int* sync;   // [0] error flag, [1 + tile] rings published by each
                          // tile; all zero before the launch
    int include_center;   // add (w_app + w_smooth) Q_p to the message
    // learnable smoothness features (ring update only): F [B][D][H][W] or
    // null; the smoothness Gaussian is then w_smooth exp2(neg_gamma |F_p -
    // F_q|^2) instead of taps.smooth
    const float* sfeat;
    int D;
    float neg_gamma, w_smooth;
    int mode;             // IterMode
    int vec;              // W % pix == 0 and planes aligned to 4*pix bytes:
                          // each thread loads and stores its pixels as one
                          // vector per plane
    float neg_beta;
    float center_w;
    TapTable taps;
};

// LDS row stride (floats) of a staged tile row: the width + 2r staged
// columns rounded up to a multiple of the per-thread pixel count, so that
// every thread's window row starts on a 4*pix-byte boundary.
constexpr int iter_lds_stride(int k, int pix, int width) {
    return (width + (k - 1) + pix - 1) / pix * pix;
}

// Streamed update (k <= 7): two pixels per thread on tiles of kStreamTW x
// kStreamRows pixels (wide and short, so that each staged row touches few
// partial cache lines); floats of one staged plane, padded to whole 64-float
// rows of LDS loads, and the LDS bytes of a work-group (C + 3 planes, the
// compatibility matrix in whole rows when given, one dummy row of 256 floats
// for padding loads).
constexpr int kStreamTW = 64, kStreamRows = 16;
constexpr int stream_plane(int k) {
    return ((kStreamRows + k - 1) * iter_lds_stride(k, 2, kStreamTW) + 63) / 64 * 64;
}
inline size_t stream_lds_bytes(int k, int C, bool with_compat) {
    return sizeof(float) * ((size_t)(C + 3) * stream_plane(k) +
                            (with_compat ? ((size_t)C * C + 63) / 64 * 64 : 0) + 256);
}

// Ring update (the later iterations, k <= 7, C = 19 or 21): tiles of
// kStreamTW x kRingRows pixels, 256 threads, the class chunks cycled through
// three LDS slots and the unary loaded into registers, so that two
// work-groups share a CU; LDS bytes of a work-group (three slots of CH
// planes, the colours, the compatibility in whole rows when given, one dummy
// row).
constexpr int kRingRows = 8, kRingSlots = 3;
constexpr int ring_plane(int k) {
    return ((kRingRows + k - 1) * iter_lds_stride(k, 2, kStreamTW) + 63) / 64 * 64;
}
// The quad form of the k = 7 ring update (lane pairs on 4-pixel quads)
// reads its staged rows with 16-byte LDS reads, so its row stride is padded
// to a multiple of 4 floats; its plane is the same size as ring_plane(7).
constexpr int kQuadStride = 72;
constexpr int quad_plane() { return ((kRingRows + 6) * kQuadStride + 63) / 64 * 64; }
static_assert(quad_plane() == ring_plane(7), "the quad update shares the ring's LDS plan");
// and the first round's, on the streamed tiles, the same size as stream_plane(7)
constexpr int quad_first_plane() { return ((kStreamRows + 6) * kQuadStride + 63) / 64 * 64; }
static_assert(quad_first_plane() == stream_plane(7), "the quad first round shares the streamed LDS plan");
inline size_t ring_lds_bytes(int k, int C, int CH, bool with_compat, int D = 0) {
    return sizeof(float) * ((size_t)(kRingSlots * CH + 3 + D) * ring_plane(k) +
                            (with_compat ? ((size_t)C * C + 63) / 64 * 64 : 0) + 256);
}

// Pooled message of the blur path: tiles of 16 x 8 cells, one wavefront per
// window row (64 k threads), chunks of at most kPmsgClasses classes; LDS
// bytes of a work-group (the chunk's planes and the colours with their halo,
// and the k row partials of every class and cell).
constexpr int kPmsgClasses = 12, kPmsgTW = 16, kPmsgTH = 8;
inline size_t pmsg_lds_bytes(int k, int D = 0) {
    const int lh = kPmsgTH + k - 1, ls = (kPmsgTW + k - 1 + 1) / 2 * 2;
    return sizeof(float) * ((size_t)(kPmsgClasses + 3 + D) * lh * ls +
                            (size_t)k * kPmsgClasses * kPmsgTW * kPmsgTH);
}

// LDS bytes of one iteration work-group for a k x k window, C classes,
// with or without the three colour planes and the C x C compatibility.
// Floats of the staged planes of one iteration work-group: Q and, unless
// materialised, the three colour planes, tile plus halo.  The C x C
// compatibility matrix, when given, follows them.
inline size_t iter_lds_stage_floats(int k, int C, TileConfig t, bool with_colour) {
    return (size_t)(C + (with_colour ? 3 : 0)) * (t.rows + (k - 1)) *
           iter_lds_stride(k, t.pix, t.width);
}

// LDS bytes of one iteration work-group for a k x k window and C classes.
inline size_t iter_lds_bytes(int k, int C, TileConfig t, bool with_colour, bool with_compat) {
    return sizeof(float) * (iter_lds_stage_floats(k, C, t, with_colour) +
                            (with_compat ? (size_t)C * C : 0));
}

// One launcher per window side k (each compiled in its own object);
// launch_iter runs one update, one work-group per tile (a.ntiles of them).
// launch_resident runs all a.iters iterations in one
// cooperative launch; with probe = true it only reports whether it would
// (hipSuccess) or not (hipErrorNotSupported / hipErrorCooperativeLaunchTooLarge).
// launch_rstream runs all a.iters iterations in one cooperative launch on
// the tiles of launch_stream (the resident variant; probe as above).
// launch_stream runs one update with the staging streamed under the
// computation (k = 3, 5, 7, C = 19 or 21, vector path; the first iteration
// applies softmax(U) in LDS); hipErrorNotSupported when the arguments are
// outside that.
#define CONVCRF_DECLARE_ITER(K)                                              \
    hipError_t launch_iter_k##K(const IterArgs& a, bool materialised,        \
                                TileConfig tile, size_t lds,                 \
                                hipStream_t stream);                         \
    hipError_t launch_stream_k##K(const IterArgs& a, size_t lds,             \
                                  hipStream_t stream);                       \
    hipError_t launch_ring_k##K(const IterArgs& a, hipStream_t stream);      \
    hipError_t launch_pmsg_k##K(const IterArgs& a, int nchunks, size_t lds,  \
                                hipStream_t stream);                         \
    hipError_t launch_rstream_k##K(const IterArgs& a, size_t lds,            \
                                   int num_cus, hipStream_t stream,          \
                                   bool probe);                              \
    hipError_t launch_resident_k##K(const IterArgs& a, TileConfig tile,      \
                                    size_t lds, int num_cus,                 \
                                    hipStream_t stream, bool probe);
CONVCRF_DECLARE_ITER(1)
CONVCRF_DECLARE_ITER(3)
CONVCRF_DECLARE_ITER(5)
CONVCRF_DECLARE_ITER(7)
CONVCRF_DECLARE_ITER(9)
CONVCRF_DECLARE_ITER(11)
CONVCRF_DECLARE_ITER(13)
CONVCRF_DECLARE_ITER(15)
#undef CONVCRF_DECLARE_ITER
// The k = 7 ring update in its quad form (Potts, no centre tap, no features;
// C = 19 or 21); hipErrorNotSupported outside that.
hipError_t launch_quad_k7(const IterArgs& a, hipStream_t stream);
// The first round (softmax(U) staged in LDS) in the same quad layout.
hipError_t launch_quad_first_k7(const IterArgs& a, hipStream_t stream);

// Fill n words with zero (the flags of a resident launch: a kernel, not a
// memset, so that the sequence may be captured in a graph).
hipError_t launch_zero_u32(unsigned int* p, int n, hipStream_t stream);

// A compatibility matrix passed by value (kernel argument), for callers that
// cannot stage it through pinned host memory: copy_compat writes its first n
// values to dst on the device.
struct CompatBlock {
    float v[kMaxC * kMaxC];
};
hipError_t launch_copy_compat(const CompatBlock& blk, int n, float* dst, hipStream_t stream);

// Q = softmax(U) over classes, per pixel (Alg. 1 initialisation).
hipError_t launch_softmax(const float* U, float* Q, int B, int C, int HW,
                          hipStream_t stream);

// Materialised kernel matrix (Eq. 5 merged over both Gaussians): for every
// pixel and every off-centre tap, K(p, p + d), or 0 where p + d lies outside
// the image.  out [B][k*k-1][H][W].
hipError_t launch_build_kernel(const float* image, float* out, int B, int H,
                               int W, int k, float neg_beta,
                               const TapTable& taps, hipStream_t stream);

// Blur path (pooled message).
// s x s average of `nch` planes per image; if `softmax_first`, each pixel's
// C values are replaced by their softmax before averaging.
hipError_t launch_pool(const float* src, float* dst, int B, int nch, int H,
                       int W, int s, int softmax_first, hipStream_t stream);
// Bilinear upsampling of the pooled message M [B][C][H/s][W/s], then
// compatibility, unary and softmax at full resolution.  q_full (if set)
// receives Q [B][C][H][W] and q_pooled (if set) the s x s average of Q,
// [B][C][H/s][W/s].
hipError_t launch_blur_update(const float* m_pooled, const float* unary,
                              const float* mu, float* q_full, float* q_pooled,
                              int B, int C, int H, int W, int s,
                              hipStream_t stream);

// ---- one fused iteration of the blur path for a 4 x 4 pooling: the pooled
// message of a work-group's 8 x 8 cells (and the one-cell ring its pixels'
// bilinear upsampling reads) and the full-resolution update of its 32 x 32
// pixels in one launch (grid ceil(Wp / 8) x ceil(Hp / 8) x B).
constexpr int kFusedBlurFactor = 4, kFusedBlurCells = 8;
constexpr int kFusedBlurRowStride = 28;   // LDS row stride of the staged footprint (floats)
struct BlurIterArgs {
    const float* qbar;    // pooled Q_t [B][C][Hp][Wp]
    const float* pcol;    // pooled colours [B][3][Hp][Wp]
    const float* unary;   // U [B][C][H][W], 8-byte aligned
    const float* mu;      // device C x C compatibility or null (Potts)
    float* qbar_out;      // pooled Q_{t+1}, or null
    float* q_full;        // Q_{t+1} [B][C][H][W] (8-byte aligned), or null (at least one
                          // of the two is given: both for the reverse mode's recompute)
    int B, C, H, W, Hp, Wp;
    int include_center;
    float center_w;       // K(p, p) = w_app + w_smooth when the centre is included
    float neg_beta;       // -log2(e) / (2 theta_beta^2)
    TapTable taps;        // per-offset constants on the pooled grid (step 4)
    const float* sfeat;   // pooled learnable features [B][D][Hp][Wp] (D > 0), else null
    int D;                // feature planes, 0 .. kMaxFeat
    float w_smooth;       // the smoothness weight (features)
    float neg_gamma;      // -log2(e) / (2 theta_gamma^2) (features)
};
// LDS of one work-group: the pooled Q_t and colours over the footprint
// ((8 + 2 + 2r) cells square, rows kFusedBlurRowStride floats apart; with
// learnable features, fd feature planes after the colours), k row
// partials of a chunk of classes over the 10 x 10 message tile (planes of
// kFusedBlurPartStride floats, two spare), the message tile, and the
// compatibility when given.  A chunk's class slots are even (two classes per
// wavefront instruction): the most that fit 160 KB with the rest,
// compatibility included, up to the classes rounded up to even.
constexpr int kFusedBlurPartStride = (kFusedBlurCells + 2) * (kFusedBlurCells + 2) + 2;
constexpr int blur_iter_slots(int k, int CM, int fd = 0) {
    const int fs = kFusedBlurCells + 2 + (k - 1), mt = (kFusedBlurCells + 2) * (kFusedBlurCells + 2);
    const int room = 160 * 1024 / 4 - (CM + 3 + fd) * fs * kFusedBlurRowStride - CM * mt - CM * CM;
    const int cap = room / (k * kFusedBlurPartStride) / 2 * 2, full = (CM + 1) / 2 * 2;
    const int sl = cap < full ? cap : full;
    return sl < 2 ? 2 : sl;
}
constexpr int blur_iter_chunk(int k, int CM, int fd = 0) {
    return blur_iter_slots(k, CM, fd) < CM ? blur_iter_slots(k, CM, fd) : CM;
}
inline size_t blur_iter_lds_bytes(int k, int CM, bool with_compat, int fd = 0) {
    const size_t fs = kFusedBlurCells + 2 + (k - 1), mt = (kFusedBlurCells + 2) * (kFusedBlurCells + 2);
    return sizeof(float) * ((size_t)(CM + 3 + fd) * fs * kFusedBlurRowStride +
                            (size_t)k * blur_iter_slots(k, CM, fd) * kFusedBlurPartStride +
                            (size_t)CM * mt + (with_compat ? (size_t)CM * CM : 0));
}
hipError_t launch_blur_iter(const BlurIterArgs& a, int k, hipStream_t stream);
hipError_t launch_blur_iter_k1(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k3(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k5(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k7(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k9(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k11(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k13(const BlurIterArgs& a, hipStream_t stream);
hipError_t launch_blur_iter_k15(const BlurIterArgs& a, hipStream_t stream);

// ---- initialisation of the fused blur path (4 x 4 pooling): softmax(U),
// the image and the learnable features (if any), averaged over the cells, in
// one launch over tiles of kBlurInitTX x kBlurInitTY cells.
constexpr int kBlurInitTX = 8, kBlurInitTY = 4;
struct BlurInitArgs {
    const float* unary;   // U [B][C][H][W], 8-byte aligned
    const float* image;   // [B][3][H][W], 8-byte aligned
    float* qbar;          // pooled softmax(U) [B][C][Hp][Wp] (out)
    float* pcol;          // pooled colours [B][3][Hp][Wp] (out)
    const float* feat;    // learnable features [B][D][H][W] (8-byte aligned), or null
    float* pfeat;         // pooled features [B][D][Hp][Wp] (out, with feat)
    float* q_full;        // softmax(U) itself [B][C][H][W] (out, 8-byte aligned), or null
    int B, C, H, W, Hp, Wp, D;
};
hipError_t launch_blur_init(const BlurInitArgs& a, hipStream_t stream);

// ---- learnable smoothness features (the "+T" variant): one update with
// the smoothness Gaussian on |F_p - F_q|^2 of a feature map F [B][D][H][W]
// instead of |p - q|^2.  32 x 8 tiles, one pixel per thread.
constexpr int kMaxFeat = 4;
struct FeatArgs {
    const float* src;    // Q_t [B][C][H][W]
    const float* unary;  // U [B][C][H][W]
    const float* image;  // [B][3][H][W]
    const float* feat;   // F [B][D][H][W]
    const float* mu;     // device C x C compatibility or null (Potts)
    float* dst;          // Q_{t+1}
    int C, H, W, D;
    int tiles_x, tiles_per_img, ntiles;
    int include_center;
    int vec4;            // stage 16-byte vectors
    float neg_beta;      // -log2(e) / (2 theta_beta^2)
    float neg_gamma;     // -log2(e) / (2 theta_gamma^2)
    float w_app, w_smooth;
    float a_log2[kMaxN + 1];  // -n log2(e) / (2 theta_alpha^2)
};
// With vec4 (k <= 7, W a multiple of 4, 16-byte aligned planes) the staged
// rows start 4 columns left of the tile and hold kFeatTW + 8 columns.
constexpr int kFeatTW = 32, kFeatTH = 8;
inline size_t feat_lds_bytes(int k, int C, int D, bool vec4 = false) {
    return sizeof(float) * (size_t)(3 + D + C) * (vec4 ? kFeatTW + 8 : kFeatTW + k - 1) *
           (kFeatTH + k - 1);
}
hipError_t launch_feat_update(const FeatArgs& a, int k, hipStream_t stream);

// ---- reverse mode (derivative of the unpooled mean-field)
// Arguments of one adjoint-message launch: for every pixel x of the grid,
//   dq_out_x(l) = sum_d K(x, x+d) dm_{x+d}(l)   (the transpose of the Eq. 6
//                 message, using K(p,q) = K(q,p) and the symmetric window)
// and the tile's sums over its pixels and taps of dk = sum_l dm_x(l) q_{x+d}(l)
// times A, A |d|^2, A |I_x - I_{x+d}|^2, S, S |d|^2, where A and S are the
// two Eq. 4 Gaussians without their weights, added into kpart[tile][group][5]
// (each class group sums its own classes' part of dk: the five sums are
// linear in it);
// with learnable smoothness features the smoothness Gaussian S is taken on
// |F_x - F_{x+d}|^2, the theta_gamma term on that distance, and
//   dfeat_x += sum_d (dk(x, x+d) + dk(x+d, x)) (-w_smooth S / theta_gamma^2)
//              (F_x - F_{x+d}),  dk(x+d, x) = sum_l dm_{x+d}(l) q_x(l)
// (the pair (x, x+d) seen from both ends; K is symmetric);
// when gpart is set, also the forward message M_x(l) = sum_d K(x, x+d)
// q_{x+d}(l) and the tile's sum over its pixels of dp_x(l) M_x(l') (the
// compatibility derivative) for every l and the group's l', added into
// gpart[tile][l * C + l'].  Partial sums are written instead of added when
// `accumulate` is 0.
struct BwdArgs {
    const float* q;      // Q^t [B][C][H][W]
    const float* dm;     // dL/dM^t [B][C][H][W]
    const float* feat;   // image [B][3][H][W]
    const float* dp;     // -dL/dZ^t [B][C][H][W] (read when gpart is set and
                         // dm_sum_scale is 0)
    float dm_sum_scale;  // Potts, C > 1: 1 / (1 - C), and -dL/dZ^t is taken from
                         // dL/dM^t as -(dM(l) + dm_sum_scale sum_l' dM(l')); else 0
    const float* sfeat;  // learnable smoothness features [B][D][H][W] or null
    float* dfeat;        // dL/dF [B][D][H][W] (with sfeat)
    long long dfeat_gstride;  // > 0: class group g stores its part of dL/dF
                              // (not accumulated) at dfeat + g * dfeat_gstride
    int D;
    float neg_gamma;     // -log2(e) / (2 theta_gamma^2) (with sfeat)
    float inv_gamma2;    // 1 / theta_gamma^2 (with sfeat)
    float* dq_out;       // dL/dQ^t [B][C][H][W]
    float* gpart;        // [ntiles][C * C] or null
    float* kpart;        // [ntiles][5]
    int C, H, W;
    int tiles_x, tiles_per_img, ntiles;
    int include_center;
    int accumulate;
    int cgroups;         // class groups: grid dim y; group g takes classes
    int cgsize;          // [g cgsize, min((g + 1) cgsize, C)) (1 group with
                         // learnable features)
    int dma;             // stage with buffer loads into LDS (each image's
                         // planes under 2 GB; see bwd_plane)
    float neg_beta;      // -log2(e) / (2 theta_beta^2)
    float w_app, w_smooth;
    float a_log2[kMaxN + 1];    // -n log2(e) / (2 theta_alpha^2)
    float smooth[kMaxN + 1];    // exp(-n / (2 theta_gamma^2))
};

// Tile of the adjoint message for window side k and C classes, one pixel
// per thread: 32 columns up to k = 7, 16 above; 16 rows where the 2C + 3
// staged planes of tile plus halo fit the 160 KB of LDS, else 8.
// The LDS then holds the staged planes; with the compatibility derivative it
// is reused afterwards for the tile's dp and M, C rounded up to a multiple
// of 3, one row of tile pixels plus one each, and for the partial sums of
// the 3 x 3 blocks (9 per thread).
// Staged with buffer loads into LDS (dma), each plane is padded to whole
// 64-float rows of loads.  160 KB of LDS less 256 bytes for the static
// partial sums.
constexpr int bwd_tile_w(int k) { return k <= 7 ? 32 : 16; }
constexpr int bwd_gram_rows(int C) { return (C + 2) / 3 * 3; }
// Floats between staged rows in LDS.  A half-wavefront (32 lanes) reads one
// row of a 32-pixel tile, but two rows of a 16-pixel one (k > 7); those rows
// are padded to 48 floats, 16 banks apart, so the two fall in disjoint banks
// (26 floats at k = 11 wrapped ten lanes onto the same banks).
constexpr int bwd_row_stride(int k) { return bwd_tile_w(k) == 16 ? 48 : bwd_tile_w(k) + k - 1; }
static_assert(bwd_row_stride(15) >= 16 + 15 - 1, "the padded rows hold the staged columns");
constexpr int bwd_plane(int k, int rows, bool dma) {
    return dma ? (bwd_row_stride(k) * (rows + k - 1) + 63) / 64 * 64
               : bwd_row_stride(k) * (rows + k - 1);
}
// cn: classes of one group (C with one group).
constexpr size_t bwd_lds_bytes(int k, int C, int rows, bool dma, int D, int cn) {
    const size_t stage = (size_t)(2 * cn + 3 + D) * bwd_plane(k, rows, dma);
    const size_t nt = (size_t)bwd_tile_w(k) * rows;
    const size_t gram = (size_t)(bwd_gram_rows(C) + bwd_gram_rows(cn)) * (nt + 1);
    const size_t red = 9 * nt;
    const size_t g = gram > red ? gram : red;
    return sizeof(float) * (stage > g ? stage : g);
}
constexpr size_t kBwdLdsLimit = 160 * 1024 - 256;
// D: learnable smoothness feature planes staged besides (0 without).
// 16 rows only for groups of more than 8 classes: with fewer, four 256-thread
// work-groups per CU wait less at their barriers than two of 512.
constexpr int bwd_tile_h(int k, int C, int D, bool dma, int cn) {
    return k <= 7 && cn > 8 && bwd_lds_bytes(k, C, 16, dma, D, cn) <= kBwdLdsLimit ? 16 : 8;
}
inline size_t bwd_lds_need(int k, int C, int D, bool dma, int cn) {
    return bwd_lds_bytes(k, C, bwd_tile_h(k, C, D, dma, cn), dma, D, cn);
}

hipError_t launch_bwd_message(const BwdArgs& a, int k, hipStream_t stream);
// one per window side k (each compiled in its own object)
hipError_t launch_bwd_msg_k1(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k3(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k5(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k7(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k9(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k11(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k13(const BwdArgs& a, hipStream_t stream);
hipError_t launch_bwd_msg_k15(const BwdArgs& a, hipStream_t stream);

// Softmax, unary and compatibility adjoints of one round, per pixel:
//   dZ = Q (dQ - <Q, dQ>);  du = dZ (+ du when accumulate);
//   dm(l') = -sum_l mu[l][l'] dZ(l) (mu null = Potts) when dm is set;
//   dp = -dZ when dp is set.
// q, dq, du, dm, dp: [B][C][H][W] with HW = H * W pixels per plane.
// s > 1: dq is dL/dQ on the s x s pooled grid [B][C][HW / s^2] of an image
// W pixels wide (s = 2, 4, 8), each pixel taking its cell's value / s^2.
hipError_t launch_bwd_point(const float* q, const float* dq, const float* mu, float* du,
                            float* dm, float* dp, int B, int C, long long HW,
                            int accumulate, hipStream_t stream, int W = 0, int s = 1);

// Blur transposes (the pooled message of Sec. 4.2), [B][C] planes:
// out [Hp][Wp] = the transpose of the bilinear x s upsampling (half-pixel
// centres, edge clamp) of in [Hp s][Wp s]: each cell gathers the values
// interpolated from it, with the same weights;
hipError_t launch_upsample_t(const float* in, float* out, int B, int C, int Hp, int Wp, int s,
                             hipStream_t stream);
// out [Hp s][Wp s] = the transpose of the s x s average pooling of in
// [Hp][Wp]: each pixel receives its cell's value / s^2.
hipError_t launch_pool_t(const float* in, float* out, int B, int C, int Hp, int Wp, int s,
                         hipStream_t stream);

// out_compat[e] = sum_g gpart[g][e] over `groups` rows (C*C entries, when
// out_compat is set);
// out_kernel[j] = scale[j] * sum_t kpart[t][j] (5 entries, when set).
// Sums in double, in a fixed order.
// out[i] = (accumulate ? out[i] : 0) + sum over g < groups of part[g n + i],
// in order of g (the class groups' parts of dL/dF).
hipError_t launch_group_sum(const float* part, int groups, long long n, float* out,
                            int accumulate, hipStream_t stream);
hipError_t launch_bwd_reduce(const float* gpart, int groups, int C, float* out_compat,
                             const float* kpart, int ntiles, const float scale[5],
                             float* out_kernel, hipStream_t stream);

constexpr float kLog2e = 1.4426950408889634f;

// Alg. 1 normalisation in registers: softmax over the first C of CM values,
// maximum subtracted, one hardware exp2 per value.
// Sum over the eight consecutive lanes of a cell (lanes 8g .. 8g + 7),
// complete in lanes 8g + 4 .. 8g + 7: two quad permutations, then the lower
// quad shifted up by four within the 16-lane row (row_shr:4).
__device__ __forceinline__ float cell_sum8(float t) {
    t += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, t), 0xB1, 0xF,
                                                            0xF, false));   // quad_perm [1, 0, 3, 2]
    t += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, t), 0x4E, 0xF,
                                                            0xF, false));   // quad_perm [2, 3, 0, 1]
    return t + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, t),
                                                                     0x114, 0xF, 0xF, false));
}

template <int CM, bool EXACT>
__device__ __forceinline__ void softmax_regs(float (&z)[CM], int C) {
    float m = z[0];
#pragma unroll
    for (int c = 1; c < CM; ++c)
        if (EXACT || c < C) m = fmaxf(m, z[c]);
    const float mb = m * kLog2e;
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (EXACT || c < C) {
            z[c] = __builtin_amdgcn_exp2f(fmaf(z[c], kLog2e, -mb));
            s += z[c];
        }
    }
    const float inv = 1.0f / s;
#pragma unroll
    for (int c = 0; c < CM; ++c) z[c] *= inv;
}

// Block-to-tile order that keeps the tiles of one XCD spatially contiguous.
// Work-groups are dispatched round-robin over the 8 XCDs of the chip, so
// block b runs on XCD b % 8; XCD x receives the contiguous tile range that
// starts at x * (n / 8) + min(x, n % 8).
__device__ __forceinline__ int xcd_tile(int b, int n) {
    const int x = b & 7;
    const int q = n >> 3;
    const int rem = n & 7;
    return x * q + (x < rem ? x : rem) + (b >> 3);
}

}  // namespace convcrf
