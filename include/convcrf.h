/*
 * convcrf.h -- C ABI of the ConvCRF mean-field library for AMD Instinct
 * MI355X (gfx950).
 *
 * The library computes truncated mean-field inference in a Convolutional CRF
 * (Teichmann & Cipolla, "Convolutional CRFs for Semantic Segmentation",
 * arXiv 1805.04777):
 *
 *   Q0 = softmax(U)                                 (Alg. 1, initialisation)
 *   repeat `iters` times:
 *     M_p(l) = sum_{q in W(p), q != p} K(p,q) Q_q(l)       (Eq. 6, Alg. 1
 *                                                            message passing)
 *     K(p,q) = w_app   exp(-|p-q|^2/2 theta_alpha^2 - |I_p-I_q|^2/2 theta_beta^2)
 *            + w_smooth exp(-|p-q|^2/2 theta_gamma^2)             (Eq. 4)
 *     Z_p(l) = U_p(l) - sum_l' mu[l][l'] M_p(l')     (Alg. 1 compatibility
 *                                                     transform, unary add)
 *     Q_p    = softmax(Z_p)                          (Alg. 1 normalisation)
 *
 * W(p) is the k x k window centred on p (Sec. 4: pixels farther apart are
 * conditionally independent); neighbours outside the image contribute
 * nothing.  U are unary logits (minus the unary energy psi_u of Eq. 2), I the
 * RGB image on its own 0..255 scale, positions are integer pixel coordinates.
 *
 * Conventions of every entry point:
 *   - Tensors are dense, C-contiguous float32 in NCHW order:
 *       unary [B][C][H][W], image [B][3][H][W], q_out [B][C][H][W].
 *     All three are DEVICE pointers on the context's GPU, owned by the
 *     caller; the library never frees or retains them.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued on it and the call returns without waiting; the
 *     caller synchronises before reading q_out.
 *   - Every function returns a status code; nothing throws.  Arguments are
 *     validated before any HIP call, so on an error nothing is enqueued and
 *     q_out is left untouched.  convcrf_last_error() gives a message.
 *   - A context is not thread-safe: use one per host thread.  Concurrent
 *     calls on one context from different streams share its workspace and
 *     must be ordered by the caller.
 */
#ifndef CONVCRF_H
#define CONVCRF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CONVCRF_OK = 0,
    CONVCRF_E_INVALID_ARG = -1,  /* NULL pointer, bad size or parameter */
    CONVCRF_E_UNSUPPORTED = -2,  /* valid by the definition but not built
                                    here (C > 24, k > 15, H or W not a
                                    multiple of the blur factor, ...) */
    CONVCRF_E_NO_DEVICE = -3,    /* no usable gfx950 device */
    CONVCRF_E_HIP = -4,          /* a HIP runtime call failed */
    CONVCRF_E_OOM = -5           /* workspace allocation failed */
} convcrf_status;

/* Which kernels compute the message (all give the same Q up to rounding). */
enum {
    CONVCRF_VARIANT_FUSED = 0,        /* weights recomputed in registers from
                                         LDS-staged colour tiles, one launch
                                         per iteration (default) */
    CONVCRF_VARIANT_MATERIALISED = 1, /* kernel matrix K[B][k*k-1][H][W]
                                         written once per call (Eq. 5), then
                                         read by every iteration */
    CONVCRF_VARIANT_RESIDENT = 2      /* the fused kernel running all
                                         iterations in one launch: each tile
                                         stays in LDS and neighbouring tiles
                                         exchange their border rings between
                                         iterations.  Used for Potts and
                                         k <= 7 when every tile's work-group
                                         fits on the device at once (and
                                         iters >= 2); otherwise the call
                                         runs as CONVCRF_VARIANT_FUSED. */
};

/* Model parameters.  Plain host struct; copied during the call. */
typedef struct {
    int32_t filter_size;    /* k, odd, 1 <= k <= 15 (Sec. 4 filter size;
                               the window is k x k, radius r = (k-1)/2) */
    int32_t blur;           /* s in {1, 2, 4, 8}.  s = 1: off.  s > 1: the
                               pooled message of Sec. 4.2 ("blur"): Q and the
                               features are s x s average pooled (pooled
                               positions = block centres, so a pooled offset d
                               is s*d pixels), the k x k message runs on the
                               pooled grid and is bilinearly upsampled (half-
                               pixel centres, edge clamp) before the
                               compatibility step.  H and W must be multiples
                               of s, H / s and B at most 65535.  Only the
                               fused variant implements it (the resident
                               variant runs it as fused). */
    int32_t include_center; /* 0: the centre tap q == p is excluded (Alg. 1
                               sums over i != j; default).  1: it is included
                               with weight K(p,p) = w_app + w_smooth, the
                               literal reading of Eq. 6. */
    int32_t variant;        /* CONVCRF_VARIANT_* */
    float w_app;            /* w(1) of Eq. 4, >= 0 */
    float theta_alpha;      /* position scale of the appearance kernel, > 0 */
    float theta_beta;       /* colour scale of the appearance kernel, > 0 */
    float w_smooth;         /* w(2) of Eq. 4, any finite value (the
                               smoothness term is added to the weight;
                               Eq. 4 leaves its sign to training) */
    float theta_gamma;      /* position scale of the smoothness kernel, > 0 */
    const float *compat;    /* HOST pointer to C*C floats, row-major
                               mu[l][l'] (the 1x1-convolution compatibility
                               of Sec. 4.2), or NULL for Potts
                               mu[l][l'] = [l != l'] (Sec. 3). */
    const float *features;  /* DEVICE pointer to learnable smoothness
                               features F [B][feature_dim][H][W], or NULL.
                               Given, the smoothness Gaussian of Eq. 4 takes
                               |F_p - F_q|^2 in place of |p - q|^2 (the "+T"
                               variant of Sec. 4.2, whose features start as
                               the pixel positions); the appearance Gaussian
                               keeps the positions.  With blur s > 1 the
                               features are s x s average pooled like the
                               colours and the pooled message takes the
                               distance of the pooled features (position
                               features then pool to the cell centres, the
                               pooled Eq. 4).  The variant field is ignored
                               (weights recomputed per pixel and tap). */
    int32_t feature_dim;    /* D, 1 <= D <= 4, with features */
} convcrf_params;

typedef struct convcrf_ctx convcrf_ctx;

/* Fill *p with the defaults used throughout the paper's experiments (Sec. 5:
 * the DenseCRF hand-crafted kernel): k = 7, no blur, centre excluded, fused,
 * w_app = 10, theta_alpha = 80, theta_beta = 13, w_smooth = 3,
 * theta_gamma = 3, Potts, no learnable features.  Returns
 * CONVCRF_E_INVALID_ARG if p is NULL. */
convcrf_status convcrf_default_params(convcrf_params *p);

/* Check sizes and parameters exactly as convcrf_meanfield does, without a
 * context, a device or any HIP call.  B, C, H, W: batch, classes, height,
 * width.  iters >= 0.  Returns CONVCRF_OK or the status meanfield would. */
convcrf_status convcrf_validate(int B, int C, int H, int W,
                                const convcrf_params *params, int iters);

/* Create a context bound to HIP device `device` (its gfx950 code objects
 * are loaded, no workspace is allocated yet).  *out receives the context,
 * or NULL on failure.  CONVCRF_E_NO_DEVICE if the device does not exist or
 * is not gfx950. */
convcrf_status convcrf_init(convcrf_ctx **out, int device);

/* Release the context and its workspace (waits for the device).  NULL is a
 * no-op. */
void convcrf_destroy(convcrf_ctx *ctx);

/* Mean-field inference (Alg. 1) for `iters` rounds; see the file comment.
 * iters = 0 writes softmax(U).  The context owns a workspace (one extra
 * [B][C][H][W] buffer for the ping-pong of Q, plus pooled buffers for blur
 * or the kernel matrix for the materialised variant); it grows on demand,
 * is reused by later calls, and is freed by convcrf_destroy.  q_out must not
 * overlap unary, image or params->features.  Returns CONVCRF_E_HIP on a
 * launch failure (the message names the HIP error). */
convcrf_status convcrf_meanfield(convcrf_ctx *ctx, const float *unary,
                                 const float *image, int B, int C, int H,
                                 int W, const convcrf_params *params,
                                 int iters, float *q_out, void *stream);

/* convcrf_meanfield for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, kernels and results as convcrf_meanfield (bit for bit), but it
 * calls no hipMalloc, hipFree, hipHostMalloc or other allocating routine:
 * the Q ping-pong buffer, the pooled buffers of the blur path and the
 * compatibility matrix live in a scratch array of 64 MiB per device, part of
 * the library's code object, loaded with it and held until the process
 * ends (its device address is taken by convcrf_init).  The compatibility
 * matrix is handed to a kernel by value, so params->compat may be ordinary
 * host memory.  Limits: the workspace of the call, 256-byte aligned slices
 * of B*C*H*W floats for the ping-pong (iters >= 2 or learnable features),
 * plus with blur s B*(H/s)*(W/s)*(2C+3+D) floats (D learnable feature
 * planes, if any), plus C*C for a given
 * compatibility, must fit in 64 MiB (1 x 21 x 512 x 512 needs 22 MB), else
 * CONVCRF_E_UNSUPPORTED with the size in the message and nothing enqueued;
 * the materialised variant is refused (CONVCRF_E_UNSUPPORTED) and the
 * resident variant runs as CONVCRF_VARIANT_FUSED.  No profiling events are
 * recorded for it.  Every call on a device shares that device's scratch
 * array and leaves its contents behind (nothing in it needs to start at
 * zero): calls that overlap on one GPU -- on different streams, or from
 * different contexts or threads -- race and must be ordered by the caller. */
convcrf_status convcrf_meanfield_noalloc(convcrf_ctx *ctx, const float *unary,
                                         const float *image, int B, int C, int H,
                                         int W, const convcrf_params *params,
                                         int iters, float *q_out, void *stream);

/* Reverse mode: the derivative of a scalar loss L through convcrf_meanfield,
 * for training the CRF by backpropagation through the unrolled
 * mean-field rounds of Alg. 1 (Sec. 1; Sec. 5.3 trains end to end through
 * five rounds).  The learnable parameters are the Eq. 4 weights and scales
 * (Sec. 3) and the compatibility (Sec. 4.2).  Given grad_q = dL/dQ for the
 * Q that convcrf_meanfield returns with the same arguments, it writes
 *   grad_unary  [B][C][H][W]  dL/dU                    (DEVICE, required)
 *   grad_compat [C][C]        dL/dmu[l][l'], the derivative with respect to
 *                             the compatibility at params->compat (at the
 *                             Potts matrix mu[l][l'] = [l != l'] when that is
 *                             NULL), summed over the batch  (DEVICE or NULL)
 *   grad_kernel [5]           dL/d(w_app, theta_alpha, theta_beta, w_smooth,
 *                             theta_gamma) of Eq. 4, summed over the batch
 *                                                         (DEVICE or NULL)
 *   grad_features [B][D][H][W] dL/dF for params->features (DEVICE or NULL;
 *                             ignored without features)
 * Each round of Alg. 1 is undone in reverse order: the softmax adjoint
 * dZ = Q (dQ - <Q, dQ>), dU += dZ, the compatibility transposed, and the
 * message transposed, which is the message itself applied to dL/dM because
 * K(p,q) = K(q,p) and the window is symmetric; the kernel-parameter terms are
 * sum over p and window neighbours q of (sum_l dL/dM_p(l) Q_q(l)) dK(p,q)/d;
 * with blur s the message is the pooled one, undone as the transpose of the
 * bilinear upsampling, the adjoint message on the pooled grid (offsets of s
 * pixels) and the transpose of the average pooling;
 * with learnable features, dK/dF_p = -w_smooth S (F_p - F_q)/theta_gamma^2
 * = -dK/dF_q, gathered per pixel from both ends of every pair (with blur on
 * the pooled features, then sent through the transpose of their pooling).
 * The forward rounds are recomputed inside the call (the unaries, image and
 * params must be those of the forward call); `variant` is ignored.
 * unary, image, grad_q: DEVICE pointers, as for convcrf_meanfield; grad_q
 * [B][C][H][W].  grad_unary must not overlap unary, image or grad_q.
 * The context's workspace grows by (iters + 1) + 1 buffers of [B][C][H][W]
 * floats (Q^0..Q^T, dL/dM), two more for dL/dQ without blur (with blur it
 * stays on the pooled grid), one more (-dL/dZ) with grad_compat and a general
 * compatibility, with blur the pooled Q^t of every round and three pooled
 * adjoint tensors, and per-tile partial sums.
 * Returns CONVCRF_E_UNSUPPORTED when the window and classes exceed the LDS of
 * one work-group (2C + 3 planes of the tile plus halo); otherwise as
 * convcrf_meanfield.  Asynchronous on `stream`. */
convcrf_status convcrf_meanfield_backward(convcrf_ctx *ctx, const float *unary,
                                          const float *image, int B, int C,
                                          int H, int W,
                                          const convcrf_params *params,
                                          int iters, const float *grad_q,
                                          float *grad_unary, float *grad_compat,
                                          float *grad_kernel, float *grad_features,
                                          void *stream);

/* Per-kernel timing with HIP events recorded on the launch stream around
 * every kernel the library enqueues, for measurement.  enable = 1 starts
 * (and clears) the record, 0 stops it.  Off by default. */
convcrf_status convcrf_profile_enable(convcrf_ctx *ctx, int enable);

/* Total elapsed milliseconds and launch count of the kernels named `name`
 * ("fused_iter", "fused_resident", "sync_reset", "softmax", "build_kernel",
 * "materialised_iter", "blur_pool" (the pooled initialisation of the blur
 * path: one launch per call for blur 4, else one per pooled tensor),
 * "blur_message", "blur_update" (one each per blur iteration), "blur_iteration"
 * (the fused pooled message and update of one iteration, used for blur 4
 * instead of those two), and for
 * convcrf_meanfield_backward "bwd_point", "bwd_message", "bwd_reduce",
 * "bwd_blur_transpose" (with blur: the upsampling's transpose, one per reverse
 * round with Potts and two with a general compatibility, and with learnable
 * features one more for dL/dF through the pooling) besides the forward's;
 * "feature_iter" with learnable
 * features, "fused_first") since profiling was enabled.  "fused_resident" is one
 * launch running all iterations of a call (CONVCRF_VARIANT_RESIDENT);
 * "fused_first" the first iteration of a fused call (it reads the unary and
 * applies the initial softmax on the fly) and "fused_iter" each later one.
 * Synchronises on the recorded events.  An unknown or unused name gives
 * 0 ms and 0 launches. */
convcrf_status convcrf_profile_read(convcrf_ctx *ctx, const char *name,
                                    double *total_ms, int64_t *launches);

/* Message describing the last failure on ctx (or of a context-free call if
 * ctx is NULL), or why the last CONVCRF_VARIANT_RESIDENT call on ctx ran one
 * launch per iteration instead.  Never NULL; valid until the next call on
 * the same ctx. */
const char *convcrf_last_error(const convcrf_ctx *ctx);

/* Static name of a status code. */
const char *convcrf_status_string(convcrf_status s);

/* The status name followed by the last detailed message on ctx (or of a
 * context-free call if ctx is NULL), for `status` as returned by a call on
 * ctx; "CONVCRF_OK" for CONVCRF_OK.  Never NULL; valid until the next call
 * of this function on the same host thread. */
const char *convcrf_strerror(const convcrf_ctx *ctx, convcrf_status status);

/* Wait until the work enqueued on `stream` (a hipStream_t as void*, NULL =
 * the null stream) has finished, then report whether a
 * CONVCRF_VARIANT_RESIDENT call on ctx since the last check passed the bound
 * of one of its neighbour waits (CONVCRF_E_HIP; its q_out is then not valid
 * and the flag is cleared).  The resident launch synchronises neighbouring
 * tiles with bounded waits so that it can never hang; a wait that gives up
 * sets a device flag instead.  Every call on ctx also checks, without
 * blocking, a copy of that flag taken after the last resident launch, and
 * returns CONVCRF_E_HIP before enqueuing anything when it is set.  Other
 * failures: CONVCRF_E_HIP with the HIP error. */
convcrf_status convcrf_synchronize(convcrf_ctx *ctx, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* CONVCRF_H */
