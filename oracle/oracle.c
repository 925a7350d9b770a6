/*
 * oracle.c -- plain double-precision CPU reference for ConvCRF mean-field
 * inference (Teichmann & Cipolla, "Convolutional CRFs for Semantic
 * Segmentation", arXiv 1805.04777).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker the GPU library is
 * compared against.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load it.  It shares no code, header, table or
 * constant with the HIP library and includes nothing from it.
 *
 * It is written to be read against the paper, not to be fast:
 *   - every quantity is a double and every exponential is libm exp();
 *   - loops follow the definitions literally (one pixel, one neighbour, one
 *     class at a time); the only concession to speed is an OpenMP split of
 *     the outer pixel loop, which does not change any summation order.
 *
 * Readings of the paper that this file fixes (each also tested):
 *   - inputs are logits U = -psi_u; Q0 = softmax(U)          (Alg. 1, init)
 *   - message M_p(l) = sum over window neighbours q != p of K(p,q) Q_q(l)
 *                                                     (Eq. 6, Alg. 1 message)
 *     window = square (2r+1)x(2r+1), r = (k-1)/2, centred on p, neighbours
 *     outside the image contribute nothing (Sec. 4 locality assumption)
 *   - K(p,q) = w_app exp(-|p-q|^2/2ta^2 - |I_p-I_q|^2/2tb^2)
 *            + w_smooth exp(-|p-q|^2/2tg^2)                     (Eq. 4)
 *     the centre tap (q == p) is excluded unless include_center is set, in
 *     which case it contributes K(p,p) = w_app + w_smooth    (Eq. 2 vs Eq. 6)
 *   - Z_p(l) = U_p(l) - sum_l' mu[l][l'] M_p(l'),  Q = softmax(Z)
 *                        (Alg. 1 compatibility, unary, normalise; Eq. 1-3)
 *     mu == NULL means Potts, mu[l][l'] = [l != l']          (Sec. 3, 4.2)
 *   - learnable smoothness features (the "+T" variant of Sec. 4.2): when a
 *     map F [d][H][W] is given, the smoothness Gaussian takes |F_p - F_q|^2
 *     in place of |p - q|^2 (F initialised to the positions reproduces
 *     Eq. 4); the appearance Gaussian keeps the positions
 *   - blur s > 1: Q and features are s x s average pooled, the message is
 *     taken on the pooled grid (positions = block centres, so pooled offsets
 *     are s times the grid offsets), then bilinearly upsampled with
 *     half-pixel centres and edge clamping before the compatibility step
 *                                                             (Sec. 4.2)
 *   - blur together with learnable smoothness features: the features are
 *     pooled like the colours (s x s block means, once per image) and the
 *     smoothness Gaussian takes the squared distance of the pooled features
 *     of the two cells; features equal to the positions pool to the block
 *     centres, which reproduces the pooled Eq. 4 above
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    int filter_size;      /* k: odd window side */
    int blur;             /* s: 1 = off; else pool factor, must divide H, W */
    int include_center;   /* 0: exclude q == p (Alg. 1); 1: include (Eq. 6) */
    int reserved;
    double w_app, theta_alpha, theta_beta;  /* appearance kernel (Eq. 4) */
    double w_smooth, theta_gamma;           /* smoothness kernel (Eq. 4) */
} oracle_params;

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Eq. 4 with the smoothness Gaussian on its own squared distance smo_d2
 * (the squared position distance, or the squared distance of the learnable
 * features of the "+T" variant). */
static double kernel_eval(double pos_d2, double col_d2, double smo_d2, const oracle_params *p)
{
    double app = p->w_app * exp(-pos_d2 / (2.0 * p->theta_alpha * p->theta_alpha)
                                - col_d2 / (2.0 * p->theta_beta * p->theta_beta));
    double smo = p->w_smooth * exp(-smo_d2 / (2.0 * p->theta_gamma * p->theta_gamma));
    return app + smo;
}

/* Eq. 4: the merged Gaussian kernel as a function of the squared position
 * distance (in full-resolution pixels) and the squared colour distance. */
double oracle_kernel(double pos_d2, double col_d2, const oracle_params *p)
{
    return kernel_eval(pos_d2, col_d2, pos_d2, p);
}

/* Squared distance of the smoothness Gaussian between pixels pi and qi of
 * one image: the feature distance when a map F [d][HW] is given, else the
 * squared position distance pos_d2. */
static double smooth_d2(const double *F, int d, long HW, long pi, long qi, double pos_d2)
{
    if (!F) return pos_d2;
    double acc = 0.0;
    for (int c = 0; c < d; ++c) {
        double t = F[c * HW + pi] - F[c * HW + qi];
        acc += t * t;
    }
    return acc;
}

/* Alg. 1 initialisation and normalisation: softmax over the C classes of one
 * pixel, with the maximum subtracted first.  Class l of the input is z[l*zs],
 * of the output q[l*qs]. */
static void softmax_pixel(const double *z, long zs, double *q, long qs, int C)
{
    double m = z[0];
    for (int l = 1; l < C; ++l)
        if (z[l * zs] > m) m = z[l * zs];
    double sum = 0.0;
    for (int l = 0; l < C; ++l) {
        double e = exp(z[l * zs] - m);
        q[l * qs] = e;
        sum += e;
    }
    for (int l = 0; l < C; ++l) q[l * qs] /= sum;
}

/* Q0 = softmax(U) for one image, layout [C][H][W]. */
void oracle_softmax(const double *U, int C, int H, int W, double *Q)
{
    long HW = (long)H * W;
    for (long i = 0; i < HW; ++i) softmax_pixel(U + i, HW, Q + i, HW, C);
}

/* Eq. 6 / Alg. 1 message passing for one image on an H x W grid.
 * Q, M: [C][H][W]; I: [3][H][W]; F: [d][H][W] smoothness features or NULL.
 * pos_scale multiplies grid offsets to give the position difference in
 * full-resolution pixels (1 without blur, s on the pooled grid).  M is
 * overwritten. */
static void message_f(const double *Q, const double *I, const double *F, int d, int C,
                      int H, int W, const oracle_params *p, double pos_scale, double *M)
{
    const int r = (p->filter_size - 1) / 2;
    const long HW = (long)H * W;
#pragma omp parallel for schedule(static)
    for (int y = 0; y < H; ++y) {
        for (int x = 0; x < W; ++x) {
            const long pi = (long)y * W + x;
            for (int l = 0; l < C; ++l) M[l * HW + pi] = 0.0;
            for (int y2 = y - r; y2 <= y + r; ++y2) {
                if (y2 < 0 || y2 >= H) continue;           /* outside: no term */
                for (int x2 = x - r; x2 <= x + r; ++x2) {
                    if (x2 < 0 || x2 >= W) continue;
                    if (y2 == y && x2 == x && !p->include_center) continue;
                    const long qi = (long)y2 * W + x2;
                    double dy = pos_scale * (y2 - y), dx = pos_scale * (x2 - x);
                    double col = 0.0;
                    for (int ch = 0; ch < 3; ++ch) {
                        double e = I[ch * HW + pi] - I[ch * HW + qi];
                        col += e * e;
                    }
                    double pos = dy * dy + dx * dx;
                    double kq = kernel_eval(pos, col, smooth_d2(F, d, HW, pi, qi, pos), p);
                    for (int l = 0; l < C; ++l) M[l * HW + pi] += kq * Q[l * HW + qi];
                }
            }
        }
    }
}

void oracle_message(const double *Q, const double *I, int C, int H, int W,
                    const oracle_params *p, double pos_scale, double *M)
{
    message_f(Q, I, NULL, 0, C, H, W, p, pos_scale, M);
}

/* Alg. 1 compatibility transform, unary addition and normalisation for
 * `npix` pixels: Z(l) = U(l) - sum_l' mu[l][l'] M(l'), Q = softmax(Z).
 * mu is row-major C x C, or NULL for Potts mu[l][l'] = [l != l']. */
void oracle_update(const double *U, const double *M, const double *mu,
                   int C, long npix, double *Q)
{
#pragma omp parallel
    {
        double *z = (double *)malloc(sizeof(double) * (size_t)C);
#pragma omp for schedule(static)
        for (long i = 0; i < npix; ++i) {
            for (int l = 0; l < C; ++l) {
                double t = 0.0;
                for (int lp = 0; lp < C; ++lp) {
                    double m = mu ? mu[l * C + lp] : (l != lp ? 1.0 : 0.0);
                    t += m * M[lp * npix + i];
                }
                z[l] = U[l * npix + i] - t;
            }
            softmax_pixel(z, 1, Q + i, npix, C);
        }
        free(z);
    }
}

/* s x s average pooling of `nch` planes of H x W into H/s x W/s. */
void oracle_avgpool(const double *X, int nch, int H, int W, int s, double *Y)
{
    const int Hp = H / s, Wp = W / s;
    for (int c = 0; c < nch; ++c)
        for (int Y0 = 0; Y0 < Hp; ++Y0)
            for (int X0 = 0; X0 < Wp; ++X0) {
                double acc = 0.0;
                for (int i = 0; i < s; ++i)
                    for (int j = 0; j < s; ++j)
                        acc += X[((long)c * H + Y0 * s + i) * W + X0 * s + j];
                Y[((long)c * Hp + Y0) * Wp + X0] = acc / (double)(s * s);
            }
}

/* Bilinear upsampling by s of `nch` planes of Hp x Wp, with half-pixel
 * centres: output pixel y samples source coordinate (y + 0.5)/s - 0.5,
 * clamped below at 0; the upper neighbour index is clamped at Hp - 1. */
static void src_coord(int o, int s, int n, int *i0, int *i1, double *f)
{
    double u = ((double)o + 0.5) / (double)s - 0.5;
    if (u < 0.0) u = 0.0;
    int a = (int)floor(u);
    if (a > n - 1) a = n - 1;
    *i0 = a;
    *i1 = a < n - 1 ? a + 1 : n - 1;
    *f = u - (double)a;
}

void oracle_upsample(const double *X, int nch, int Hp, int Wp, int s, double *Y)
{
    const int H = Hp * s, W = Wp * s;
    for (int c = 0; c < nch; ++c)
        for (int y = 0; y < H; ++y) {
            int y0, y1;
            double fy;
            src_coord(y, s, Hp, &y0, &y1, &fy);
            for (int x = 0; x < W; ++x) {
                int x0, x1;
                double fx;
                src_coord(x, s, Wp, &x0, &x1, &fx);
                const double *P = X + (long)c * Hp * Wp;
                double top = (1.0 - fx) * P[y0 * Wp + x0] + fx * P[y0 * Wp + x1];
                double bot = (1.0 - fx) * P[y1 * Wp + x0] + fx * P[y1 * Wp + x1];
                Y[((long)c * H + y) * W + x] = (1.0 - fy) * top + fy * bot;
            }
        }
}

/* Alg. 1 end to end: T rounds of message passing, compatibility transform,
 * unary addition and softmax, starting from softmax(U).  U, Q: [B][C][H][W];
 * I: [B][3][H][W] (RGB on its own 0..255 scale).  Returns 0 on success, -1 on
 * an argument the definition does not cover. */
/* F: learnable smoothness features [B][d][H][W], or NULL for the positions
 * (with blur, pooled to the s x s cells like the colours). */
int oracle_meanfield_f(const double *U, const double *I, const double *F, int d, int B,
                       int C, int H, int W, const oracle_params *p, const double *mu, int T,
                       double *Q)
{
    if (B < 0 || C < 1 || H < 1 || W < 1 || T < 0 || !p) return -1;
    if (p->filter_size < 1 || (p->filter_size & 1) == 0) return -1;
    const int s = p->blur;
    if (s < 1 || H % s || W % s) return -1;
    if (F && d < 1) return -1;
    const long HW = (long)H * W;
    const int Hp = H / s, Wp = W / s;
    const long HWp = (long)Hp * Wp;

    double *Qt = (double *)malloc(sizeof(double) * C * HW);
    double *M = (double *)malloc(sizeof(double) * C * HW);
    double *Qp = s > 1 ? (double *)malloc(sizeof(double) * C * HWp) : NULL;
    double *Mp = s > 1 ? (double *)malloc(sizeof(double) * C * HWp) : NULL;
    double *Ip = s > 1 ? (double *)malloc(sizeof(double) * 3 * HWp) : NULL;
    double *Fp = s > 1 && F ? (double *)malloc(sizeof(double) * d * HWp) : NULL;

    for (int b = 0; b < B; ++b) {
        const double *Ub = U + (long)b * C * HW;
        const double *Ib = I + (long)b * 3 * HW;
        const double *Fb = F ? F + (long)b * d * HW : NULL;
        oracle_softmax(Ub, C, H, W, Qt);
        if (s > 1) oracle_avgpool(Ib, 3, H, W, s, Ip);
        if (Fp) oracle_avgpool(Fb, d, H, W, s, Fp);
        for (int t = 0; t < T; ++t) {
            if (s == 1) {
                message_f(Qt, Ib, Fb, d, C, H, W, p, 1.0, M);
            } else {
                oracle_avgpool(Qt, C, H, W, s, Qp);
                message_f(Qp, Ip, Fp, d, C, Hp, Wp, p, (double)s, Mp);
                oracle_upsample(Mp, C, Hp, Wp, s, M);
            }
            oracle_update(Ub, M, mu, C, HW, Qt);
        }
        memcpy(Q + (long)b * C * HW, Qt, sizeof(double) * C * HW);
    }
    free(Qt);
    free(M);
    free(Qp);
    free(Mp);
    free(Ip);
    free(Fp);
    return 0;
}

int oracle_meanfield(const double *U, const double *I, int B, int C, int H, int W,
                     const oracle_params *p, const double *mu, int T, double *Q)
{
    return oracle_meanfield_f(U, I, NULL, 0, B, C, H, W, p, mu, T, Q);
}

/* ------------------------------------------------------------------------
 * Reverse-mode derivative of oracle_meanfield.
 *
 * The loss is a scalar L whose derivative with respect to the returned Q^T
 * is G.  Every round of Alg. 1 is undone in reverse order, each step being
 * the derivative of the forward step it undoes:
 *   normalise   Q = softmax(Z):  dZ(l) = Q(l) (dQ(l) - sum_l' Q(l') dQ(l'))
 *   unary add   Z = U - P:       dU += dZ,   dP = -dZ
 *   compat      P(l) = sum_l' mu[l][l'] M(l'):
 *                                dM(l') = sum_l mu[l][l'] dP(l)
 *                                dmu[l][l'] += sum_p dP_p(l) M_p(l')
 *   message     M_p(l) = sum_{q in W(p)} K(p,q) Q_q(l)            (Eq. 6):
 *                                dQ_q(l) = sum over p with q in W(p) of
 *                                          K(p,q) dM_p(l)   (the transpose)
 *                                dK(p,q) = sum_l dM_p(l) Q_q(l)
 *   kernel      K of Eq. 4 through its five parameters (w_app, theta_alpha,
 *               theta_beta, w_smooth, theta_gamma), with A, S the two
 *               Gaussians without their weights and D the squared distance
 *               of the smoothness Gaussian (|p-q|^2, or |F_p-F_q|^2):
 *                 dK/dw_app = A,  dK/dtheta_alpha = w_app A |p-q|^2/ta^3,
 *                 dK/dtheta_beta = w_app A |I_p-I_q|^2/tb^3,
 *                 dK/dw_smooth = S,  dK/dtheta_gamma = w_smooth S D/tg^3
 *               and, with learnable features, through F at both ends:
 *                 dK/dF_p = -w_smooth S (F_p - F_q)/tg^2 = -dK/dF_q
 *   initialise  Q0 = softmax(U):  dU += Q0 (dQ0 - <Q0, dQ0>)
 * The forward rounds are recomputed first and every Q^t and M^t is kept.
 * dU [B][C][H][W] is written; dmu (C*C, row-major, the derivative with
 * respect to mu at the given mu, Potts included) and dparams (5 values in
 * the order above) are written when not NULL, summed over the batch.
 * With blur s > 1 the message is the pooled one (the pooled Q^t's message
 * on the pooled grid, bilinearly upsampled), undone as the transpose of the
 * upsampling, the pooled message transposed, and the transpose of the
 * pooling.  Returns 0, or -1 on arguments outside the definition.
 * ------------------------------------------------------------------------ */

/* dK(p,q)/d(parameter) for the five Eq. 4 parameters; smo_d2 is the
 * squared distance of the smoothness Gaussian. */
static void kernel_param_derivs(double pos_d2, double col_d2, double smo_d2,
                                const oracle_params *p, double out[5])
{
    const double ta = p->theta_alpha, tb = p->theta_beta, tg = p->theta_gamma;
    const double A = exp(-pos_d2 / (2.0 * ta * ta) - col_d2 / (2.0 * tb * tb));
    const double S = exp(-smo_d2 / (2.0 * tg * tg));
    out[0] = A;
    out[1] = p->w_app * A * pos_d2 / (ta * ta * ta);
    out[2] = p->w_app * A * col_d2 / (tb * tb * tb);
    out[3] = S;
    out[4] = p->w_smooth * S * smo_d2 / (tg * tg * tg);
}

/* q lies in the message window of p (Eq. 6 / Alg. 1 neighbourhood). */
static int in_window(int py, int px, int qy, int qx, int r, int include_center)
{
    if (qy < py - r || qy > py + r || qx < px - r || qx > px + r) return 0;
    if (qy == py && qx == px && !include_center) return 0;
    return 1;
}

/* Transpose of the Eq. 6 message for one image: dQ_q(l) = sum over the
 * pixels p whose window holds q of K(p,q) dM_p(l). */
static void message_transpose(const double *dM, const double *I, const double *F, int d,
                              int C, int H, int W, const oracle_params *p, double pos_scale,
                              double *dQ)
{
    const int r = (p->filter_size - 1) / 2;
    const long HW = (long)H * W;
#pragma omp parallel for schedule(static)
    for (int qy = 0; qy < H; ++qy) {
        for (int qx = 0; qx < W; ++qx) {
            const long qi = (long)qy * W + qx;
            for (int l = 0; l < C; ++l) dQ[l * HW + qi] = 0.0;
            /* a window of radius r holds q only if its centre p lies within
             * r of q: scan that box, test the window itself */
            for (int py = qy - r; py <= qy + r; ++py) {
                if (py < 0 || py >= H) continue;
                for (int px = qx - r; px <= qx + r; ++px) {
                    if (px < 0 || px >= W) continue;
                    if (!in_window(py, px, qy, qx, r, p->include_center)) continue;
                    const long pi = (long)py * W + px;
                    double col = 0.0;
                    for (int ch = 0; ch < 3; ++ch) {
                        double e = I[ch * HW + pi] - I[ch * HW + qi];
                        col += e * e;
                    }
                    double dy = pos_scale * (py - qy), dx = pos_scale * (px - qx);
                    double pos = dy * dy + dx * dx;
                    double kpq = kernel_eval(pos, col, smooth_d2(F, d, HW, pi, qi, pos), p);
                    for (int l = 0; l < C; ++l) dQ[l * HW + qi] += kpq * dM[l * HW + pi];
                }
            }
        }
    }
}

/* Parameter derivative of one message: sum over p, q in W(p) of
 * dK(p,q) * dK(p,q)/d(parameter), dK(p,q) = sum_l dM_p(l) Q_q(l). */
static void message_param_grad(const double *dM, const double *Q, const double *I,
                               const double *F, int d, int C, int H, int W,
                               const oracle_params *p, double pos_scale, double acc[5])
{
    const int r = (p->filter_size - 1) / 2;
    const long HW = (long)H * W;
    for (int py = 0; py < H; ++py) {
        for (int px = 0; px < W; ++px) {
            const long pi = (long)py * W + px;
            for (int qy = py - r; qy <= py + r; ++qy) {
                if (qy < 0 || qy >= H) continue;
                for (int qx = px - r; qx <= px + r; ++qx) {
                    if (qx < 0 || qx >= W) continue;
                    if (!in_window(py, px, qy, qx, r, p->include_center)) continue;
                    const long qi = (long)qy * W + qx;
                    double col = 0.0;
                    for (int ch = 0; ch < 3; ++ch) {
                        double e = I[ch * HW + pi] - I[ch * HW + qi];
                        col += e * e;
                    }
                    double dy = pos_scale * (qy - py), dx = pos_scale * (qx - px);
                    double pos = dy * dy + dx * dx;
                    double g[5];
                    kernel_param_derivs(pos, col, smooth_d2(F, d, HW, pi, qi, pos), p, g);
                    double dk = 0.0;
                    for (int l = 0; l < C; ++l) dk += dM[l * HW + pi] * Q[l * HW + qi];
                    for (int j = 0; j < 5; ++j) acc[j] += dk * g[j];
                }
            }
        }
    }
}

/* Feature derivative of one message ("+T" variant): for every pixel p and
 * window neighbour q, dk(p,q) = sum_l dM_p(l) Q_q(l) times dK/dF_p is added
 * into dF_p and times dK/dF_q = -dK/dF_p into dF_q. */
static void message_feature_grad(const double *dM, const double *Q, const double *F, int d,
                                 int C, int H, int W, const oracle_params *p, double *dF)
{
    const int r = (p->filter_size - 1) / 2;
    const long HW = (long)H * W;
    const double tg = p->theta_gamma;
    for (int py = 0; py < H; ++py) {
        for (int px = 0; px < W; ++px) {
            const long pi = (long)py * W + px;
            for (int qy = py - r; qy <= py + r; ++qy) {
                if (qy < 0 || qy >= H) continue;
                for (int qx = px - r; qx <= px + r; ++qx) {
                    if (qx < 0 || qx >= W) continue;
                    if (!in_window(py, px, qy, qx, r, p->include_center)) continue;
                    const long qi = (long)qy * W + qx;
                    double dk = 0.0;
                    for (int l = 0; l < C; ++l) dk += dM[l * HW + pi] * Q[l * HW + qi];
                    const double S = exp(-smooth_d2(F, d, HW, pi, qi, 0.0) / (2.0 * tg * tg));
                    for (int c = 0; c < d; ++c) {
                        const double dkdfp = -p->w_smooth * S * (F[c * HW + pi] - F[c * HW + qi])
                                             / (tg * tg);
                        dF[c * HW + pi] += dk * dkdfp;
                        dF[c * HW + qi] -= dk * dkdfp;
                    }
                }
            }
        }
    }
}

/* Transpose of oracle_upsample for `nch` planes: every full-resolution
 * value Y[y][x] is sent back to the (up to four) pooled cells it was
 * interpolated from, with the same weights.  X [nch][Hp][Wp] is overwritten. */
static void upsample_transpose(const double *Y, int nch, int Hp, int Wp, int s, double *X)
{
    const int H = Hp * s, W = Wp * s;
    memset(X, 0, sizeof(double) * (size_t)nch * Hp * Wp);
    for (int c = 0; c < nch; ++c)
        for (int y = 0; y < H; ++y) {
            int y0, y1;
            double fy;
            src_coord(y, s, Hp, &y0, &y1, &fy);
            for (int x = 0; x < W; ++x) {
                int x0, x1;
                double fx;
                src_coord(x, s, Wp, &x0, &x1, &fx);
                const double v = Y[((long)c * H + y) * W + x];
                double *P = X + (long)c * Hp * Wp;
                P[y0 * Wp + x0] += (1.0 - fy) * (1.0 - fx) * v;
                P[y0 * Wp + x1] += (1.0 - fy) * fx * v;
                P[y1 * Wp + x0] += fy * (1.0 - fx) * v;
                P[y1 * Wp + x1] += fy * fx * v;
            }
        }
}

/* Transpose of oracle_avgpool: each full-resolution pixel receives its
 * cell's value divided by s^2.  X [nch][H][W] is overwritten. */
static void avgpool_transpose(const double *Y, int nch, int H, int W, int s, double *X)
{
    const int Hp = H / s, Wp = W / s;
    for (int c = 0; c < nch; ++c)
        for (int y = 0; y < H; ++y)
            for (int x = 0; x < W; ++x)
                X[((long)c * H + y) * W + x] =
                    Y[((long)c * Hp + y / s) * Wp + x / s] / (double)(s * s);
}

/* Derivative of the softmax of one pixel: dz(l) = q(l) (dq(l) - <q, dq>). */
static void softmax_adjoint_pixel(const double *q, const double *dq, long s, double *dz,
                                  long zs, int C)
{
    double dot = 0.0;
    for (int l = 0; l < C; ++l) dot += q[l * s] * dq[l * s];
    for (int l = 0; l < C; ++l) dz[l * zs] = q[l * s] * (dq[l * s] - dot);
}

/* F: learnable smoothness features [B][d][H][W] or NULL; dF (same shape,
 * written when F and dF are given) receives dL/dF. */
int oracle_meanfield_backward_f(const double *U, const double *I, const double *F, int d,
                                int B, int C, int H, int W, const oracle_params *p,
                                const double *mu, int T, const double *G, double *dU,
                                double *dmu, double *dparams, double *dF)
{
    if (B < 0 || C < 1 || H < 1 || W < 1 || T < 0 || !p) return -1;
    if (p->filter_size < 1 || (p->filter_size & 1) == 0) return -1;
    const int s = p->blur;
    if (s < 1 || H % s || W % s) return -1;
    if (C > 64 || (F && d < 1)) return -1;
    const long HW = (long)H * W;
    const long n = (long)C * HW;
    const int Hp = H / s, Wp = W / s;
    const long np = (long)C * Hp * Wp;
    double *Qs = (double *)malloc(sizeof(double) * (size_t)(T + 1) * n);
    double *Ms = (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * n);
    double *dQ = (double *)malloc(sizeof(double) * n);
    double *dQprev = (double *)malloc(sizeof(double) * n);
    double *dP = (double *)malloc(sizeof(double) * n);
    double *dM = (double *)malloc(sizeof(double) * n);
    /* blur: pooled Q^t and message of every round, pooled image, and the
     * pooled derivatives */
    double *Qps = s > 1 ? (double *)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * np) : NULL;
    double *Mp = s > 1 ? (double *)malloc(sizeof(double) * np) : NULL;
    double *Ip = s > 1 ? (double *)malloc(sizeof(double) * 3 * Hp * Wp) : NULL;
    double *dMp = s > 1 ? (double *)malloc(sizeof(double) * np) : NULL;
    double *dQp = s > 1 ? (double *)malloc(sizeof(double) * np) : NULL;
    /* blur with features: the pooled features and their derivative */
    double *Fp = s > 1 && F ? (double *)malloc(sizeof(double) * (size_t)d * Hp * Wp) : NULL;
    double *dFp = s > 1 && F ? (double *)malloc(sizeof(double) * (size_t)d * Hp * Wp) : NULL;
    if (dmu) memset(dmu, 0, sizeof(double) * (size_t)C * C);
    if (dparams) memset(dparams, 0, sizeof(double) * 5);

    for (int b = 0; b < B; ++b) {
        const double *Ub = U + (long)b * n;
        const double *Ib = I + (long)b * 3 * HW;
        const double *Fb = F ? F + (long)b * d * HW : NULL;
        double *dFb = F && dF ? dF + (long)b * d * HW : NULL;
        double *dUb = dU + (long)b * n;
        if (dFb) memset(dFb, 0, sizeof(double) * (size_t)d * HW);
        if (dFp) memset(dFp, 0, sizeof(double) * (size_t)d * Hp * Wp);
        /* forward, keeping every Q^t and M^t (and the pooled Q^t with blur) */
        oracle_softmax(Ub, C, H, W, Qs);
        if (s > 1) oracle_avgpool(Ib, 3, H, W, s, Ip);
        if (Fp) oracle_avgpool(Fb, d, H, W, s, Fp);
        for (int t = 0; t < T; ++t) {
            if (s == 1) {
                message_f(Qs + (long)t * n, Ib, Fb, d, C, H, W, p, 1.0, Ms + (long)t * n);
            } else {
                oracle_avgpool(Qs + (long)t * n, C, H, W, s, Qps + (long)t * np);
                message_f(Qps + (long)t * np, Ip, Fp, d, C, Hp, Wp, p, (double)s, Mp);
                oracle_upsample(Mp, C, Hp, Wp, s, Ms + (long)t * n);
            }
            oracle_update(Ub, Ms + (long)t * n, mu, C, HW, Qs + (long)(t + 1) * n);
        }
        /* reverse */
        memcpy(dQ, G + (long)b * n, sizeof(double) * n);
        memset(dUb, 0, sizeof(double) * n);
        for (int t = T - 1; t >= 0; --t) {
            const double *Qn = Qs + (long)(t + 1) * n;   /* Q^{t+1} */
            const double *Qt = Qs + (long)t * n;         /* Q^t */
            const double *Mt = Ms + (long)t * n;         /* M^t */
            for (long i = 0; i < HW; ++i) {
                double dz[64];
                softmax_adjoint_pixel(Qn + i, dQ + i, HW, dz, 1, C);
                for (int l = 0; l < C; ++l) {
                    dUb[l * HW + i] += dz[l];
                    dP[l * HW + i] = -dz[l];
                }
            }
            for (long i = 0; i < HW; ++i)
                for (int lp = 0; lp < C; ++lp) {
                    double acc = 0.0;
                    for (int l = 0; l < C; ++l) {
                        double m = mu ? mu[l * C + lp] : (l != lp ? 1.0 : 0.0);
                        acc += m * dP[l * HW + i];
                    }
                    dM[lp * HW + i] = acc;
                }
            if (dmu)
                for (int l = 0; l < C; ++l)
                    for (int lp = 0; lp < C; ++lp) {
                        double acc = 0.0;
                        for (long i = 0; i < HW; ++i) acc += dP[l * HW + i] * Mt[lp * HW + i];
                        dmu[l * C + lp] += acc;
                    }
            if (s == 1) {
                if (dparams) message_param_grad(dM, Qt, Ib, Fb, d, C, H, W, p, 1.0, dparams);
                if (dFb) message_feature_grad(dM, Qt, Fb, d, C, H, W, p, dFb);
                message_transpose(dM, Ib, Fb, d, C, H, W, p, 1.0, dQprev);
            } else {
                /* M = upsample(pooled message of avgpool(Q^t)): undo the
                 * upsampling, the pooled message, then the pooling */
                upsample_transpose(dM, C, Hp, Wp, s, dMp);
                if (dparams)
                    message_param_grad(dMp, Qps + (long)t * np, Ip, Fp, d, C, Hp, Wp, p,
                                       (double)s, dparams);
                if (dFb)
                    message_feature_grad(dMp, Qps + (long)t * np, Fp, d, C, Hp, Wp, p, dFp);
                message_transpose(dMp, Ip, Fp, d, C, Hp, Wp, p, (double)s, dQp);
                avgpool_transpose(dQp, C, H, W, s, dQprev);
            }
            memcpy(dQ, dQprev, sizeof(double) * n);
        }
        /* blur: dL/dF is the transpose of the pooling applied to the
         * derivative with respect to the pooled features */
        if (dFb && s > 1) avgpool_transpose(dFp, d, H, W, s, dFb);
        for (long i = 0; i < HW; ++i) {
            double dz[64];
            softmax_adjoint_pixel(Qs + i, dQ + i, HW, dz, 1, C);
            for (int l = 0; l < C; ++l) dUb[l * HW + i] += dz[l];
        }
    }
    free(Qs);
    free(Ms);
    free(dQ);
    free(dQprev);
    free(dP);
    free(dM);
    free(Qps);
    free(Mp);
    free(Ip);
    free(dMp);
    free(dQp);
    free(Fp);
    free(dFp);
    return 0;
}

int oracle_meanfield_backward(const double *U, const double *I, int B, int C, int H, int W,
                              const oracle_params *p, const double *mu, int T,
                              const double *G, double *dU, double *dmu, double *dparams)
{
    return oracle_meanfield_backward_f(U, I, NULL, 0, B, C, H, W, p, mu, T, G, dU, dmu,
                                       dparams, NULL);
}
