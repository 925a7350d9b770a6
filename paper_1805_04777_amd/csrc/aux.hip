// aux.hip -- the kernels around the fused iteration on gfx950:
//   zero_u32_kernel      clears the synchronisation flags of a resident launch
//   copy_compat_kernel   writes a compatibility matrix passed by value
//   softmax_kernel       Q = softmax(U)                 (Alg. 1 initialisation)
//   build_kernel_kernel  kernel matrix of Eq. 5, merged over both Gaussians
//                        (materialised comparison variant, Sec. 4.1)
//   pool_kernel          s x s average pooling (blur path, Sec. 4.2)
//   blur_update_kernel   bilinear upsampling of the pooled message, then
//                        compatibility, unary and softmax (Alg. 1), writing
//                        Q, its s x s average for the next pooled message,
//                        or both (any s; blur_update4_kernel for s = 4, 8)
//   blur_init_kernel     initialisation of the fused blur path (4 x 4):
//                        softmax(U), the image and the features, pooled,
//                        in one launch, and optionally softmax(U) itself
#include "crf_internal.h"

namespace convcrf {
namespace {



// ---------------------------------------------------------------- softmax
template <int CM, bool EXACT>
__global__ __launch_bounds__(256) void softmax_kernel(const float* __restrict__ U,
                                                      float* __restrict__ Q, int B, int C,
                                                      int HW) {
    const long long n = (long long)B * HW;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= n) return;
    const int b = (int)(gid / HW);
    const int p = (int)(gid - (long long)b * HW);
    const size_t base = (size_t)b * C * HW + p;
    float z[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) z[c] = (EXACT || c < C) ? U[base + (size_t)c * HW] : 0.f;
    softmax_regs<CM, EXACT>(z, C);
#pragma unroll
    for (int c = 0; c < CM; ++c)
        if (EXACT || c < C) Q[base + (size_t)c * HW] = z[c];
}

// ----------------------------------------------------------- kernel matrix
// One thread per pixel; writes the k*k-1 off-centre taps, 0 outside the image.
__global__ __launch_bounds__(256) void build_kernel_kernel(const float* __restrict__ image,
                                                           float* __restrict__ out, int B,
                                                           int H, int W, int k, float neg_beta,
                                                           const TapTable taps) {
    const long long HW = (long long)H * W;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long long)B * HW) return;
    const int b = (int)(gid / HW);
    const int p = (int)(gid - b * HW);
    const int y = p / W, x = p - (p / W) * W;
    const float* img = image + (size_t)b * 3 * HW;
    const float r0 = img[p], g0 = img[HW + p], b0 = img[2 * HW + p];
    const int r = (k - 1) / 2;
    const int ctr = r * k + r;
    float* o = out + (size_t)b * (k * k - 1) * HW + p;
    for (int t = 0; t < k * k; ++t) {
        if (t == ctr) continue;
        const int dy = t / k - r, dx = t % k - r;
        const int n = dx * dx + dy * dy;
        const int yy = y + dy, xx = x + dx;
        float w = 0.f;
        if (yy >= 0 && yy < H && xx >= 0 && xx < W) {
            const long long q = (long long)yy * W + xx;
            const float d0 = r0 - img[q], d1 = g0 - img[HW + q], d2 = b0 - img[2 * HW + q];
            const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
            w = __builtin_amdgcn_exp2f(fmaf(col2, neg_beta, taps.app_log2[n])) + taps.smooth[n];
        }
        o[(size_t)(t < ctr ? t : t - 1) * HW] = w;
    }
}

// ------------------------------------------------------------------ pooling
// Blur path layout: one thread per full-resolution pixel; a block covers the
// s rows of one pooled row Y and 64 columns (block = s waves, lanes along x,
// so every load and store is a contiguous row piece).  The s x s average of
// a cell is a sum over its s adjacent lanes (shuffles; W and 64 are
// multiples of s) and then over the block's s waves (LDS).
constexpr int kPoolCols = 64;

// Average of v over the s x s cell of this thread; valid in the threads of
// row 0 whose column is the cell's first (returns true there).
template <int CM, bool EXACT>
__device__ __forceinline__ bool cell_average(float (&v)[CM], int C, int s, float* red) {
    const int l = threadIdx.x % kPoolCols, r = threadIdx.x / kPoolCols;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        for (int off = 1; off < s; off <<= 1) v[c] += __shfl_xor(v[c], off, 64);
    }
    if (l % s == 0) {
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C) red[(r * (kPoolCols / s) + l / s) * CM + c] = v[c];
    }
    __syncthreads();
    if (r != 0 || l % s != 0) return false;
    const float inv = 1.0f / (float)(s * s);
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        float t = 0.f;
        for (int rr = 0; rr < s; ++rr) t += red[(rr * (kPoolCols / s) + l / s) * CM + c];
        v[c] = t * inv;
    }
    return true;
}

// s x s average pooling of nch planes (Sec. 4.2), optionally of softmax(src)
// over the planes.  Grid (ceil(W / 64), H / s, B), block s * 64.
template <int CM, bool EXACT>
__global__ __launch_bounds__(512) void pool_kernel(const float* __restrict__ src,
                                                   float* __restrict__ dst, int nch, int H,
                                                   int W, int s, int softmax_first) {
    __shared__ float red[kPoolCols * CM];
    const int Hp = H / s, Wp = W / s;
    const int Y = blockIdx.y, b = blockIdx.z;
    const int x = blockIdx.x * kPoolCols + threadIdx.x % kPoolCols;
    const int y = Y * s + threadIdx.x / kPoolCols;
    const bool active = x < W;
    const size_t HW = (size_t)H * W;
    const float* sp = src + (size_t)b * nch * HW + (size_t)y * W + (active ? x : W - 1);
    float v[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) v[c] = (EXACT || c < nch) ? sp[c * HW] : 0.f;
    if (softmax_first) softmax_regs<CM, EXACT>(v, nch);
    if (cell_average<CM, EXACT>(v, nch, s, red) && active) {
        const size_t HWp = (size_t)Hp * Wp;
        float* dp = dst + (size_t)b * nch * HWp + (size_t)Y * Wp + x / s;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < nch) dp[c * HWp] = v[c];
    }
}

// ------------------------------------------------------------- blur update
// Half-pixel-centred bilinear source coordinate of output o on a grid of n
// cells of s pixels: o samples (o + 0.5) / s - 0.5, clamped at 0 and n - 1.
__device__ __forceinline__ void src_coord(int o, int s, int n, int& i0, int& i1, float& f) {
    float u = ((float)o + 0.5f) / (float)s - 0.5f;
    u = fmaxf(u, 0.f);
    int a = (int)u;
    if (a > n - 1) a = n - 1;
    i0 = a;
    i1 = a < n - 1 ? a + 1 : n - 1;
    f = u - (float)a;
}

// One blur iteration after the pooled message: bilinear upsampling of the
// message, compatibility, unary and softmax (Alg. 1) per pixel, then the
// full Q, its s x s average for the next pooled message, or both (each
// output is written when its pointer is set).
// Same layout as pool_kernel.
template <int CM, bool EXACT>
__global__ __launch_bounds__(512) void blur_update_kernel(
    const float* __restrict__ mp, const float* __restrict__ unary, const float* __restrict__ mu,
    float* __restrict__ q_full, float* __restrict__ q_pooled, int C, int H, int W, int s) {
    __shared__ float red[kPoolCols * CM];
    const int Hp = H / s, Wp = W / s;
    const int Y = blockIdx.y, b = blockIdx.z;
    const int x = blockIdx.x * kPoolCols + threadIdx.x % kPoolCols;
    const int y = Y * s + threadIdx.x / kPoolCols;
    const bool active = x < W;
    const int xc = active ? x : W - 1;
    const size_t HW = (size_t)H * W, HWp = (size_t)Hp * Wp;
    int x0, x1, y0, y1;
    float fx, fy;
    src_coord(xc, s, Wp, x0, x1, fx);
    src_coord(y, s, Hp, y0, y1, fy);
    const float* m = mp + (size_t)b * C * HWp;
    const int o00 = y0 * Wp + x0, o01 = y0 * Wp + x1, o10 = y1 * Wp + x0, o11 = y1 * Wp + x1;
    const float* u = unary + (size_t)b * C * HW + (size_t)y * W + xc;
    // every load first (the four bilinear taps of each class and the unary),
    // so that they are in flight together rather than one class at a time
    float t00[CM], t01[CM], t10[CM], t11[CM], uv[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        const bool on = EXACT || c < C;
        const float* mc = m + (size_t)(on ? c : 0) * HWp;
        t00[c] = on ? mc[o00] : 0.f;
        t01[c] = on ? mc[o01] : 0.f;
        t10[c] = on ? mc[o10] : 0.f;
        t11[c] = on ? mc[o11] : 0.f;
        uv[c] = on ? u[(size_t)c * HW] : 0.f;
    }
    float z[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        const float top = fmaf(fx, t01[c] - t00[c], t00[c]);
        const float bot = fmaf(fx, t11[c] - t10[c], t10[c]);
        z[c] = fmaf(fy, bot - top, top);
    }
    if (mu != nullptr) {
        float t[CM];
#pragma unroll
        for (int l = 0; l < CM; ++l) {
            t[l] = 0.f;
            if (EXACT || l < C) {
#pragma unroll
                for (int lp = 0; lp < CM; ++lp)
                    if (EXACT || lp < C) t[l] = fmaf(mu[l * C + lp], z[lp], t[l]);
            }
        }
#pragma unroll
        for (int l = 0; l < CM; ++l) z[l] = -t[l];
    }
#pragma unroll
    for (int c = 0; c < CM; ++c) z[c] += uv[c];
    softmax_regs<CM, EXACT>(z, C);
    if (q_full != nullptr) {
        if (active) {
            float* q = q_full + (size_t)b * C * HW + (size_t)y * W + x;
#pragma unroll
            for (int c = 0; c < CM; ++c)
                if (EXACT || c < C) q[c * HW] = z[c];
        }
        if (q_pooled == nullptr) return;          // uniform over the grid
    }
    if (cell_average<CM, EXACT>(z, C, s, red) && active) {
        float* dp = q_pooled + (size_t)b * C * HWp + (size_t)Y * Wp + x / s;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C) dp[c * HWp] = z[c];
    }
}

// ---------------------------------------------- four pixels per thread
// For s = 4 and 8 (W a multiple of 4, 16-byte aligned tensors): a thread
// owns four adjacent pixels of one row, which lie in one pooled cell, so it
// loads and stores float4 row pieces (a quarter of the memory instructions)
// and its bilinear taps come from pooled columns X - 1, X, X + 1 only.  A
// block covers the s rows of one pooled row Y and 256 columns; the cell sum
// is in-thread, over the s / 4 lanes of a cell (shuffles) and over the s
// rows (LDS).
constexpr int kPool4Lanes = 64;

// red holds s * 64 / (s / 4) = 256 cells of CM values.
template <int CM, bool EXACT>
__device__ __forceinline__ bool cell_average4(float (&v)[CM], int C, int s, float* red) {
    const int l = threadIdx.x % kPool4Lanes, r = threadIdx.x / kPool4Lanes;
    const int lpc = s / 4;                         // lanes per cell: 1 or 2
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        if (lpc == 2) v[c] += __shfl_xor(v[c], 1, 64);
    }
    if (l % lpc == 0) {
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C) red[(r * (kPool4Lanes / lpc) + l / lpc) * CM + c] = v[c];
    }
    __syncthreads();
    if (r != 0 || l % lpc != 0) return false;
    const float inv = 1.0f / (float)(s * s);
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        float t = 0.f;
        for (int rr = 0; rr < s; ++rr) t += red[(rr * (kPool4Lanes / lpc) + l / lpc) * CM + c];
        v[c] = t * inv;
    }
    return true;
}

// Grid (ceil(W / 256), H / s, B), block 64 s.
template <int CM, bool EXACT>
__global__ __launch_bounds__(512) void pool4_kernel(const float* __restrict__ src,
                                                    float* __restrict__ dst, int nch, int H,
                                                    int W, int s, int softmax_first) {
    __shared__ float red[4 * kPool4Lanes * CM];   // s rows x 64 / (s / 4) cells
    const int Hp = H / s, Wp = W / s;
    const int Y = blockIdx.y, b = blockIdx.z;
    const int x = (blockIdx.x * kPool4Lanes + threadIdx.x % kPool4Lanes) * 4;
    const int y = Y * s + threadIdx.x / kPool4Lanes;
    const bool active = x < W;
    const size_t HW = (size_t)H * W;
    const float* sp = src + (size_t)b * nch * HW + (size_t)y * W + (active ? x : W - 4);
    float v[4][CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        const float4 t = (EXACT || c < nch) ? *reinterpret_cast<const float4*>(sp + c * HW)
                                            : make_float4(0.f, 0.f, 0.f, 0.f);
        v[0][c] = t.x; v[1][c] = t.y; v[2][c] = t.z; v[3][c] = t.w;
    }
    float a[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) a[c] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        if (softmax_first) softmax_regs<CM, EXACT>(v[j], nch);
#pragma unroll
        for (int c = 0; c < CM; ++c) a[c] += v[j][c];
    }
    if (cell_average4<CM, EXACT>(a, nch, s, red) && active) {
        const size_t HWp = (size_t)Hp * Wp;
        float* dp = dst + (size_t)b * nch * HWp + (size_t)Y * Wp + x / s;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < nch) dp[c * HWp] = a[c];
    }
}

template <int CM, bool EXACT>
__global__ __launch_bounds__(512) void blur_update4_kernel(
    const float* __restrict__ mp, const float* __restrict__ unary, const float* __restrict__ mu,
    float* __restrict__ q_full, float* __restrict__ q_pooled, int C, int H, int W, int s) {
    __shared__ float red[4 * kPool4Lanes * CM];   // s rows x 64 / (s / 4) cells
    const int Hp = H / s, Wp = W / s;
    const int Y = blockIdx.y, b = blockIdx.z;
    const int x = (blockIdx.x * kPool4Lanes + threadIdx.x % kPool4Lanes) * 4;
    const int y = Y * s + threadIdx.x / kPool4Lanes;
    const bool active = x < W;
    const int xc = active ? x : W - 4;
    const int X = xc / s;                          // the cell of all four pixels
    const size_t HW = (size_t)H * W, HWp = (size_t)Hp * Wp;
    int y0, y1;
    float fy;
    src_coord(y, s, Hp, y0, y1, fy);
    const int cm = X > 0 ? X - 1 : 0, cp = X < Wp - 1 ? X + 1 : Wp - 1;
    // per pixel: the horizontal interpolation as weights on the pooled
    // columns (X - 1, X, X + 1) -- its two source columns are among them,
    // and at the clamped ends the two coincide
    float wx[4][3];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        int a0, a1;
        float f;
        src_coord(xc + j, s, Wp, a0, a1, f);
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            const int col = X - 1 + k;
            wx[j][k] = (a0 == col ? 1.f - f : 0.f) + (a1 == col ? f : 0.f);
        }
        if (X == 0) { wx[j][1] += wx[j][0]; wx[j][0] = 0.f; }            // column -1 is column 0
        if (X == Wp - 1) { wx[j][1] += wx[j][2]; wx[j][2] = 0.f; }       // column Wp is Wp - 1
    }
    const float* m = mp + (size_t)b * C * HWp;
    const float* u = unary + (size_t)b * C * HW + (size_t)y * W + xc;
    // logits of the four pixels, built in groups of classes (each group's
    // loads in flight together, registers bounded)
    constexpr int G = 7;
    float z[4][CM];
#pragma unroll
    for (int g0 = 0; g0 < CM; g0 += G) {
        float mv[2][3][G];
        float4 uv[G];
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const int c = g0 + i;
            const bool on = c < CM && (EXACT || c < C);
            const float* mc = m + (size_t)(on ? c : 0) * HWp;
            mv[0][0][i] = on ? mc[y0 * Wp + cm] : 0.f;
            mv[0][1][i] = on ? mc[y0 * Wp + X] : 0.f;
            mv[0][2][i] = on ? mc[y0 * Wp + cp] : 0.f;
            mv[1][0][i] = on ? mc[y1 * Wp + cm] : 0.f;
            mv[1][1][i] = on ? mc[y1 * Wp + X] : 0.f;
            mv[1][2][i] = on ? mc[y1 * Wp + cp] : 0.f;
            uv[i] = on ? *reinterpret_cast<const float4*>(u + (size_t)c * HW)
                       : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const int c = g0 + i;
            if (c >= CM) continue;
            const float ua[4] = {uv[i].x, uv[i].y, uv[i].z, uv[i].w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float top = fmaf(wx[j][2], mv[0][2][i], fmaf(wx[j][1], mv[0][1][i], wx[j][0] * mv[0][0][i]));
                const float bot = fmaf(wx[j][2], mv[1][2][i], fmaf(wx[j][1], mv[1][1][i], wx[j][0] * mv[1][0][i]));
                // Potts: U + M; with a general compatibility the unary
                // is read again after the matvec below
                z[j][c] = fmaf(fy, bot - top, top);
                if (mu == nullptr) z[j][c] += ua[j];
            }
        }
    }
    if (mu != nullptr) {
        // general compatibility: z <- U - mu M, pixel by pixel
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            float t[CM];
#pragma unroll
            for (int l = 0; l < CM; ++l) {
                t[l] = 0.f;
                if (EXACT || l < C) {
#pragma unroll
                    for (int lp = 0; lp < CM; ++lp)
                        if (EXACT || lp < C) t[l] = fmaf(mu[l * C + lp], z[j][lp], t[l]);
                }
            }
#pragma unroll
            for (int l = 0; l < CM; ++l) {
                const bool on = EXACT || l < C;
                z[j][l] = on ? u[(size_t)l * HW + j] - t[l] : 0.f;
            }
        }
    }
    float psum[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) psum[c] = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        softmax_regs<CM, EXACT>(z[j], C);
#pragma unroll
        for (int c = 0; c < CM; ++c) psum[c] += z[j][c];
    }
    if (q_full != nullptr) {
        if (active) {
            float* qd = q_full + (size_t)b * C * HW + (size_t)y * W + x;
#pragma unroll
            for (int c = 0; c < CM; ++c)
                if (EXACT || c < C)
                    *reinterpret_cast<float4*>(qd + (size_t)c * HW) =
                        make_float4(z[0][c], z[1][c], z[2][c], z[3][c]);
        }
        if (q_pooled == nullptr) return;          // uniform over the grid
    }
    if (cell_average4<CM, EXACT>(psum, C, s, red) && active) {
        float* dp = q_pooled + (size_t)b * C * HWp + (size_t)Y * Wp + x / s;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C) dp[c * HWp] = psum[c];
    }
}

// ------------------------------------------- blur initialisation, 4 x 4 cells
// Initialisation of the blur path for a 4 x 4 pooling (Alg. 1, Sec. 4.2):
// Q_0 = softmax(U) per pixel and its 4 x 4 cell averages, and the cell
// averages of the image (the pooled colours of the message's weights) and of
// the learnable features when given, in one launch; optionally Q_0 itself as
// well.  A work-group owns 8 x 4 cells (32 x 16 pixels): eight
// consecutive lanes per cell and two horizontally adjacent pixels per lane,
// so a wavefront reads 128-byte rows of every plane; a cell's sums are taken
// across its eight lanes.
template <int CM, bool EXACT>
__global__ __launch_bounds__(256) void blur_init_kernel(const BlurInitArgs a) {
    constexpr int TX = kBlurInitTX, TY = kBlurInitTY, S4 = kFusedBlurFactor;
    static_assert(TX * TY * 8 == 256, "eight lanes per cell");
    const int C = EXACT ? CM : a.C;
    const int H = a.H, W = a.W, Hp = a.Hp, Wp = a.Wp;
    const int b = blockIdx.z;
    const size_t HW = (size_t)H * W, HWp = (size_t)Hp * Wp;
    const int tid = threadIdx.x, ci = tid >> 3, jj = tid & 7;
    const int ccy = blockIdx.y * TY + ci / TX, ccx = blockIdx.x * TX + ci % TX;   // own cell
    const int py = ccy * S4 + (jj >> 1), px = ccx * S4 + 2 * (jj & 1);
    const bool pix_ok = ccy < Hp && ccx < Wp;                                     // H, W multiples of 4
    // every load is issued (planes past C read plane 0 and are ignored)
    const size_t poff = (size_t)(pix_ok ? py : 0) * W + (pix_ok ? px : 0);
    float z0[CM], z1[CM];
    {
        const float* up = a.unary + (size_t)b * a.C * HW + poff;
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            const float2 t =
                *reinterpret_cast<const float2*>(up + (size_t)(EXACT || c < C ? c : 0) * HW);
            z0[c] = t.x;
            z1[c] = t.y;
        }
    }
    float2 im[3];
    {
        const float* ip = a.image + (size_t)b * 3 * HW + poff;
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) im[ch] = *reinterpret_cast<const float2*>(ip + (size_t)ch * HW);
    }
    softmax_regs<CM, EXACT>(z0, C);
    softmax_regs<CM, EXACT>(z1, C);
    if (a.q_full && pix_ok) {   // Q_0 itself, for the reverse mode's recompute
        float* qf = a.q_full + (size_t)b * a.C * HW + poff;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C)
                *reinterpret_cast<float2*>(qf + (size_t)c * HW) = make_float2(z0[c], z1[c]);
    }
    const size_t cell = (size_t)(pix_ok ? ccy : 0) * Wp + (pix_ok ? ccx : 0);
    constexpr float inv = 1.0f / (S4 * S4);
    float* dq = a.qbar + (size_t)b * a.C * HWp + cell;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        const float t = cell_sum8(z0[c] + z1[c]);
        if (jj == 4 && pix_ok) dq[(size_t)c * HWp] = t * inv;
    }
    float* dc = a.pcol + (size_t)b * 3 * HWp + cell;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        const float t = cell_sum8(im[ch].x + im[ch].y);
        if (jj == 4 && pix_ok) dc[(size_t)ch * HWp] = t * inv;
    }
    if (a.feat) {   // uniform over the grid
        const float* fp = a.feat + (size_t)b * a.D * HW + poff;
        float* df = a.pfeat + (size_t)b * a.D * HWp + cell;
        for (int d = 0; d < a.D; ++d) {
            const float2 v = *reinterpret_cast<const float2*>(fp + (size_t)d * HW);
            const float t = cell_sum8(v.x + v.y);
            if (jj == 4 && pix_ok) df[(size_t)d * HWp] = t * inv;
        }
    }
}

__global__ __launch_bounds__(256) void zero_u32_kernel(unsigned int* p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = 0u;
}

inline unsigned nblocks(long long n, int bs) { return (unsigned)((n + bs - 1) / bs); }

}  // namespace

__global__ __launch_bounds__(256) void copy_compat_kernel(const CompatBlock blk, int n,
                                                          float* dst) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) dst[i] = blk.v[i];
}

hipError_t launch_copy_compat(const CompatBlock& blk, int n, float* dst, hipStream_t stream) {
    if (n < 0 || n > kMaxC * kMaxC) return hipErrorInvalidValue;
    hipLaunchKernelGGL(copy_compat_kernel, dim3(1), dim3(256), 0, stream, blk, n, dst);
    return hipGetLastError();
}

hipError_t launch_zero_u32(unsigned int* p, int n, hipStream_t stream) {
    hipLaunchKernelGGL(zero_u32_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, p, n);
    return hipGetLastError();
}

hipError_t launch_softmax(const float* U, float* Q, int B, int C, int HW, hipStream_t stream) {
    const long long n = (long long)B * HW;
    const dim3 grid(nblocks(n, 256)), block(256);
    if (C == 21) hipLaunchKernelGGL((softmax_kernel<21, true>), grid, block, 0, stream, U, Q, B, C, HW);
    else if (C == 19) hipLaunchKernelGGL((softmax_kernel<19, true>), grid, block, 0, stream, U, Q, B, C, HW);
    else if (C <= 8) hipLaunchKernelGGL((softmax_kernel<8, false>), grid, block, 0, stream, U, Q, B, C, HW);
    else hipLaunchKernelGGL((softmax_kernel<24, false>), grid, block, 0, stream, U, Q, B, C, HW);
    return hipGetLastError();
}

hipError_t launch_build_kernel(const float* image, float* out, int B, int H, int W, int k,
                               float neg_beta, const TapTable& taps, hipStream_t stream) {
    const long long n = (long long)B * H * W;
    hipLaunchKernelGGL(build_kernel_kernel, dim3(nblocks(n, 256)), dim3(256), 0, stream, image, out,
                       B, H, W, k, neg_beta, taps);
    return hipGetLastError();
}

// The four-pixel kernels need s >= 4, W a multiple of 4 and 16-byte aligned
// full-resolution tensors.
inline bool four_ok(int s, int W, const void* a, const void* b) {
    return (s == 4 || s == 8) && W % 4 == 0 && reinterpret_cast<uintptr_t>(a) % 16 == 0 &&
           reinterpret_cast<uintptr_t>(b) % 16 == 0;
}

hipError_t launch_pool(const float* src, float* dst, int B, int nch, int H, int W, int s,
                       int softmax_first, hipStream_t stream) {
    if ((long long)B * H * W == 0) return hipSuccess;
    if (four_ok(s, W, src, src)) {
        const dim3 grid((W + 4 * kPool4Lanes - 1) / (4 * kPool4Lanes), H / s, B), block(kPool4Lanes * s);
        if (nch == 21) hipLaunchKernelGGL((pool4_kernel<21, true>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
        else if (nch == 19) hipLaunchKernelGGL((pool4_kernel<19, true>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
        else if (nch == 3) hipLaunchKernelGGL((pool4_kernel<3, true>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
        else if (nch <= 8) hipLaunchKernelGGL((pool4_kernel<8, false>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
        else hipLaunchKernelGGL((pool4_kernel<24, false>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
        return hipGetLastError();
    }
    const dim3 grid((W + kPoolCols - 1) / kPoolCols, H / s, B), block(kPoolCols * s);
    if (nch == 21) hipLaunchKernelGGL((pool_kernel<21, true>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
    else if (nch == 19) hipLaunchKernelGGL((pool_kernel<19, true>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
    else if (nch == 3) hipLaunchKernelGGL((pool_kernel<3, true>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
    else if (nch <= 8) hipLaunchKernelGGL((pool_kernel<8, false>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
    else hipLaunchKernelGGL((pool_kernel<24, false>), grid, block, 0, stream, src, dst, nch, H, W, s, softmax_first);
    return hipGetLastError();
}

hipError_t launch_blur_update(const float* m_pooled, const float* unary, const float* mu,
                              float* q_full, float* q_pooled, int B, int C, int H, int W, int s,
                              hipStream_t stream) {
    if ((long long)B * H * W == 0) return hipSuccess;
    // (built for 19, 21 and up to 8 classes; other counts hold too many
    // values per thread and take the one-pixel kernel)
    if (four_ok(s, W, unary, q_full ? q_full : unary) && (C == 19 || C == 21 || C <= 8)) {
        const dim3 grid((W + 4 * kPool4Lanes - 1) / (4 * kPool4Lanes), H / s, B), block(kPool4Lanes * s);
        if (C == 21) hipLaunchKernelGGL((blur_update4_kernel<21, true>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
        else if (C == 19) hipLaunchKernelGGL((blur_update4_kernel<19, true>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
        else hipLaunchKernelGGL((blur_update4_kernel<8, false>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
        return hipGetLastError();
    }
    const dim3 grid((W + kPoolCols - 1) / kPoolCols, H / s, B), block(kPoolCols * s);
    if (C == 21) hipLaunchKernelGGL((blur_update_kernel<21, true>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
    else if (C == 19) hipLaunchKernelGGL((blur_update_kernel<19, true>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
    else if (C <= 8) hipLaunchKernelGGL((blur_update_kernel<8, false>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
    else hipLaunchKernelGGL((blur_update_kernel<24, false>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, C, H, W, s);
    return hipGetLastError();
}

hipError_t launch_blur_init(const BlurInitArgs& a, hipStream_t stream) {
    const auto al8 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 8 == 0; };
    if (a.C < 1 || a.C > kMaxC || a.B < 1 || a.B > 65535 || a.Hp < 1 || a.Wp < 1 ||
        a.Hp * kFusedBlurFactor != a.H || a.Wp * kFusedBlurFactor != a.W ||
        (a.Hp + kBlurInitTY - 1) / kBlurInitTY > 65535 || !a.unary || !a.image || !a.qbar ||
        !a.pcol || !al8(a.unary) || !al8(a.image) || a.D < 0 || a.D > kMaxFeat ||
        (a.feat && (!a.pfeat || a.D < 1 || !al8(a.feat))) || (a.q_full && !al8(a.q_full)))
        return hipErrorInvalidValue;
    const dim3 grid((a.Wp + kBlurInitTX - 1) / kBlurInitTX, (a.Hp + kBlurInitTY - 1) / kBlurInitTY,
                    a.B);
    const dim3 block(256);
    if (a.C == 21) hipLaunchKernelGGL((blur_init_kernel<21, true>), grid, block, 0, stream, a);
    else if (a.C == 19) hipLaunchKernelGGL((blur_init_kernel<19, true>), grid, block, 0, stream, a);
    else if (a.C <= 8) hipLaunchKernelGGL((blur_init_kernel<8, false>), grid, block, 0, stream, a);
    else hipLaunchKernelGGL((blur_init_kernel<24, false>), grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace convcrf
