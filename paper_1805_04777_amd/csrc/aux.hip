// aux.hip -- the kernels around the fused iteration on gfx950:
//   zero_u32_kernel      clears the synchronisation flags of a resident launch
//   softmax_kernel       Q = softmax(U)                 (Alg. 1 initialisation)
//   build_kernel_kernel  kernel matrix of Eq. 5, merged over both Gaussians
//                        (materialised comparison variant, Sec. 4.1)
//   pool_kernel          s x s average pooling (blur path, Sec. 4.2)
//   blur_update_kernel   bilinear upsampling of the pooled message, then
//                        compatibility, unary and softmax (Alg. 1), writing
//                        Q or its s x s average for the next pooled message
#include "crf_internal.h"

namespace convcrf {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

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
// One thread per pooled cell; `nch` planes (up to CM), optional softmax.
template <int CM, bool EXACT>
__global__ __launch_bounds__(256) void pool_kernel(const float* __restrict__ src,
                                                   float* __restrict__ dst, int B, int nch,
                                                   int H, int W, int s, int softmax_first) {
    const int Hp = H / s, Wp = W / s;
    const long long HWp = (long long)Hp * Wp;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long long)B * HWp) return;
    const int b = (int)(gid / HWp);
    const int pc = (int)(gid - b * HWp);
    const int Y = pc / Wp, X = pc - (pc / Wp) * Wp;
    const size_t HW = (size_t)H * W;
    const float* sp = src + (size_t)b * nch * HW;
    float acc[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) acc[c] = 0.f;
    for (int i = 0; i < s; ++i) {
        for (int j = 0; j < s; ++j) {
            const size_t p = (size_t)(Y * s + i) * W + X * s + j;
            float v[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c) v[c] = (EXACT || c < nch) ? sp[c * HW + p] : 0.f;
            if (softmax_first) softmax_regs<CM, EXACT>(v, nch);
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[c] += v[c];
        }
    }
    const float inv = 1.0f / (float)(s * s);
    float* dp = dst + (size_t)b * nch * HWp + pc;
#pragma unroll
    for (int c = 0; c < CM; ++c)
        if (EXACT || c < nch) dp[c * HWp] = acc[c] * inv;
}

// ------------------------------------------------------------- blur update
// Thread order: (b, Y, X) pooled cell major, (i, j) within the s x s block
// minor, so that the s*s pixels of one pooled cell are adjacent lanes of one
// wavefront (s*s divides 64) and their average is a lane reduction.
__device__ __forceinline__ void src_coord(int o, int s, int n, int& i0, int& i1, float& f) {
    // half-pixel centres: output o samples (o + 0.5) / s - 0.5, clamped at 0
    float u = ((float)o + 0.5f) / (float)s - 0.5f;
    u = fmaxf(u, 0.f);
    int a = (int)u;
    if (a > n - 1) a = n - 1;
    i0 = a;
    i1 = a < n - 1 ? a + 1 : n - 1;
    f = u - (float)a;
}

template <int CM, bool EXACT>
__global__ __launch_bounds__(256) void blur_update_kernel(
    const float* __restrict__ mp, const float* __restrict__ unary, const float* __restrict__ mu,
    float* __restrict__ q_full, float* __restrict__ q_pooled, int B, int C, int H, int W, int s) {
    const int Hp = H / s, Wp = W / s;
    const int ss = s * s;
    const long long HWp = (long long)Hp * Wp;
    const long long n = (long long)B * HWp * ss;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    // every lane of a block group is active or inactive together (ss | 64)
    const bool active = gid < n;
    const long long cell = active ? gid / ss : 0;
    const int within = (int)(gid - cell * ss);
    const int b = (int)(cell / HWp);
    const int pc = (int)(cell - b * HWp);
    const int Y = pc / Wp, X = pc - (pc / Wp) * Wp;
    const int y = Y * s + within / s, x = X * s + (within - (within / s) * s);

    float z[CM];
    if (active) {
        int y0, y1, x0, x1;
        float fy, fx;
        src_coord(y, s, Hp, y0, y1, fy);
        src_coord(x, s, Wp, x0, x1, fx);
        const float* m = mp + (size_t)b * C * HWp;
        const int o00 = y0 * Wp + x0, o01 = y0 * Wp + x1, o10 = y1 * Wp + x0, o11 = y1 * Wp + x1;
        float mv[CM];
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            if (EXACT || c < C) {
                const float* mc = m + (size_t)c * HWp;
                const float top = fmaf(fx, mc[o01] - mc[o00], mc[o00]);
                const float bot = fmaf(fx, mc[o11] - mc[o10], mc[o10]);
                mv[c] = fmaf(fy, bot - top, top);
            } else {
                mv[c] = 0.f;
            }
        }
        if (mu != nullptr) {
#pragma unroll
            for (int l = 0; l < CM; ++l) {
                float t = 0.f;
                if (EXACT || l < C) {
#pragma unroll
                    for (int lp = 0; lp < CM; ++lp)
                        if (EXACT || lp < C) t = fmaf(mu[l * C + lp], mv[lp], t);
                }
                z[l] = -t;
            }
        } else {
#pragma unroll
            for (int l = 0; l < CM; ++l) z[l] = mv[l];
        }
        const size_t HW = (size_t)H * W;
        const float* u = unary + (size_t)b * C * HW + (size_t)y * W + x;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C) z[c] += u[c * HW];
        softmax_regs<CM, EXACT>(z, C);
        if (q_full != nullptr) {
            float* q = q_full + (size_t)b * C * HW + (size_t)y * W + x;
#pragma unroll
            for (int c = 0; c < CM; ++c)
                if (EXACT || c < C) q[c * HW] = z[c];
        }
    }
    if (q_full != nullptr) return;
    // s*s-lane average (lanes of one cell are contiguous and aligned)
    const float inv = 1.0f / (float)ss;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        float v = active ? z[c] : 0.f;
        for (int off = 1; off < ss; off <<= 1) v += __shfl_xor(v, off, 64);
        if (active && within == 0) q_pooled[(size_t)b * C * HWp + (size_t)c * HWp + pc] = v * inv;
    }
}

__global__ __launch_bounds__(256) void zero_u32_kernel(unsigned int* p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = 0u;
}

inline unsigned nblocks(long long n, int bs) { return (unsigned)((n + bs - 1) / bs); }

}  // namespace

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

hipError_t launch_pool(const float* src, float* dst, int B, int nch, int H, int W, int s,
                       int softmax_first, hipStream_t stream) {
    const long long n = (long long)B * (H / s) * (W / s);
    const dim3 grid(nblocks(n, 256)), block(256);
    if (nch == 21) hipLaunchKernelGGL((pool_kernel<21, true>), grid, block, 0, stream, src, dst, B, nch, H, W, s, softmax_first);
    else if (nch == 19) hipLaunchKernelGGL((pool_kernel<19, true>), grid, block, 0, stream, src, dst, B, nch, H, W, s, softmax_first);
    else if (nch == 3) hipLaunchKernelGGL((pool_kernel<3, true>), grid, block, 0, stream, src, dst, B, nch, H, W, s, softmax_first);
    else if (nch <= 8) hipLaunchKernelGGL((pool_kernel<8, false>), grid, block, 0, stream, src, dst, B, nch, H, W, s, softmax_first);
    else hipLaunchKernelGGL((pool_kernel<24, false>), grid, block, 0, stream, src, dst, B, nch, H, W, s, softmax_first);
    return hipGetLastError();
}

hipError_t launch_blur_update(const float* m_pooled, const float* unary, const float* mu,
                              float* q_full, float* q_pooled, int B, int C, int H, int W, int s,
                              hipStream_t stream) {
    const long long n = (long long)B * H * W;
    const dim3 grid(nblocks(n, 256)), block(256);
    if (C == 21) hipLaunchKernelGGL((blur_update_kernel<21, true>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, B, C, H, W, s);
    else if (C == 19) hipLaunchKernelGGL((blur_update_kernel<19, true>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, B, C, H, W, s);
    else if (C <= 8) hipLaunchKernelGGL((blur_update_kernel<8, false>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, B, C, H, W, s);
    else hipLaunchKernelGGL((blur_update_kernel<24, false>), grid, block, 0, stream, m_pooled, unary, mu, q_full, q_pooled, B, C, H, W, s);
    return hipGetLastError();
}

}  // namespace convcrf
