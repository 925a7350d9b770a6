// features.hip -- one mean-field update with learnable smoothness features
// (the "+T" variant of Sec. 4.2: the inputs of the smoothness Gaussian of
// Eq. 4 are a learnable per-pixel map F instead of the pixel positions).
//
//   K(p, q) = w_app exp(-|p-q|^2 / 2 theta_alpha^2 - |I_p-I_q|^2 / 2 theta_beta^2)
//           + w_smooth exp(-|F_p-F_q|^2 / 2 theta_gamma^2)
//   M_p = sum_{q in W(p)} K(p, q) Q_q       (Eq. 6 / Alg. 1 message)
//   Q'_p = softmax(U_p - mu M_p)            (Alg. 1 compatibility, unary,
//                                            normalisation)
//
// 32 x 8 tiles, one pixel per thread; the colours, the D feature planes and
// the C planes of Q_t are staged with their halo in LDS (zero outside the
// image, so that taps there contribute nothing).  Both Gaussians are
// evaluated per pixel and tap.
#include "crf_internal.h"

namespace convcrf {
namespace {

template <int K, int CM>
__global__ __launch_bounds__(kFeatTW * kFeatTH) void feat_update_kernel(FeatArgs a) {
    constexpr int TW = kFeatTW, TH = kFeatTH, NT = TW * TH;
    constexpr int R = (K - 1) / 2, LW = TW + K - 1, PL = LW * (TH + K - 1);
    extern __shared__ float lds[];
    const int C = a.C, D = a.D;
    const float* sc = lds;                 // 3 colour planes
    const float* sf = lds + 3 * PL;        // D feature planes
    const float* sq = sf + D * PL;         // C planes of Q_t
    const int tile = blockIdx.x;
    const int b = tile / a.tiles_per_img;
    const int tr = tile - b * a.tiles_per_img;
    const int ty = tr / a.tiles_x, tx = tr - ty * a.tiles_x;
    const int y0 = ty * TH - R, x0 = tx * TW - R;
    const long long hw = (long long)a.H * a.W;
    const float* ib = a.image + (long long)b * 3 * hw;
    const float* fb = a.feat + (long long)b * D * hw;
    const float* qb = a.src + (long long)b * C * hw;
    const int nplanes = 3 + D + C;
#pragma unroll 16
    for (int e = threadIdx.x; e < nplanes * PL; e += NT) {
        const int pl = e / PL, o = e - pl * PL;
        const int ly = o / LW, lx = o - ly * LW;
        const int gy = y0 + ly, gx = x0 + lx;
        const float* src = pl < 3 ? ib + pl * hw
                                  : (pl < 3 + D ? fb + (pl - 3) * hw : qb + (pl - 3 - D) * hw);
        const bool ok = gy >= 0 && gy < a.H && gx >= 0 && gx < a.W;
        const float v = src[ok ? (long long)gy * a.W + gx : 0];
        lds[e] = ok ? v : 0.f;
    }
    __syncthreads();

    const int lx = threadIdx.x % TW, ly = threadIdx.x / TW;
    const int px = tx * TW + lx, py = ty * TH + ly;
    if (px >= a.W || py >= a.H) return;
    const int oc = (ly + R) * LW + lx + R;
    const float ir = sc[oc], ig = sc[PL + oc], ibl = sc[2 * PL + oc];
    float fo[kMaxFeat];
#pragma unroll
    for (int c = 0; c < kMaxFeat; ++c) fo[c] = c < D ? sf[c * PL + oc] : 0.f;
    float acc[CM];
    int poff[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        poff[c] = (c < C ? c : C - 1) * PL;
        acc[c] = 0.f;
    }
    constexpr int kRowUnroll = K <= 7 ? K : 1;
#pragma unroll 1
    for (int dy = -R; dy <= R; ++dy) {
#pragma unroll kRowUnroll
        for (int dx = -R; dx <= R; ++dx) {
            if (dx == 0 && dy == 0 && !a.include_center) continue;
            const int o = oc + dy * LW + dx;
            const float er = ir - sc[o], eg = ig - sc[PL + o], eb = ibl - sc[2 * PL + o];
            const float cd2 = fmaf(er, er, fmaf(eg, eg, eb * eb));
            float fd2 = 0.f;
#pragma unroll
            for (int c = 0; c < kMaxFeat; ++c) {
                const float t = c < D ? fo[c] - sf[c * PL + o] : 0.f;
                fd2 = fmaf(t, t, fd2);
            }
            const int n = dx * dx + dy * dy;
            const float w = fmaf(a.w_app, exp2f(fmaf(a.neg_beta, cd2, a.a_log2[n])),
                                 a.w_smooth * exp2f(a.neg_gamma * fd2));
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[c] = fmaf(w, sq[poff[c] + o], acc[c]);
        }
    }
    // Z = U - mu M, then softmax.  Potts, mu[l][l'] = [l != l'], gives
    // Z(l) = U(l) - (sum_l' M(l') - M(l)); the sum is the same for every
    // class and the softmax ignores it, so Z(l) = U(l) + M(l) is used (no
    // difference of two large sums)
    const long long pix = (long long)b * C * hw + (long long)py * a.W + px;
    float z[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (c < C) {
            float t;
            if (a.mu) {
                t = 0.f;
#pragma unroll
                for (int lp = 0; lp < CM; ++lp)
                    if (lp < C) t = fmaf(a.mu[c * C + lp], acc[lp], t);
                t = -t;
            } else {
                t = acc[c];
            }
            z[c] = a.unary[pix + c * hw] + t;
        } else {
            z[c] = -INFINITY;
        }
    }
    float mx = z[0];
#pragma unroll
    for (int c = 1; c < CM; ++c) mx = fmaxf(mx, z[c]);
    float den = 0.f;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        z[c] = c < C ? exp2f((z[c] - mx) * 1.4426950408889634f) : 0.f;
        den += z[c];
    }
    const float inv = 1.f / den;
#pragma unroll
    for (int c = 0; c < CM; ++c)
        if (c < C) a.dst[pix + c * hw] = z[c] * inv;
}

template <int K>
hipError_t launch_k(const FeatArgs& a, hipStream_t stream) {
    const size_t lds = feat_lds_bytes(K, a.C, a.D);
    const dim3 grid(a.ntiles), block(kFeatTW * kFeatTH);
    if (a.C <= 8)
        hipLaunchKernelGGL((feat_update_kernel<K, 8>), grid, block, lds, stream, a);
    else
        hipLaunchKernelGGL((feat_update_kernel<K, kMaxC>), grid, block, lds, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_feat_update(const FeatArgs& a, int k, hipStream_t stream) {
    if (a.C < 1 || a.C > kMaxC || a.D < 1 || a.D > kMaxFeat || a.ntiles <= 0)
        return hipErrorInvalidValue;
    if (feat_lds_bytes(k, a.C, a.D) > 160 * 1024) return hipErrorInvalidValue;
    switch (k) {
        case 1: return launch_k<1>(a, stream);
        case 3: return launch_k<3>(a, stream);
        case 5: return launch_k<5>(a, stream);
        case 7: return launch_k<7>(a, stream);
        case 9: return launch_k<9>(a, stream);
        case 11: return launch_k<11>(a, stream);
        case 13: return launch_k<13>(a, stream);
        case 15: return launch_k<15>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace convcrf
