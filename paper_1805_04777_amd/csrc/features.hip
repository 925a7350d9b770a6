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

template <int K, int CM, bool V4>
__global__ __launch_bounds__(kFeatTW * kFeatTH) void feat_update_kernel(FeatArgs a) {
    constexpr int TW = kFeatTW, TH = kFeatTH, NT = TW * TH;
    constexpr int R = (K - 1) / 2, LW = V4 ? TW + 8 : TW + K - 1, PL = LW * (TH + K - 1);
    constexpr int XO = V4 ? 4 : R;   // staged columns left of the tile
    static_assert(XO >= R, "vector staging needs k <= 9");
    extern __shared__ float lds[];
    const int C = a.C, D = a.D;
    const float* sc = lds;                 // 3 colour planes
    const float* sf = lds + 3 * PL;        // D feature planes
    const float* sq = sf + D * PL;         // C planes of Q_t
    const int tile = blockIdx.x;
    const int b = tile / a.tiles_per_img;
    const int tr = tile - b * a.tiles_per_img;
    const int ty = tr / a.tiles_x, tx = tr - ty * a.tiles_x;
    const int y0 = ty * TH - R, x0 = tx * TW - XO;
    const long long hw = (long long)a.H * a.W;
    const float* ib = a.image + (long long)b * 3 * hw;
    const float* fb = a.feat + (long long)b * D * hw;
    const float* qb = a.src + (long long)b * C * hw;
    const int nplanes = 3 + D + C;
    if constexpr (V4) {
        // 16-byte vectors: x0 and LW multiples of 4, W a multiple of 4, so
        // a vector lies wholly inside or outside the image
        constexpr int LQ = LW / 4, LH = PL / LW;
#pragma unroll 8
        for (int e = threadIdx.x; e < nplanes * LH * LQ; e += NT) {
            const int pl = e / (LH * LQ), o = e - pl * (LH * LQ);
            const int ly = o / LQ, lq = o - ly * LQ;
            const int gy = y0 + ly, gx = x0 + 4 * lq;
            const float* src = pl < 3 ? ib + pl * hw
                                      : (pl < 3 + D ? fb + (pl - 3) * hw : qb + (pl - 3 - D) * hw);
            const bool ok = gy >= 0 && gy < a.H && gx >= 0 && gx < a.W;
            const float4 v = *reinterpret_cast<const float4*>(
                src + (ok ? (long long)gy * a.W + gx : 0));
            *reinterpret_cast<float4*>(lds + pl * PL + ly * LW + 4 * lq) =
                ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    } else {
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
    }
    __syncthreads();

    const int lx = threadIdx.x % TW, ly = threadIdx.x / TW;
    const int px = tx * TW + lx, py = ty * TH + ly;
    if (px >= a.W || py >= a.H) return;
    const int oc = (ly + R) * LW + lx + XO;
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

template <int K, bool V4>
hipError_t launch_kv(const FeatArgs& a, hipStream_t stream) {
    const size_t lds = feat_lds_bytes(K, a.C, a.D, V4);
    const dim3 grid(a.ntiles), block(kFeatTW * kFeatTH);
    if (a.C <= 8)
        hipLaunchKernelGGL((feat_update_kernel<K, 8, V4>), grid, block, lds, stream, a);
    else if (a.C <= 21)
        hipLaunchKernelGGL((feat_update_kernel<K, 21, V4>), grid, block, lds, stream, a);
    else
        hipLaunchKernelGGL((feat_update_kernel<K, kMaxC, V4>), grid, block, lds, stream, a);
    return hipGetLastError();
}

template <int K>
hipError_t launch_k(const FeatArgs& a, hipStream_t stream) {
    if constexpr (K <= 7) {
        if (a.vec4) return launch_kv<K, true>(a, stream);
    }
    return launch_kv<K, false>(a, stream);
}

}  // namespace

hipError_t launch_feat_update(const FeatArgs& a, int k, hipStream_t stream) {
    if (a.C < 1 || a.C > kMaxC || a.D < 1 || a.D > kMaxFeat || a.ntiles <= 0)
        return hipErrorInvalidValue;
    if (feat_lds_bytes(k, a.C, a.D, a.vec4) > 160 * 1024) return hipErrorInvalidValue;
    if (a.vec4 && (k > 7 || a.W % 4 != 0)) return hipErrorInvalidValue;
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
