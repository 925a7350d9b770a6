// backward.hip -- reverse-mode derivative of the unpooled mean-field
// (Alg. 1 unrolled over its T rounds, Eq. 4 kernel, Eq. 6 message).
//
// Each round is undone by two kernels:
//   bwd_point_kernel   the adjoints of the softmax (normalisation), the unary
//                      addition and the compatibility transform, per pixel;
//   bwd_msg_kernel     the adjoint of the message: because K(p,q) = K(q,p)
//                      and q lies in the window of p exactly when p lies in
//                      the window of q, the transpose of the message is the
//                      message itself applied to dL/dM.  The same pass sums
//                      the derivative with respect to the Eq. 4 parameters
//                      and, when the compatibility derivative is wanted,
//                      recomputes the forward message M^t and sums
//                      dP_p(l) M_p(l') over the tile's pixels.
// bwd_reduce_kernel folds the per-tile partial sums; group_sum_kernel adds
// the class groups' parts of dL/dF (learnable features).  upsample_t_kernel
// and pool_t_kernel are the transposes of the blur variant's upsampling and
// pooling.
//
// Built once per window side k with -DCRF_BWD_K=k (the adjoint-message
// kernels of that k) and once without (the pointwise and reduction kernels
// and the dispatch over k).
#include "crf_internal.h"
#include "lds_dma.h"

namespace convcrf {
namespace {

#if defined(CRF_BWD_K)

// ---------------------------------------------------------- adjoint message

// Tile plus halo of the 3 colour planes, the D feature planes (FT), the C
// planes of Q^t and the C planes of dL/dM^t into LDS (LW x LH each, rows LS
// >= LW floats apart and planes PS floats apart, the first staged column is
// x0, the first row y0); zero outside the image and in the row padding, so
// that taps there contribute nothing to any sum.
//
// DMA: every wave issues buffer loads that write 64 consecutive floats of a
// plane straight into LDS (rows of the padded plane, spread over the waves),
// with an out-of-range offset, which reads zero, for positions outside the
// image; then waits for all of them.  Otherwise scalar loads through
// registers, branch-free (an in-image address is read for every element and
// the value dropped outside) so that many are in flight per thread.
template <int NT, int LW, int LS, int PL, int PS, bool DMA>
__device__ __forceinline__ void stage_planes(float* lds, const BwdArgs& a, int b, int y0,
                                             int x0, int c0, int CN) {
    const int C = a.C;
    const long long hw = (long long)a.H * a.W;
    const float* fb = a.feat + (long long)b * 3 * hw;
    const float* qb = a.q + (long long)b * C * hw;
    const float* mb = a.dm + (long long)b * C * hw;
    const int D = a.sfeat ? a.D : 0;
    const float* sb = a.sfeat ? a.sfeat + (long long)b * D * hw : fb;
    if constexpr (DMA) {
        constexpr int RP = PS / 64, NW = NT / 64, NS = (RP + NW - 1) / NW;
        const int H = a.H, W = a.W;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int lane = threadIdx.x & 63;
        unsigned voff[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int f = (wave + NW * s) * 64 + lane;
            const int ly = f / LS, lx = f - ly * LS;
            const int gy = y0 + ly, gx = x0 + lx;
            const bool ok = f < PL && lx < LW && gy >= 0 && gy < H && gx >= 0 && gx < W;
            voff[s] = ok ? (unsigned)(gy * W + gx) * 4u : kDmaOob;
        }
        const unsigned lds0 = (unsigned)(size_t)(__attribute__((address_space(3))) float*)lds;
        auto issue = [&](rsrc_t r, int p, int lp) {
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const int jr = wave + NW * s;
                if (jr < RP)
                    lds_dma(r, voff[s], (int)(p * hw * 4), lds0 + (unsigned)((lp * PS + jr * 64) * 4));
            }
        };
        const rsrc_t rf = buffer_rsrc(fb, (unsigned)(3 * hw * 4));
        const rsrc_t rs = buffer_rsrc(sb, (unsigned)((D > 0 ? D : 3) * hw * 4));
        const rsrc_t rq = buffer_rsrc(qb, (unsigned)(C * hw * 4));
        const rsrc_t rm = buffer_rsrc(mb, (unsigned)(C * hw * 4));
        for (int ch = 0; ch < 3; ++ch) issue(rf, ch, ch);
        for (int c = 0; c < D; ++c) issue(rs, c, 3 + c);
        for (int c = 0; c < CN; ++c) issue(rq, c0 + c, 3 + D + c);
        for (int c = 0; c < CN; ++c) issue(rm, c0 + c, 3 + D + CN + c);
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
        return;
    }
    const int nplanes = 2 * CN + 3 + D;
#pragma unroll 16
    for (int e = threadIdx.x; e < nplanes * PL; e += NT) {
        const int pl = e / PL, o = e - pl * PL;
        const int ly = o / LS, lx = o - ly * LS;
        const int gy = y0 + ly, gx = x0 + lx;
        const int pq = pl - 3 - D;   // index among the group's Q and dL/dM planes
        const float* src = pl < 3 ? fb + pl * hw
                                  : (pq < 0 ? sb + (pl - 3) * hw
                                            : (pq < CN ? qb + (c0 + pq) * hw
                                                       : mb + (c0 + pq - CN) * hw));
        const bool ok = lx < LW && gy >= 0 && gy < a.H && gx >= 0 && gx < a.W;
        const float v = src[ok ? (long long)gy * a.W + gx : 0];
        lds[pl * PS + o] = ok ? v : 0.f;
    }
}

// The tile's sums of the five parameter terms over its threads, in a fixed
// order, added into kpart[tile] (or written).
template <int NT>
__device__ __forceinline__ void tile_param_sums(float (&g)[5], const BwdArgs& a, int row) {
    __shared__ float red[5][NT / 64];
#pragma unroll
    for (int j = 0; j < 5; ++j)
        for (int off = 32; off > 0; off >>= 1) g[j] += __shfl_xor(g[j], off, 64);
    const int wave = threadIdx.x / 64;
    if ((threadIdx.x & 63) == 0)
#pragma unroll
        for (int j = 0; j < 5; ++j) red[j][wave] = g[j];
    __syncthreads();
    if (threadIdx.x < 5) {
        const int j = threadIdx.x;
        float s = 0.f;
        for (int w = 0; w < NT / 64; ++w) s += red[j][w];
        float* o = a.kpart + (long long)row * 5 + j;
        *o = a.accumulate ? *o + s : s;
    }
}

// The tile's sum of dp_x(l) M_x(l') over its NT * PX pixels, added into
// gpart[tile] (or written).  Each thread hands in PX pixels: their forward
// message mv, whether they lie in the image, and their offset in the
// [B][C][H][W] planes.  dp and M go to LDS (zero for pixels outside the
// image and rows past C), then each thread sums one 3 x 3 block of (l, l')
// over one group of pixels, and the groups are added in order.
// dp of all C classes (rows) against the M of the group's CN classes
// c0 .. c0 + CN - 1 (columns); pix[i] is the offset of the pixel in plane 0.
template <int NT, int PX, int CM>
__device__ __forceinline__ void tile_gram(float* lds, const BwdArgs& a, int tile, int c0,
                                          int CN, const float (&mv)[PX][CM],
                                          const bool (&in)[PX], const long long (&pix)[PX]) {
    constexpr int NPIX = NT * PX, SP = NPIX + 1;
    const int C = a.C;
    const long long hw = (long long)a.H * a.W;
    const int CP = bwd_gram_rows(C), CQ = bwd_gram_rows(CN);
    float* gp = lds;
    float* gm = lds + CP * SP;
    __syncthreads();  // the staged planes have been read
#pragma unroll
    for (int i = 0; i < PX; ++i) {
        const int col = PX * threadIdx.x + i;
        // every class of the pixel loaded before the first is stored, all in
        // flight at once (pixels outside the image read pixel 0 of image 0
        // and classes past C the last class, both dropped)
        const bool potts = a.dm_sum_scale != 0.f;
        const float* src = (potts ? a.dm : a.dp) + (in[i] ? pix[i] : 0);
        float v[kMaxC];
#pragma unroll
        for (int c = 0; c < kMaxC; ++c) v[c] = src[(long long)(c < C ? c : C - 1) * hw];
        if (potts) {
            // Potts: dM(l) = dZ(l) - sum_l' dZ(l'), so sum_l dM(l) = (1 - C)
            // sum_l' dZ(l') and dZ(l) = dM(l) + sum_l' dM(l') / (1 - C)
            float sum = 0.f;
#pragma unroll
            for (int c = 0; c < kMaxC; ++c) {
                if (c < CP) {
                    const float x = in[i] && c < C ? v[c] : 0.f;
                    gp[c * SP + col] = x;
                    sum += x;
                }
            }
            const float sh = sum * a.dm_sum_scale;
#pragma unroll
            for (int c = 0; c < kMaxC; ++c)
                if (c < C) gp[c * SP + col] = -((in[i] ? v[c] : 0.f) + sh);
        } else {
#pragma unroll
            for (int c = 0; c < kMaxC; ++c)
                if (c < CP) gp[c * SP + col] = in[i] && c < C ? v[c] : 0.f;
        }
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (c < CQ) gm[c * SP + col] = in[i] && c < CN ? mv[i][c] : 0.f;
        for (int c = CM; c < CQ; ++c) gm[c * SP + col] = 0.f;   // past the held classes
    }
    __syncthreads();
    const int nbr = CP / 3, nbc = CQ / 3, nb = nbr * nbc;
    const int ng = NT / nb;
    const int bi = threadIdx.x % nb, pg = threadIdx.x / nb;
    const int l0 = 3 * (bi / nbc), m0 = 3 * (bi % nbc);
    float s9[9];
#pragma unroll
    for (int e = 0; e < 9; ++e) s9[e] = 0.f;
    if (pg < ng) {
        for (int x = pg; x < NPIX; x += ng) {
            const float p0 = gp[l0 * SP + x], p1 = gp[(l0 + 1) * SP + x],
                        p2 = gp[(l0 + 2) * SP + x];
            const float q0 = gm[m0 * SP + x], q1 = gm[(m0 + 1) * SP + x],
                        q2 = gm[(m0 + 2) * SP + x];
            s9[0] = fmaf(p0, q0, s9[0]); s9[1] = fmaf(p0, q1, s9[1]); s9[2] = fmaf(p0, q2, s9[2]);
            s9[3] = fmaf(p1, q0, s9[3]); s9[4] = fmaf(p1, q1, s9[4]); s9[5] = fmaf(p1, q2, s9[5]);
            s9[6] = fmaf(p2, q0, s9[6]); s9[7] = fmaf(p2, q1, s9[7]); s9[8] = fmaf(p2, q2, s9[8]);
        }
    }
    __syncthreads();  // dp and M have been read
    float* gr = lds;   // [ng][nb][9]
    if (pg < ng)
#pragma unroll
        for (int e = 0; e < 9; ++e) gr[(pg * nb + bi) * 9 + e] = s9[e];
    __syncthreads();
    for (int idx = threadIdx.x; idx < nb * 9; idx += NT) {
        float sum = 0.f;
        for (int g = 0; g < ng; ++g) sum += gr[g * nb * 9 + idx];
        const int blk = idx / 9, e = idx - blk * 9;
        const int l = 3 * (blk / nbc) + e / 3, lp = 3 * (blk % nbc) + e % 3;
        if (l < C && lp < CN) {
            float* o = a.gpart + (long long)tile * C * C + l * C + c0 + lp;
            *o = a.accumulate ? *o + sum : sum;
        }
    }
}

// One pixel per thread, 32 x TH tiles up to k = 7 (16 x 8 above).  CM >= C
// classes are computed without branches: planes past C - 1 read plane C - 1 again and
// are never stored, and their dL/dM is zero, so they add nothing to dk.
template <int K, int TH, int CM, bool WM, bool DMA, bool FT>
__global__ __launch_bounds__(bwd_tile_w(K) * TH) void bwd_msg_kernel(BwdArgs a) {
    constexpr int TW = bwd_tile_w(K), NT = TW * TH;
    constexpr int R = (K - 1) / 2, LW = TW + K - 1, LS = bwd_row_stride(K);
    constexpr int PL = LS * (TH + K - 1);
    constexpr int PS = bwd_plane(K, TH, DMA);   // plane stride in LDS
    constexpr int XO = R;                       // staged columns left of the tile
    extern __shared__ float lds[];
    const int C = a.C;
    const int D = FT ? a.D : 0;
    const float* sc = lds;               // 3 colour planes
    const float* sf = lds + 3 * PS;      // D feature planes (FT)
    const int tile = blockIdx.x;
    const int b = tile / a.tiles_per_img;
    const int tr = tile - b * a.tiles_per_img;
    const int ty = tr / a.tiles_x, tx = tr - ty * a.tiles_x;
    const long long hw = (long long)a.H * a.W;
    // this work-group's class group: classes c0 .. c0 + CN - 1
    const int c0 = blockIdx.y * a.cgsize;
    const int CN = C - c0 < a.cgsize ? C - c0 : a.cgsize;
    stage_planes<NT, LW, LS, PL, PS, DMA>(lds, a, b, ty * TH - R, tx * TW - XO, c0, CN);
    const float* sq = sf + D * PS;       // the group's CN planes of Q^t
    const float* sm = sq + CN * PS;      // the group's CN planes of dL/dM^t
    __syncthreads();

    const int lx = threadIdx.x % TW, ly = threadIdx.x / TW;
    const int px = tx * TW + lx, py = ty * TH + ly;
    const bool in = px < a.W && py < a.H;
    const long long pix = (long long)b * C * hw + (long long)py * a.W + px;
    float g[5] = {0.f, 0.f, 0.f, 0.f, 0.f};
    float ma[1][CM];   // the forward message of the pixel (compatibility derivative)
#pragma unroll
    for (int c = 0; c < CM; ++c) ma[0][c] = 0.f;
    if (in) {
        const int oc = (ly + R) * LS + lx + XO;
        const float ir = sc[oc], ig = sc[PS + oc], ib = sc[2 * PS + oc];
        float dmq[CM], dqa[CM];
        int poff[CM];
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            poff[c] = (c < CN ? c : CN - 1) * PS;
            dmq[c] = c < CN ? sm[poff[c] + oc] : 0.f;
            dqa[c] = 0.f;
        }
        // FT: own features and Q, and the feature derivative of the pixel
        float fo[kMaxFeat], dfa[kMaxFeat], qo[FT ? CM : 1];
#pragma unroll
        for (int c = 0; c < kMaxFeat; ++c) {
            fo[c] = FT && c < D ? sf[c * PS + oc] : 0.f;
            dfa[c] = 0.f;
        }
        if constexpr (FT) {
#pragma unroll
            for (int c = 0; c < CM; ++c) qo[c] = c < CN ? sq[poff[c] + oc] : 0.f;
        }
        // one tap: the offset's appearance log-prefactor al = a_log2[n], its
        // smoothness Gaussian s0 = smooth[n] (positions) and nf = n
        auto tap = [&](int dx, int dy, float al, float s0, float nf) {
            const int o = oc + dy * LS + dx;
            const float er = ir - sc[o], eg = ig - sc[PS + o], eb = ib - sc[2 * PS + o];
            const float cd2 = fmaf(er, er, fmaf(eg, eg, eb * eb));
            const float av = __builtin_amdgcn_exp2f(fmaf(a.neg_beta, cd2, al));
            // the smoothness Gaussian and its squared distance: the
            // positions, or the learnable features (FT)
            float sd2 = nf, sv = s0;
            float fdif[kMaxFeat];
            if constexpr (FT) {
                sd2 = 0.f;
#pragma unroll
                for (int c = 0; c < kMaxFeat; ++c) {
                    fdif[c] = c < D ? fo[c] - sf[c * PS + o] : 0.f;
                    sd2 = fmaf(fdif[c], fdif[c], sd2);
                }
                sv = __builtin_amdgcn_exp2f(a.neg_gamma * sd2);
            }
            const float w = fmaf(a.w_app, av, a.w_smooth * sv);
            float dk = 0.f, dkr = 0.f;
#pragma unroll
            for (int c = 0; c < CM; ++c) {
                const float qn = sq[poff[c] + o];
                const float mn = sm[poff[c] + o];
                dk = fmaf(dmq[c], qn, dk);
                dqa[c] = fmaf(w, mn, dqa[c]);
                if (WM) ma[0][c] = fmaf(w, qn, ma[0][c]);
                if (FT) dkr = fmaf(mn, qo[c], dkr);
            }
            const float da = dk * av, ds = dk * sv;
            g[0] += da;
            g[1] = fmaf(da, nf, g[1]);
            g[2] = fmaf(da, cd2, g[2]);
            g[3] += ds;
            g[4] = fmaf(ds, sd2, g[4]);
            if constexpr (FT) {
                const float coef = -(dk + dkr) * a.w_smooth * sv * a.inv_gamma2;
#pragma unroll
                for (int c = 0; c < kMaxFeat; ++c) dfa[c] = fmaf(coef, fdif[c], dfa[c]);
            }
        };
        // a window row at once; the per-offset constants of the row are read
        // once per row (n = dx^2 + dy^2 takes R + 1 values in it), so no
        // table load waits inside the row
#pragma unroll 1
        for (int dy = -R; dy <= R; ++dy) {
            float ra[R + 1], rs[R + 1], rn[R + 1];
#pragma unroll
            for (int j = 0; j <= R; ++j) {
                const int n = j * j + dy * dy;
                ra[j] = a.a_log2[n];
                rs[j] = a.smooth[n];
                rn[j] = (float)n;
            }
#pragma unroll
            for (int dx = -R; dx <= R; ++dx) {
                if (dx == 0 && dy == 0 && !a.include_center) continue;
                const int j = dx < 0 ? -dx : dx;
                tap(dx, dy, ra[j], rs[j], rn[j]);
            }
        }
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (c < CN) a.dq_out[pix + (c0 + c) * hw] = dqa[c];
        if constexpr (FT) {
            float* df = a.dfeat + (long long)b * D * hw + (long long)py * a.W + px;
            if (a.dfeat_gstride > 0) {
                // this class group's part; the parts are added after the launch
                df += blockIdx.y * a.dfeat_gstride;
#pragma unroll
                for (int c = 0; c < kMaxFeat; ++c)
                    if (c < D) df[c * hw] = dfa[c];
            } else {
#pragma unroll
                for (int c = 0; c < kMaxFeat; ++c)
                    if (c < D) df[c * hw] = a.accumulate ? df[c * hw] + dfa[c] : dfa[c];
            }
        }
    }
    if constexpr (WM) {
        const bool ins[1] = {in};
        const long long pixs[1] = {pix};
        tile_gram<NT, 1, CM>(lds, a, tile, c0, CN, ma, ins, pixs);
    }
    tile_param_sums<NT>(g, a, tile * a.cgroups + blockIdx.y);
}

template <int K, int TH, int CM, bool DMA, bool FT>
hipError_t launch_msg_ktc(const BwdArgs& a, hipStream_t stream) {
    const size_t lds = bwd_lds_bytes(K, a.C, TH, DMA, FT ? a.D : 0, a.cgsize);
    const dim3 block(bwd_tile_w(K) * TH), grid(a.ntiles, a.cgroups);
    if (a.gpart)
        hipLaunchKernelGGL((bwd_msg_kernel<K, TH, CM, true, DMA, FT>), grid, block, lds, stream,
                           a);
    else
        hipLaunchKernelGGL((bwd_msg_kernel<K, TH, CM, false, DMA, FT>), grid, block, lds,
                           stream, a);
    return hipGetLastError();
}

template <int K, int TH, int CM>
hipError_t launch_msg_ktv(const BwdArgs& a, hipStream_t stream) {
    if (a.dma) {
        if (a.sfeat) return launch_msg_ktc<K, TH, CM, true, true>(a, stream);
        return launch_msg_ktc<K, TH, CM, true, false>(a, stream);
    }
    if (a.sfeat) return launch_msg_ktc<K, TH, CM, false, true>(a, stream);
    return launch_msg_ktc<K, TH, CM, false, false>(a, stream);
}

// The class loop runs CM >= cgsize classes; groups of up to 8 classes (8-row
// tiles only) are instantiated at their own size.
template <int K, int TH>
hipError_t launch_msg_kt(const BwdArgs& a, hipStream_t stream) {
    if constexpr (TH == 8) {
        switch (a.cgsize) {
            case 1: case 2: case 3: return launch_msg_ktv<K, TH, 3>(a, stream);
            case 4: return launch_msg_ktv<K, TH, 4>(a, stream);
            case 5: return launch_msg_ktv<K, TH, 5>(a, stream);
            case 6: return launch_msg_ktv<K, TH, 6>(a, stream);
            case 7: return launch_msg_ktv<K, TH, 7>(a, stream);
            case 8: return launch_msg_ktv<K, TH, 8>(a, stream);
            default: break;
        }
    }
    if (a.cgsize <= 21) return launch_msg_ktv<K, TH, 21>(a, stream);
    return launch_msg_ktv<K, TH, kMaxC>(a, stream);
}

// The host derives the tiling (tiles_x, tiles_per_img, ntiles) from the
// same bwd_tile_w / bwd_tile_h.
template <int K>
hipError_t launch_msg_k(const BwdArgs& a, hipStream_t stream) {
    if constexpr (K <= 7) {
        if (bwd_tile_h(K, a.C, a.sfeat ? a.D : 0, a.dma != 0, a.cgsize) == 16)
            return launch_msg_kt<K, 16>(a, stream);
    }
    return launch_msg_kt<K, 8>(a, stream);
}

}  // namespace

#define CONVCRF_BWD_CAT2(a, b) a##b
#define CONVCRF_BWD_CAT(a, b) CONVCRF_BWD_CAT2(a, b)
hipError_t CONVCRF_BWD_CAT(launch_bwd_msg_k, CRF_BWD_K)(const BwdArgs& a, hipStream_t stream) {
    return launch_msg_k<CRF_BWD_K>(a, stream);
}

}  // namespace convcrf

#else

// ---------------------------------------------------------------- pointwise
// S > 1: dL/dQ is given on the S x S pooled grid (the pooled adjoint of the
// blur variant's message); pixel (y, x) takes its cell's value / S^2, the
// transpose of the average pooling, read in place (W is the image width).
template <int CM, int S>
__global__ __launch_bounds__(256) void bwd_point_kernel(
    const float* __restrict__ q, const float* __restrict__ dq, const float* __restrict__ mu,
    float* __restrict__ du, float* __restrict__ dm, float* __restrict__ dp, int C,
    long long hw, long long npix, int accumulate, int W) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= npix) return;
    const long long b = i / hw;
    const long long base = b * C * hw + (i - b * hw);
    long long dbase = base, dstride = hw;
    if constexpr (S > 1) {
        const int pix = (int)(i - b * hw);   // hw < 2^31
        const int y = pix / W, x = pix - y * W;
        dstride = hw / (S * S);
        dbase = b * C * dstride + (long long)(y / S) * (W / S) + x / S;
    }
    constexpr float inv = 1.f / (float)(S * S);
    // every load issued before the first is used (classes past C re-read
    // the last class and are dropped)
    float qv[CM], dz[CM], uo[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        const int cc = c < C ? c : C - 1;
        qv[c] = q[base + cc * hw];
        dz[c] = S > 1 ? dq[dbase + cc * dstride] * inv : dq[base + cc * hw];
    }
    if (accumulate) {
#pragma unroll
        for (int c = 0; c < CM; ++c) uo[c] = du[base + (c < C ? c : C - 1) * hw];
    } else {
#pragma unroll
        for (int c = 0; c < CM; ++c) uo[c] = 0.f;
    }
    float dot = 0.f;
#pragma unroll
    for (int c = 0; c < CM; ++c)
        if (c < C) dot = fmaf(qv[c], dz[c], dot);
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (c < C) {
            dz[c] = qv[c] * (dz[c] - dot);
            sum += dz[c];
            du[base + c * hw] = accumulate ? uo[c] + dz[c] : dz[c];
            if (dp) dp[base + c * hw] = -dz[c];
        }
    }
    if (!dm) return;
    if (mu) {
        for (int lp = 0; lp < C; ++lp) {
            float acc = 0.f;
#pragma unroll
            for (int l = 0; l < CM; ++l)
                if (l < C) acc = fmaf(mu[l * C + lp], -dz[l], acc);
            dm[base + lp * hw] = acc;
        }
    } else {
        // Potts, mu[l][l'] = [l != l']: dm(l') = -(sum_l dZ(l) - dZ(l'))
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (c < C) dm[base + c * hw] = dz[c] - sum;
    }
}

// ------------------------------------------------------- blur transposes
// Weight of pooled cell `cell` in the bilinear sample of output o, as the
// forward upsampling takes it: source coordinate (o + 0.5) / s - 0.5,
// clamped below at 0; cells i0 and i1 (clamped at n - 1) with 1 - f and f.
// s is 2, 4 or 8, so the product with 1 / s is the exact quotient.
__device__ __forceinline__ float up_weight(int o, int cell, float inv_s, int n) {
    float u = ((float)o + 0.5f) * inv_s - 0.5f;
    u = fmaxf(u, 0.f);
    int a = (int)u;
    if (a > n - 1) a = n - 1;
    const int i1 = a < n - 1 ? a + 1 : n - 1;
    const float f = u - (float)a;
    return (cell == a ? 1.f - f : 0.f) + (cell == i1 ? f : 0.f);
}

// Output o samples cell i0 = floor((o + 0.5) / s - 0.5) and i0 + 1, so the
// full-resolution pixels that sample cell (Y, X) lie in rows [s Y - s/2,
// s Y + 3s/2) and the same columns (the clamps at the edges only move
// pixels inside that range onto the edge cells).  A work-group takes a
// block of kUpTX x kUpTY cells of one plane: it stages the full-resolution
// pixels under the block (zero outside the image) into LDS with coalesced
// loads, then each thread sums the 2s x 2s window of its cell, row by row.
constexpr int kUpTX = 64, kUpTY = 4;
template <int S>
constexpr int up_cols() { return S * kUpTX + S; }
template <int S>
constexpr int up_rows() { return S * kUpTY + S; }
template <int S>
__global__ __launch_bounds__(256) void upsample_t_kernel(const float* __restrict__ in,
                                                         float* __restrict__ out, int Hp,
                                                         int Wp, int nbx, int nby) {
    constexpr int h = S / 2, NX = 2 * S, COLS = up_cols<S>(), ROWS = up_rows<S>();
    extern __shared__ float st[];                 // [ROWS][COLS]
    const int H = Hp * S, W = Wp * S;
    const long long blk = blockIdx.x;
    const long long plane = blk / ((long long)nbx * nby);
    const int rem = (int)(blk - plane * nbx * nby);
    const int by = rem / nbx, bx = rem - by * nbx;
    const int X0 = bx * kUpTX, Y0 = by * kUpTY;
    const int gy0 = S * Y0 - h, gx0 = S * X0 - h;
    const float* src = in + plane * H * W;
    // every load of the thread issued before the first LDS store
    constexpr int NE = (ROWS * COLS + 255) / 256;
    float v[NE];
#pragma unroll
    for (int k = 0; k < NE; ++k) {
        const int e = threadIdx.x + 256 * k;
        const int ly = e / COLS, lx = e - ly * COLS;
        const int gy = gy0 + ly, gx = gx0 + lx;
        const bool ok = e < ROWS * COLS && gy >= 0 && gy < H && gx >= 0 && gx < W;
        v[k] = ok ? src[(long long)gy * W + gx] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < NE; ++k) {
        const int e = threadIdx.x + 256 * k;
        if (e < ROWS * COLS) st[e] = v[k];
    }
    __syncthreads();
    const int tx = threadIdx.x % kUpTX, ty = threadIdx.x / kUpTX;
    const int X = X0 + tx, Y = Y0 + ty;
    if (X >= Wp || Y >= Hp) return;
    const float inv_s = 1.f / (float)S;
    float wx[NX];
#pragma unroll
    for (int j = 0; j < NX; ++j) {
        const int x = S * X - h + j;
        wx[j] = x >= 0 && x < W ? up_weight(x, X, inv_s, Wp) : 0.f;
    }
    float acc = 0.f;
#pragma unroll
    for (int jy = 0; jy < NX; ++jy) {
        const int y = S * Y - h + jy;
        if (y < 0 || y >= H) continue;
        const float wy = up_weight(y, Y, inv_s, Hp);
        const float* row = st + (S * ty + jy) * COLS + S * tx;
        float t = 0.f;
#pragma unroll
        for (int j = 0; j < NX; ++j) t = fmaf(wx[j], row[j], t);
        acc = fmaf(wy, t, acc);
    }
    out[(plane * Hp + Y) * Wp + X] = acc;
}

// blockIdx.y strides over the B * C * H full-resolution rows, kPoolTRows at
// a time; V consecutive pixels per thread (one pooled cell when V <= S), a
// vector store when V = 4.
constexpr int kPoolTRows = 8;
template <int S, int V>
__global__ __launch_bounds__(256) void pool_t_kernel(const float* __restrict__ in,
                                                     float* __restrict__ out, int Hp, int Wp,
                                                     long long nrows) {
    const int W = Wp * S, H = Hp * S;
    const int x = (blockIdx.x * blockDim.x + threadIdx.x) * V;
    if (x >= W) return;
    constexpr float inv = 1.f / (float)(S * S);
    for (long long r0 = (long long)blockIdx.y * kPoolTRows; r0 < nrows;
         r0 += (long long)gridDim.y * kPoolTRows) {
#pragma unroll
        for (int k = 0; k < kPoolTRows; ++k) {
            const long long r = r0 + k;
            if (r >= nrows) break;
            const long long plane = r / H;
            const int y = (int)(r - plane * H);
            const float* src = in + (plane * Hp + y / S) * Wp;
            if constexpr (V == 4) {
                const float val = src[x / S] * inv;
                *reinterpret_cast<float4*>(out + r * W + x) = make_float4(val, val, val, val);
            } else {
                out[r * W + x] = src[x / S] * inv;
            }
        }
    }
}

// ---------------------------------------------------------------- reduce
constexpr int kMaxGroupSum = kMaxC / 3;
__global__ __launch_bounds__(256) void group_sum_kernel(const float* __restrict__ part,
                                                        int groups, long long n,
                                                        float* __restrict__ out,
                                                        int accumulate) {
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    // at most kMaxGroupSum parts (groups of at least three of at most kMaxC
    // classes), all loaded before the first is added; the sum in group order
    float v[kMaxGroupSum];
#pragma unroll
    for (int g = 0; g < kMaxGroupSum; ++g)
        v[g] = part[(long long)(g < groups ? g : groups - 1) * n + i];
    float s = accumulate ? out[i] : 0.f;
#pragma unroll
    for (int g = 0; g < kMaxGroupSum; ++g)
        if (g < groups) s += v[g];
    out[i] = s;
}

struct ReduceArgs {
    const float* gpart;
    const float* kpart;
    float* out_compat;
    float* out_kernel;
    int groups, C, ntiles;
    float scale[5];
};

// Block e < C*C folds column e of gpart over its groups rows; block C*C + j
// folds column j of kpart over its ntiles rows.  Strided per-thread sums,
// then a tree, all in double.
__global__ __launch_bounds__(256) void bwd_reduce_kernel(ReduceArgs a) {
    __shared__ double red[256];
    const int ne = a.C * a.C;
    const int e = blockIdx.x;
    const bool compat = e < ne;
    if (compat ? !a.out_compat : !a.out_kernel) return;
    const int rows = compat ? a.groups : a.ntiles;
    const int stride = compat ? ne : 5;
    const float* col = compat ? a.gpart + e : a.kpart + (e - ne);
    // four rows' loads in flight at a time, added in row order
    double s = 0.0;
    int r = threadIdx.x;
    for (; r + 3 * 256 < rows; r += 4 * 256) {
        float v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = col[(long long)(r + 256 * j) * stride];
#pragma unroll
        for (int j = 0; j < 4; ++j) s += (double)v[j];
    }
    for (; r < rows; r += 256) s += (double)col[(long long)r * stride];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (compat) a.out_compat[e] = (float)red[0];
        else a.out_kernel[e - ne] = (float)(red[0] * (double)a.scale[e - ne]);
    }
}

}  // namespace

hipError_t launch_bwd_message(const BwdArgs& a, int k, hipStream_t stream) {
    if (a.C < 1 || a.C > kMaxC || a.ntiles <= 0) return hipErrorInvalidValue;
    const int D = a.sfeat ? a.D : 0;
    if (a.sfeat && (a.D < 1 || a.D > kMaxFeat || !a.dfeat)) return hipErrorInvalidValue;
    if (a.cgsize < 1 || a.cgroups < 1 || (long long)a.cgroups * a.cgsize < a.C ||
        (a.cgroups - 1) * a.cgsize >= a.C ||
        (a.sfeat && a.cgroups != 1 && a.dfeat_gstride <= 0) || a.cgroups > 65535)
        return hipErrorInvalidValue;
    if (bwd_lds_need(k, a.C, D, a.dma != 0, a.cgsize) > kBwdLdsLimit) return hipErrorInvalidValue;
    // buffer offsets of the DMA staging stay under 2 GB
    const long long hw = (long long)a.H * a.W;
    const int mp = a.C > 3 ? (a.C > D ? a.C : D) : (3 > D ? 3 : D);
    if (a.dma && (long long)mp * hw * 4 >= (1LL << 31)) return hipErrorInvalidValue;
    switch (k) {
        case 1: return launch_bwd_msg_k1(a, stream);
        case 3: return launch_bwd_msg_k3(a, stream);
        case 5: return launch_bwd_msg_k5(a, stream);
        case 7: return launch_bwd_msg_k7(a, stream);
        case 9: return launch_bwd_msg_k9(a, stream);
        case 11: return launch_bwd_msg_k11(a, stream);
        case 13: return launch_bwd_msg_k13(a, stream);
        case 15: return launch_bwd_msg_k15(a, stream);
        default: return hipErrorInvalidValue;
    }
}

template <int S>
void launch_bwd_point_s(const float* q, const float* dq, const float* mu, float* du, float* dm,
                        float* dp, int C, long long HW, long long npix, int accumulate, int W,
                        unsigned blocks, hipStream_t stream) {
    if (C <= 8)
        hipLaunchKernelGGL((bwd_point_kernel<8, S>), dim3(blocks), dim3(256), 0, stream, q, dq,
                           mu, du, dm, dp, C, HW, npix, accumulate, W);
    else
        hipLaunchKernelGGL((bwd_point_kernel<kMaxC, S>), dim3(blocks), dim3(256), 0, stream, q,
                           dq, mu, du, dm, dp, C, HW, npix, accumulate, W);
}

hipError_t launch_bwd_point(const float* q, const float* dq, const float* mu, float* du,
                            float* dm, float* dp, int B, int C, long long HW, int accumulate,
                            hipStream_t stream, int W, int s) {
    const long long npix = (long long)B * HW;
    if (npix == 0) return hipSuccess;
    if (C < 1 || C > kMaxC) return hipErrorInvalidValue;
    if (s > 1 && (W < s || W % s != 0 || HW % W != 0 || (HW / W) % s != 0 || HW > 0x7fffffffLL))
        return hipErrorInvalidValue;
    const long long blocks = (npix + 255) / 256;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    const unsigned nb = (unsigned)blocks;
    switch (s) {
        case 1: launch_bwd_point_s<1>(q, dq, mu, du, dm, dp, C, HW, npix, accumulate, W, nb, stream); break;
        case 2: launch_bwd_point_s<2>(q, dq, mu, du, dm, dp, C, HW, npix, accumulate, W, nb, stream); break;
        case 4: launch_bwd_point_s<4>(q, dq, mu, du, dm, dp, C, HW, npix, accumulate, W, nb, stream); break;
        case 8: launch_bwd_point_s<8>(q, dq, mu, du, dm, dp, C, HW, npix, accumulate, W, nb, stream); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int S>
hipError_t launch_up_t(const float* in, float* out, int B, int C, int Hp, int Wp,
                       hipStream_t stream) {
    const int nbx = (Wp + kUpTX - 1) / kUpTX, nby = (Hp + kUpTY - 1) / kUpTY;
    const long long blocks = (long long)B * C * nbx * nby;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    const size_t lds = sizeof(float) * up_rows<S>() * up_cols<S>();
    auto fn = upsample_t_kernel<S>;
    if (lds > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                                 hipFuncAttributeMaxDynamicSharedMemorySize,
                                                 (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(256), lds, stream, in, out, Hp, Wp, nbx,
                       nby);
    return hipGetLastError();
}

hipError_t launch_upsample_t(const float* in, float* out, int B, int C, int Hp, int Wp, int s,
                             hipStream_t stream) {
    if ((long long)B * C * Hp * Wp == 0) return hipSuccess;
    switch (s) {
        case 2: return launch_up_t<2>(in, out, B, C, Hp, Wp, stream);
        case 4: return launch_up_t<4>(in, out, B, C, Hp, Wp, stream);
        case 8: return launch_up_t<8>(in, out, B, C, Hp, Wp, stream);
        default: return hipErrorInvalidValue;
    }
}

template <int S, int V>
hipError_t launch_pool_t_sv(const float* in, float* out, int Hp, int Wp, long long nrows,
                            hipStream_t stream) {
    const long long W = (long long)Wp * S;
    const long long ry = (nrows + kPoolTRows - 1) / kPoolTRows;
    const dim3 grid((unsigned)((W / V + 255) / 256), (unsigned)(ry < 65535 ? ry : 65535));
    hipLaunchKernelGGL((pool_t_kernel<S, V>), grid, dim3(256), 0, stream, in, out, Hp, Wp, nrows);
    return hipGetLastError();
}

hipError_t launch_pool_t(const float* in, float* out, int B, int C, int Hp, int Wp, int s,
                         hipStream_t stream) {
    const long long nrows = (long long)B * C * Hp * s;
    const long long W = (long long)Wp * s;
    if (nrows == 0 || W == 0) return hipSuccess;
    if (W > 0x7fffffffLL) return hipErrorInvalidValue;
    const bool vec = reinterpret_cast<uintptr_t>(out) % 16 == 0;   // W % 4 == 0 for s >= 4
    switch (s) {
        case 2: return launch_pool_t_sv<2, 1>(in, out, Hp, Wp, nrows, stream);
        case 4: return vec ? launch_pool_t_sv<4, 4>(in, out, Hp, Wp, nrows, stream)
                           : launch_pool_t_sv<4, 1>(in, out, Hp, Wp, nrows, stream);
        case 8: return vec ? launch_pool_t_sv<8, 4>(in, out, Hp, Wp, nrows, stream)
                           : launch_pool_t_sv<8, 1>(in, out, Hp, Wp, nrows, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_group_sum(const float* part, int groups, long long n, float* out,
                            int accumulate, hipStream_t stream) {
    if (n == 0) return hipSuccess;
    const long long blocks = (n + 255) / 256;
    if (blocks > 0x7fffffffLL || groups < 1 || groups > kMaxGroupSum) return hipErrorInvalidValue;
    hipLaunchKernelGGL(group_sum_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, part,
                       groups, n, out, accumulate);
    return hipGetLastError();
}

hipError_t launch_bwd_reduce(const float* gpart, int groups, int C, float* out_compat,
                             const float* kpart, int ntiles, const float scale[5],
                             float* out_kernel, hipStream_t stream) {
    if (C < 1 || C > kMaxC) return hipErrorInvalidValue;
    ReduceArgs a{gpart, kpart, out_compat, out_kernel, groups, C, ntiles, {}};
    for (int j = 0; j < 5; ++j) a.scale[j] = scale[j];
    hipLaunchKernelGGL(bwd_reduce_kernel, dim3(C * C + 5), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace convcrf

#endif
