// blur.hip -- one whole iteration of the pooled ("blur") mean-field of
// Sec. 4.2 per launch, for a 4 x 4 pooling on gfx950.
//
// Compiled once per window side k (-DCRF_BLUR_K=k).  The pooled grid has one
// cell per 4 x 4 pixels.  A work-group owns 8 x 8 cells (32 x 32 pixels) of
// one image and, in one launch:
//   1. stages the pooled Q_t and the pooled colours of its cells, a one-cell
//      ring around them and the r-cell window halo of that ring into LDS
//      (zero outside the grid), then prefetches the unary of its 1024 pixels
//      into registers, which arrives under the message;
//   2. computes the pooled message (Eq. 6 on the pooled grid, offsets of 4
//      pixels, Eq. 4 weights from pooled colours) for its 8 x 8 cells and the
//      one-cell ring that the bilinear upsampling of its pixels reads: each
//      of the 8 wavefronts takes window rows w and w + 8, each lane two
//      horizontally adjacent cells, the rows' weights in registers and
//      applied to every class; the k row partials are summed in LDS (all
//      classes at once where they fit, else a chunk at a time);
//   3. per pixel: bilinear upsampling of the message (half-pixel centres,
//      edge clamp), compatibility, unary and softmax (Alg. 1), then either
//      the full-resolution Q (the last iteration) or its 4 x 4 cell average,
//      the pooled Q_{t+1} the next launch reads.
// So each iteration reads the unary once and the pooled state, and the
// pooled message is never written to memory.
#include "crf_internal.h"

#ifndef CRF_BLUR_K
#error "compile with -DCRF_BLUR_K=<odd window side>"
#endif

namespace convcrf {
namespace {

constexpr int kS = kFusedBlurFactor;          // pixels per cell side
constexpr int kNC = kFusedBlurCells;          // own cells per work-group side
constexpr int kMT = kNC + 2;                  // message tile side: own cells and a ring of one

template <int K>
struct BlurShape {
    static constexpr int R = (K - 1) / 2;
    static constexpr int FS = kMT + 2 * R;                  // footprint side (cells)
    static constexpr int FP = FS * FS;
    static constexpr int NWAVE = 8;
    static constexpr int NT = 64 * NWAVE;                  // threads
    static constexpr int RW = (K + NWAVE - 1) / NWAVE;     // window rows per wave
    static constexpr int NPAIR = kMT / 2 * kMT;            // lanes with a pair of cells
};


// Half-pixel-centred bilinear source of output pixel o on a grid of n cells
// of kS pixels: (o + 0.5) / kS - 0.5, clamped at 0 and n - 1.
__device__ __forceinline__ void src_coord(int o, int n, int& i0, int& i1, float& f) {
    float u = ((float)o + 0.5f) / (float)kS - 0.5f;
    u = fmaxf(u, 0.f);
    int a = (int)u;
    if (a > n - 1) a = n - 1;
    i0 = a;
    i1 = a < n - 1 ? a + 1 : n - 1;
    f = u - (float)a;
}

template <int K, int CM, bool EXACT>
__global__ __launch_bounds__(BlurShape<K>::NT) void blur_iter_kernel(const BlurIterArgs a) {
    using BS = BlurShape<K>;
    constexpr int R = BS::R, FS = BS::FS, FP = BS::FP, NT = BS::NT, RW = BS::RW;
    constexpr int MTC = kMT * kMT;
    constexpr int NW = K + 1;                      // footprint cells one lane's row reads (even)
    constexpr int kChunk = blur_iter_chunk(K, CM); // classes per row-partial round
    static_assert(NW % 2 == 0 && FS % 2 == 0 && FP % 2 == 0, "8-byte rows");
    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qf = smem;                        // [CM][FS][FS] pooled Q_t
    float* const Cf = Qf + CM * FP;                // [3][FS][FS] pooled colours
    float* const Pt = Cf + 3 * FP;                 // [K][kChunk][MTC] row partials
    float* const Mt = Pt + K * kChunk * MTC;       // [CM][MTC] pooled message
    float* const Mu = Mt + CM * MTC;               // [CM][CM] compatibility, when given

    const int C = EXACT ? CM : a.C;
    const int Hp = a.Hp, Wp = a.Wp, H = a.H, W = a.W;
    const int b = blockIdx.z;
    const int cy0 = blockIdx.y * kNC, cx0 = blockIdx.x * kNC;     // first own cell
    const size_t HWp = (size_t)Hp * Wp, HW = (size_t)H * W;
    const int tid = threadIdx.x;

    // ---- staging loads (pooled Q_t and colours over the footprint, zero
    // outside the grid), all issued before any LDS store
    constexpr int NST = (CM + 3) * FP;
    constexpr int PER = (NST + NT - 1) / NT;
    const float* __restrict__ qsrc = a.qbar + (size_t)b * a.C * HWp;
    const float* __restrict__ csrc = a.pcol + (size_t)b * 3 * HWp;
    float v[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int idx = tid + j * NT;
        const int pl = idx / FP, rem = idx - pl * FP;
        const int r = rem / FS, cc = rem - r * FS;
        const int gy = cy0 - 1 - R + r, gx = cx0 - 1 - R + cc;
        const bool plane_ok = idx < NST && (pl >= CM || EXACT || pl < C);
        const bool in = plane_ok && gy >= 0 && gy < Hp && gx >= 0 && gx < Wp;
        const size_t g = in ? (size_t)gy * Wp + gx : 0;
        v[j] = in ? (pl < CM ? qsrc[(size_t)pl * HWp + g] : csrc[(size_t)(pl - CM) * HWp + g]) : 0.f;
    }

#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int idx = tid + j * NT;
        if (idx < NST) smem[idx] = v[j];
    }
    if (a.mu)
        for (int i = tid; i < C * C; i += NT) Mu[(i / C) * CM + i % C] = a.mu[i];

    // ---- unary prefetch, issued once the staged values are stored so that
    // no wait above covers it: every thread owns two horizontally adjacent
    // pixels, eight threads per cell (cell-major, so that a cell's threads
    // are consecutive lanes); every load is issued (planes past C read plane
    // 0 and are ignored)
    static_assert(NT == kNC * kNC * 8, "two pixels per thread");
    const int ci = tid >> 3, jj = tid & 7;
    const int ccy = cy0 + ci / kNC, ccx = cx0 + ci % kNC;           // own cell
    const int py = ccy * kS + (jj >> 1), px = ccx * kS + 2 * (jj & 1);
    const bool pix_ok = ccy < Hp && ccx < Wp;                       // H, W multiples of kS
    float u0[CM], u1[CM];
    {
        const float* up = a.unary + (size_t)b * a.C * HW + (size_t)(pix_ok ? py : 0) * W +
                          (pix_ok ? px : 0);
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            const float2 t =
                *reinterpret_cast<const float2*>(up + (size_t)(EXACT || c < C ? c : 0) * HW);
            u0[c] = t.x;
            u1[c] = t.y;
        }
    }
    __syncthreads();

    // ---- pooled message: wave w takes window rows w + 8 j (j < RW), lane
    // l < NPAIR the cells (mi, mj) and (mi, mj + 1) of the message tile
    const int wave = tid >> 6, lane = tid & 63;
    const bool msg = lane < BS::NPAIR;
    const int mi = lane / (kMT / 2), mj = 2 * (lane % (kMT / 2));
    float w[RW][2][K];
    if (msg) {
        float own[3][2];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
#pragma unroll
            for (int i = 0; i < 2; ++i) own[ch][i] = Cf[ch * FP + (mi + R) * FS + mj + R + i];
#pragma unroll
        for (int j = 0; j < RW; ++j) {
            const int dy = wave + BS::NWAVE * j;
            if (dy >= K) continue;
            float nc[3][NW];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch)
#pragma unroll
                for (int x = 0; x < NW; ++x) nc[ch][x] = Cf[ch * FP + (mi + dy) * FS + mj + x];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    const int n = (dx - R) * (dx - R) + (dy - R) * (dy - R);
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    const float k = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[n])) +
                                    a.taps.smooth[n];
                    // the centre tap: excluded, or K(p, p) when included
                    w[j][i][dx] = (dy == R && dx == R) ? (a.include_center ? a.center_w : 0.f) : k;
                }
            }
        }
    }
    for (int c0 = 0; c0 < C; c0 += kChunk) {
        const int cn = C - c0 < kChunk ? C - c0 : kChunk;
        if (msg) {
#pragma unroll
            for (int j = 0; j < RW; ++j) {
                const int dy = wave + BS::NWAVE * j;
                if (dy >= K) continue;
                for (int cl = 0; cl < cn; ++cl) {
                    // FS and mj are even: the row starts on 8 bytes
                    const float2* row = reinterpret_cast<const float2*>(
                        Qf + (c0 + cl) * FP + (mi + dy) * FS + mj);
                    float q[NW];
#pragma unroll
                    for (int x = 0; x < NW / 2; ++x) {
                        const float2 t = row[x];
                        q[2 * x] = t.x;
                        q[2 * x + 1] = t.y;
                    }
                    float m0 = 0.f, m1 = 0.f;
#pragma unroll
                    for (int dx = 0; dx < K; ++dx) {
                        m0 = fmaf(w[j][0][dx], q[dx], m0);
                        m1 = fmaf(w[j][1][dx], q[dx + 1], m1);
                    }
                    *reinterpret_cast<float2*>(Pt + (dy * kChunk + cl) * MTC + mi * kMT + mj) =
                        make_float2(m0, m1);
                }
            }
        }
        __syncthreads();
        for (int i = tid; i < cn * MTC; i += NT) {
            const int cl = i / MTC, cell = i - cl * MTC;
            float m = 0.f;
#pragma unroll
            for (int r = 0; r < K; ++r) m += Pt[(r * kChunk + cl) * MTC + cell];
            Mt[(c0 + cl) * MTC + cell] = m;
        }
        __syncthreads();
    }

    // ---- per pixel: bilinear message, compatibility, unary, softmax
    int ya, yb, xa, xb, xa1, xb1;
    float fy, fx0, fx1;
    src_coord(py, Hp, ya, yb, fy);
    src_coord(px, Wp, xa, xb, fx0);
    src_coord(px + 1, Wp, xa1, xb1, fx1);
    // message-tile coordinates of the four taps (the ring covers them)
    const int ty0 = ya - (cy0 - 1), ty1 = yb - (cy0 - 1);
    const int o00 = ty0 * kMT + xa - (cx0 - 1), o01 = ty0 * kMT + xb - (cx0 - 1);
    const int o10 = ty1 * kMT + xa - (cx0 - 1), o11 = ty1 * kMT + xb - (cx0 - 1);
    const int p00 = ty0 * kMT + xa1 - (cx0 - 1), p01 = ty0 * kMT + xb1 - (cx0 - 1);
    const int p10 = ty1 * kMT + xa1 - (cx0 - 1), p11 = ty1 * kMT + xb1 - (cx0 - 1);
    float z0[CM], z1[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) {
            z0[c] = z1[c] = 0.f;
            continue;
        }
        const float* m = Mt + c * MTC;
        {
            const float top = fmaf(fx0, m[o01] - m[o00], m[o00]);
            const float bot = fmaf(fx0, m[o11] - m[o10], m[o10]);
            z0[c] = fmaf(fy, bot - top, top);
        }
        {
            const float top = fmaf(fx1, m[p01] - m[p00], m[p00]);
            const float bot = fmaf(fx1, m[p11] - m[p10], m[p10]);
            z1[c] = fmaf(fy, bot - top, top);
        }
    }
    if (a.mu) {
        float t0[CM], t1[CM];
#pragma unroll
        for (int l = 0; l < CM; ++l) {
            t0[l] = t1[l] = 0.f;
            if (!EXACT && l >= C) continue;
#pragma unroll
            for (int lp = 0; lp < CM; ++lp) {
                if (!EXACT && lp >= C) continue;
                const float mu = Mu[l * CM + lp];
                t0[l] = fmaf(mu, z0[lp], t0[l]);
                t1[l] = fmaf(mu, z1[lp], t1[l]);
            }
        }
#pragma unroll
        for (int l = 0; l < CM; ++l) {
            z0[l] = u0[l] - t0[l];
            z1[l] = u1[l] - t1[l];
        }
    } else {
        // Potts: softmax(U + M), a per-pixel shift of U - (sum M - M)
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            z0[c] += u0[c];
            z1[c] += u1[c];
        }
    }
    softmax_regs<CM, EXACT>(z0, C);
    softmax_regs<CM, EXACT>(z1, C);
    if (a.q_full) {
        if (!pix_ok) return;
        float* q = a.q_full + (size_t)b * a.C * HW + (size_t)py * W + px;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C)
                *reinterpret_cast<float2*>(q + (size_t)c * HW) = make_float2(z0[c], z1[c]);
        return;
    }
    // the cell's 16 pixels: two per lane, eight consecutive lanes
    float* dq = a.qbar_out + (size_t)b * a.C * HWp + (size_t)ccy * Wp + ccx;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        float t = z0[c] + z1[c];
        t += __shfl_xor(t, 1, 64);
        t += __shfl_xor(t, 2, 64);
        t += __shfl_xor(t, 4, 64);
        if (jj == 0 && pix_ok) dq[(size_t)c * HWp] = t * (1.0f / (kS * kS));
    }
}

template <int K, int CM, bool EXACT>
hipError_t launch_one(const BlurIterArgs& a, size_t lds, hipStream_t stream) {
    auto fn = blur_iter_kernel<K, CM, EXACT>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const dim3 grid((a.Wp + kNC - 1) / kNC, (a.Hp + kNC - 1) / kNC, a.B);
    hipLaunchKernelGGL(fn, grid, dim3(BlurShape<K>::NT), lds, stream, a);
    return hipGetLastError();
}

}  // namespace

#define CRF_CAT2(a, b) a##b
#define CRF_CAT(a, b) CRF_CAT2(a, b)

hipError_t CRF_CAT(launch_blur_iter_k, CRF_BLUR_K)(const BlurIterArgs& a, hipStream_t stream) {
    constexpr int K = CRF_BLUR_K;
    if constexpr (K < 3) {
        return hipErrorNotSupported;
    } else {
        if (a.C < 1 || a.C > kMaxC || a.Hp * kS != a.H || a.Wp * kS != a.W || a.B < 1 ||
            a.B > 65535 || a.Hp > 65535 * kNC)
            return hipErrorInvalidValue;
        const bool mu = a.mu != nullptr;
        switch (a.C) {
            case 19: return launch_one<K, 19, true>(a, blur_iter_lds_bytes(K, 19, mu), stream);
            case 21: return launch_one<K, 21, true>(a, blur_iter_lds_bytes(K, 21, mu), stream);
            default: break;
        }
        if (a.C <= 8) return launch_one<K, 8, false>(a, blur_iter_lds_bytes(K, 8, mu), stream);
        return launch_one<K, 24, false>(a, blur_iter_lds_bytes(K, 24, mu), stream);
    }
}

}  // namespace convcrf
