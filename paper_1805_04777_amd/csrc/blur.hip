// blur.hip -- one whole iteration of the pooled ("blur") mean-field of
// Sec. 4.2 per launch, for a 4 x 4 pooling on gfx950.
//
// Compiled once per window side k (-DCRF_BLUR_K=k).  The pooled grid has one
// cell per 4 x 4 pixels.  A work-group owns 8 x 8 cells (32 x 32 pixels) of
// one image and, in one launch:
//   1. stages the pooled Q_t and the pooled colours of its cells, a one-cell
//      ring around them and the r-cell window halo of that ring into LDS
//      (zero outside the grid; 16-byte loads where the grid rows allow);
//   2. computes the pooled message (Eq. 6 on the pooled grid, offsets of 4
//      pixels, Eq. 4 weights from pooled colours) for its 8 x 8 cells and the
//      one-cell ring that the bilinear upsampling of its pixels reads: one
//      wavefront per window row for k = 9, 11 (up to 21 classes, with or
//      without feature planes), else eight wavefronts taking rows w and w + 8 (the first 512
//      threads also own the pixels); a lane holds the
//      rows' weights of four horizontally adjacent cells in registers and
//      reads each staged row once (16-byte reads) for all four, the two
//      halves of a wavefront taking the even and the odd classes; the k row
//      partials are summed in LDS (all classes at once where they fit, else a
//      chunk at a time).  The unary of its 1024 pixels is prefetched into
//      registers under this step;
//   3. per pixel: bilinear upsampling of the message (half-pixel centres,
//      edge clamp), compatibility, unary and softmax (Alg. 1), then the
//      full-resolution Q (the last iteration), its 4 x 4 cell average (the
//      pooled Q_{t+1} the next launch reads), or both (every round of the
//      reverse mode's recompute, which keeps Q^t and its pooled form).
// So each iteration reads the unary once and the pooled state, and the
// pooled message is never written to memory.  The first iteration's input,
// softmax(U), the image and the learnable features averaged over the cells,
// comes from one initialisation launch (blur_init_kernel).
#include "crf_internal.h"

#ifndef CRF_BLUR_K
#error "compile with -DCRF_BLUR_K=<odd window side>"
#endif

namespace convcrf {
namespace {

constexpr int kS = kFusedBlurFactor;          // pixels per cell side
constexpr int kNC = kFusedBlurCells;          // own cells per work-group side
constexpr int kMT = kNC + 2;                  // message tile side: own cells and a ring of one

template <int K, int CM, bool FT>
struct BlurShape {
    static constexpr int R = (K - 1) / 2;
    static constexpr int FS = kMT + 2 * R;                  // footprint side (cells)
    static constexpr int FP = FS * FS;
    static constexpr int LS = kFusedBlurRowStride;          // LDS row stride (floats)
    static constexpr int FPL = FS * LS;                     // LDS plane (floats)
    static_assert(LS >= FS && LS % 2 == 0, "whole 8-byte rows");
    // one wavefront per window row for k = 9, 11 (three per SIMD, so at
    // most 168 VGPRs: up to 21 classes, with or without feature planes),
    // else eight; the first NPIX threads also own the pixels
    static constexpr int NWAVE = K > 8 && K <= 11 && CM <= 21 ? K : 8;
    static constexpr int FD = FT ? kMaxFeat : 0;           // staged feature planes
    static constexpr int NT = 64 * NWAVE;                  // threads
    static constexpr int RW = (K + NWAVE - 1) / NWAVE;     // window rows per wave
    static constexpr int NPIX = kNC * kNC * 8;             // threads with two pixels each
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

// VEC: 16-byte staging loads (Wp a multiple of 4, 16-byte aligned planes):
// each footprint row is read as whole float4s of its grid row, which never
// straddle the grid's edges, and shifted into place in LDS.
// FT: learnable smoothness features (the "+T" variant): D <= kMaxFeat pooled
// feature planes are staged after the colours (planes past D read zero) and
// the smoothness Gaussian of a tap is w_smooth exp(-|F_p - F_q|^2 / 2 theta_gamma^2)
// on them instead of the per-offset constant.
template <int K, int CM, bool EXACT, bool VEC, bool FT>
__global__ __launch_bounds__((BlurShape<K, CM, FT>::NT)) void blur_iter_kernel(const BlurIterArgs a) {
    using BS = BlurShape<K, CM, FT>;
    constexpr int FD = BS::FD;
    constexpr int NAUX = 3 + FD;                   // colour and feature planes
    constexpr int R = BS::R, FS = BS::FS, FP = BS::FP, NT = BS::NT, RW = BS::RW;
    constexpr int LS = BS::LS, FPL = BS::FPL;
    constexpr int MTC = kMT * kMT;
    constexpr int NW = K + 1;                      // footprint cells one lane's row reads (even)
    constexpr int kChunk = blur_iter_chunk(K, CM, FD); // classes per row-partial round
    constexpr int kSlots = blur_iter_slots(K, CM, FD); // its class slots (even)
    constexpr int MTCP = kFusedBlurPartStride;     // row-partial plane (floats)
    static_assert(NW % 2 == 0 && FS % 2 == 0 && FP % 2 == 0, "8-byte rows");
    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qf = smem;                        // [CM][FS][LS] pooled Q_t
    float* const Cf = Qf + CM * FPL;               // [3][FS][LS] pooled colours
    float* const Ff = Cf + 3 * FPL;                // [FD][FS][LS] pooled features (FT)
    float* const Pt = Ff + FD * FPL;               // [K][kSlots][MTCP] row partials
    float* const Mt = Pt + K * kSlots * MTCP;      // [CM][MTC] pooled message
    float* const Mu = Mt + CM * MTC;               // [CM][CM] compatibility, when given

    const int C = EXACT ? CM : a.C;
    const int Hp = a.Hp, Wp = a.Wp, H = a.H, W = a.W;
    const int b = blockIdx.z;
    const int cy0 = blockIdx.y * kNC, cx0 = blockIdx.x * kNC;     // first own cell
    const size_t HWp = (size_t)Hp * Wp, HW = (size_t)H * W;
    const int tid = threadIdx.x;

    // every thread owns two horizontally adjacent pixels, eight threads per
    // cell (cell-major, so that a cell's threads are consecutive lanes)
    static_assert(BS::NPIX == 512 && NT >= BS::NPIX, "two pixels per thread");
    const bool pix_thread = tid < BS::NPIX;            // uniform over the wavefront
    const int ci = tid >> 3, jj = tid & 7;
    const int ccy = cy0 + ci / kNC, ccx = cx0 + ci % kNC;           // own cell
    const int py = ccy * kS + (jj >> 1), px = ccx * kS + 2 * (jj & 1);
    const bool pix_ok = pix_thread && ccy < Hp && ccx < Wp;         // H, W multiples of kS
    // unary prefetch, issued after the window weights (under the message,
    // which needs none of it; issued with the staging loads it would compete
    // with them); every load is issued (planes past C read plane 0 and are
    // ignored)
    float u0[CM], u1[CM];
    const auto load_unary = [&] {
        const float* up = a.unary + (size_t)b * a.C * HW + (size_t)(pix_ok ? py : 0) * W +
                          (pix_ok ? px : 0);
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            const float2 t =
                *reinterpret_cast<const float2*>(up + (size_t)(EXACT || c < C ? c : 0) * HW);
            u0[c] = t.x;
            u1[c] = t.y;
        }
    };

    // the tap constants of this wavefront's window rows, read into scalar
    // registers now so that their latency passes under the staging (rows past
    // the window read row k - 1's and are not used)
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    float tca[RW][K], tcs[RW][K];
#pragma unroll
    for (int j = 0; j < RW; ++j) {
        const int dy = wave + BS::NWAVE * j < K ? wave + BS::NWAVE * j : K - 1;
#pragma unroll
        for (int dx = 0; dx < K; ++dx) {
            const int n = (dx - R) * (dx - R) + (dy - R) * (dy - R);
            tca[j][dx] = a.taps.app_log2[n];
            tcs[j][dx] = a.taps.smooth[n];
            asm volatile("" : "+s"(tca[j][dx]), "+s"(tcs[j][dx]));
        }
    }

    // ---- staging loads (pooled Q_t and colours over the footprint, zero
    // outside the grid), all issued before any LDS store
    const float* __restrict__ qsrc = a.qbar + (size_t)b * a.C * HWp;
    const float* __restrict__ csrc = a.pcol + (size_t)b * 3 * HWp;
    const float* __restrict__ fsrc = FT ? a.sfeat + (size_t)b * a.D * HWp : csrc;
    // plane pl of the staged block: Q (pl < CM), colours, features (FT)
    const auto plane_src = [&](int pl) {
        return pl < CM ? qsrc + (size_t)pl * HWp
                       : (pl < CM + 3 ? csrc + (size_t)(pl - CM) * HWp
                                      : fsrc + (size_t)(pl - CM - 3) * HWp);
    };
    const auto plane_ok = [&](int pl) {
        return pl < CM ? (EXACT || pl < C) : (pl < CM + 3 || pl - CM - 3 < a.D);
    };
    if constexpr (VEC) {
        constexpr int RA = (R + 1 + 3) / 4 * 4;         // left halo (R + 1) in whole float4s
        constexpr int OFF = RA - (R + 1);               // LDS column = 4 f + e - OFF
        constexpr int NV = (RA + kNC + 1 + R + 3) / 4;  // float4s per footprint row
        constexpr int NSTV = (CM + NAUX) * FS * NV;
        constexpr int PER = (NSTV + NT - 1) / NT;
        static_assert(kNC % 4 == 0 && 4 * NV - OFF >= FS, "the float4s cover the footprint");
        float4 v[PER];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int idx = tid + j * NT;
            const int pl = idx / (FS * NV), rem = idx - pl * (FS * NV);
            const int r = rem / NV, f = rem - r * NV;
            const int gy = cy0 - 1 - R + r, gx = cx0 - RA + 4 * f;
            const bool in =
                idx < NSTV && plane_ok(pl) && gy >= 0 && gy < Hp && gx >= 0 && gx < Wp;
            const size_t g = in ? (size_t)gy * Wp + gx : 0;
            v[j] = in ? *reinterpret_cast<const float4*>(plane_src(in ? pl : 0) + g)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int idx = tid + j * NT;
            if (idx >= NSTV) continue;
            const int pl = idx / (FS * NV), rem = idx - pl * (FS * NV);
            const int r = rem / NV, f = rem - r * NV;
            float* row = smem + pl * FPL + r * LS;
            const float e4[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int col = 4 * f + e - OFF;
                if (col >= 0 && col < FS) row[col] = e4[e];
            }
        }
    } else {
        constexpr int NST = (CM + NAUX) * FP;
        constexpr int PER = (NST + NT - 1) / NT;
        float v[PER];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int idx = tid + j * NT;
            const int pl = idx / FP, rem = idx - pl * FP;
            const int r = rem / FS, cc = rem - r * FS;
            const int gy = cy0 - 1 - R + r, gx = cx0 - 1 - R + cc;
            const bool in =
                idx < NST && plane_ok(pl) && gy >= 0 && gy < Hp && gx >= 0 && gx < Wp;
            const size_t g = in ? (size_t)gy * Wp + gx : 0;
            v[j] = in ? plane_src(in ? pl : 0)[g] : 0.f;
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int idx = tid + j * NT;
            if (idx >= NST) continue;
            const int pl = idx / FP, rem = idx - pl * FP;
            const int r = rem / FS, cc = rem - r * FS;
            smem[pl * FPL + r * LS + cc] = v[j];
        }
    }
    if (a.mu)
        for (int i = tid; i < C * C; i += NT) Mu[(i / C) * CM + i % C] = a.mu[i];
    __syncthreads();

    // ---- pooled message: wavefront w takes window rows w + NWAVE j (j < RW).
    // Lane (h, mi, qd): half h = lane / 32 takes the classes of parity h,
    // (mi, qd) the four cells (mi, 4 qd + i), i < 4, of the 10 x 10 message
    // tile (qd = 2 computes two cells past the tile, which are discarded), so
    // one 16-byte-aligned row read of k + 3 staged values feeds 4k FMAs and a
    // wavefront instruction serves two classes.
    const int lane = tid & 63;
    const int h = lane >> 5, sub = lane & 31;
    const bool msg = sub < 3 * kMT;
    const int mi = msg ? sub / 3 : 0, qd = msg ? sub % 3 : 0, mj = 4 * qd;
    constexpr int QW = (K + 3 + 3) / 4 * 4;       // staged values one row read covers
    static_assert(kMT == 10 && LS % 4 == 0 && LS >= 8 + QW, "16-byte reads inside a staged row");
    // window weights of the lane's four cells: this half computes cells
    // 2h, 2h + 1 and takes the other two from its partner lane (lane ^ 32,
    // the same cells in the other half)
    float w[RW][4][K];
    if (msg) {
        // own colours (and features, FT) of the lane's two cells: the colour
        // and feature planes follow each other in LDS
        float own[NAUX][2];
#pragma unroll
        for (int ch = 0; ch < NAUX; ++ch)
#pragma unroll
            for (int i = 0; i < 2; ++i)
                own[ch][i] = Cf[ch * FPL + (mi + R) * LS + mj + 2 * h + R + i];
#pragma unroll
        for (int j = 0; j < RW; ++j) {
            const int dy = wave + BS::NWAVE * j;
            if (dy >= K) continue;
            float nc[NAUX][NW];
#pragma unroll
            for (int ch = 0; ch < NAUX; ++ch) {
                const float2* r2 =
                    reinterpret_cast<const float2*>(Cf + ch * FPL + (mi + dy) * LS + mj + 2 * h);
#pragma unroll
                for (int x = 0; x < NW / 2; ++x) {
                    const float2 t = r2[x];
                    nc[ch][2 * x] = t.x;
                    nc[ch][2 * x + 1] = t.y;
                }
            }
#pragma unroll
            for (int i = 0; i < 2; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    float smo = tcs[j][dx];
                    if constexpr (FT) {
                        float fd2 = 0.f;
#pragma unroll
                        for (int d = 0; d < FD; ++d) {
                            const float e = own[3 + d][i] - nc[3 + d][i + dx];
                            fd2 = fmaf(e, e, fd2);
                        }
                        smo = a.w_smooth * __builtin_amdgcn_exp2f(a.neg_gamma * fd2);
                    }
                    const float k =
                        __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, tca[j][dx])) + smo;
                    // the centre tap: excluded, or K(p, p) when included
                    const float mine =
                        (dy == R && dx == R) ? (a.include_center ? a.center_w : 0.f) : k;
                    // the partner's value by v_permlane32_swap of (mine, mine); both
                    // results are read through h, which is right whether the two
                    // operands get one register (both results then the swapped
                    // value) or two (lanes 0..31 of the first and 32..63 of the
                    // second unchanged, the other halves swapped)
                    const auto sw = __builtin_amdgcn_permlane32_swap(
                        __builtin_bit_cast(unsigned, mine), __builtin_bit_cast(unsigned, mine),
                        false, false);
                    const float other = __builtin_bit_cast(float, h ? sw[0] : sw[1]);
                    w[j][i][dx] = h ? other : mine;
                    w[j][2 + i][dx] = h ? mine : other;
                }
            }
        }
    }
    if (pix_thread) load_unary();
    for (int c0 = 0; c0 < C; c0 += kChunk) {
        const int cn = C - c0 < kChunk ? C - c0 : kChunk;
        if (msg) {
#pragma unroll
            for (int j = 0; j < RW; ++j) {
                const int dy = wave + BS::NWAVE * j;   // uniform over the wavefront
                if (dy >= K) continue;
                // class slots cl = 2 t + h of the chunk, straight-line, the row
                // of slot t + 1 read while slot t is summed (slots past C read a
                // zero or unused plane; their partials are never summed)
                const auto load_row = [&](int t, float (&q)[QW]) {
                    const int cl = 2 * t + h;
                    const int c = c0 + cl < CM ? c0 + cl : CM - 1;
                    const float4* row =
                        reinterpret_cast<const float4*>(Qf + c * FPL + (mi + dy) * LS + mj);
#pragma unroll
                    for (int x = 0; x < QW / 4; ++x) {
                        const float4 v4 = row[x];
                        q[4 * x] = v4.x;
                        q[4 * x + 1] = v4.y;
                        q[4 * x + 2] = v4.z;
                        q[4 * x + 3] = v4.w;
                    }
                };
                constexpr int NSL = kSlots / 2;
                float qb[2][QW];
                load_row(0, qb[0]);
                // the second pair of cells of qd = 2 lies past the tile: its
                // partials go to the plane's spare floats
                const int far = (qd < 2 ? mi * kMT + mj + 2 : MTC);
#pragma unroll
                for (int t = 0; t < NSL; ++t) {
                    if (t + 1 < NSL) load_row(t + 1, qb[(t + 1) & 1]);
                    // keep those reads above the FMAs
                    __builtin_amdgcn_sched_barrier(0);
                    const float (&q)[QW] = qb[t & 1];
                    float m[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int dx = 0; dx < K; ++dx)
#pragma unroll
                        for (int i = 0; i < 4; ++i) m[i] = fmaf(w[j][i][dx], q[i + dx], m[i]);
                    float* pp = Pt + (dy * kSlots + 2 * t + h) * MTCP;
                    *reinterpret_cast<float2*>(pp + mi * kMT + mj) = make_float2(m[0], m[1]);
                    *reinterpret_cast<float2*>(pp + far) = make_float2(m[2], m[3]);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
        __syncthreads();
        for (int i = tid; i < cn * MTC; i += NT) {
            const int cl = i / MTC, cell = i - cl * MTC;
            float m = 0.f;
#pragma unroll
            for (int r = 0; r < K; ++r) m += Pt[(r * kSlots + cl) * MTCP + cell];
            Mt[(c0 + cl) * MTC + cell] = m;
        }
        __syncthreads();
    }
    // the message-only wavefronts are done (no barrier follows)
    if (!pix_thread) return;

    // ---- per pixel: bilinear message, compatibility, unary, softmax
    // both pixels of a lane lie in the same half of their cell (px is even),
    // so they have the same two source columns and differ only in the
    // horizontal fraction
    int ya, yb, xa, xb, xa1, xb1;
    float fy, fx0, fx1;
    src_coord(py, Hp, ya, yb, fy);
    src_coord(px, Wp, xa, xb, fx0);
    src_coord(px + 1, Wp, xa1, xb1, fx1);
    // message-tile coordinates of the four taps (the ring covers them)
    const int ty0 = ya - (cy0 - 1), ty1 = yb - (cy0 - 1);
    const int o00 = ty0 * kMT + xa - (cx0 - 1), o10 = ty1 * kMT + xa - (cx0 - 1);
    float z0[CM], z1[CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) {
            z0[c] = z1[c] = 0.f;
            continue;
        }
        // the two source columns are adjacent, or one column at the right
        // edge (the ring keeps o00 + 1 inside the tile row): paired reads
        const float* m = Mt + c * MTC;
        const float a00 = m[o00], n01 = m[o00 + 1], a10 = m[o10], n11 = m[o10 + 1];
        const float a01 = xb != xa ? n01 : a00, a11 = xb != xa ? n11 : a10;
        const float d0 = a01 - a00, d1 = a11 - a10;
        const float t0 = fmaf(fx0, d0, a00), b0 = fmaf(fx0, d1, a10);
        const float t1 = fmaf(fx1, d0, a00), b1 = fmaf(fx1, d1, a10);
        z0[c] = fmaf(fy, b0 - t0, t0);
        z1[c] = fmaf(fy, b1 - t1, t1);
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
    if (a.q_full && pix_ok) {
        float* q = a.q_full + (size_t)b * a.C * HW + (size_t)py * W + px;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C)
                *reinterpret_cast<float2*>(q + (size_t)c * HW) = make_float2(z0[c], z1[c]);
    }
    if (!a.qbar_out) return;   // uniform over the grid
    // the cell's 16 pixels: two per lane, eight consecutive lanes
    float* dq = a.qbar_out + (size_t)b * a.C * HWp + (size_t)(pix_ok ? ccy : 0) * Wp +
                (pix_ok ? ccx : 0);
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        const float t = cell_sum8(z0[c] + z1[c]);
        if (jj == 4 && pix_ok) dq[(size_t)c * HWp] = t * (1.0f / (kS * kS));
    }
}

template <int K, int CM, bool EXACT, bool VEC, bool FT>
hipError_t launch_vec(const BlurIterArgs& a, hipStream_t stream) {
    const size_t lds = blur_iter_lds_bytes(K, CM, a.mu != nullptr, FT ? kMaxFeat : 0);
    auto fn = blur_iter_kernel<K, CM, EXACT, VEC, FT>;
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    const dim3 grid((a.Wp + kNC - 1) / kNC, (a.Hp + kNC - 1) / kNC, a.B);
    hipLaunchKernelGGL(fn, grid, dim3(BlurShape<K, CM, FT>::NT), lds, stream, a);
    return hipGetLastError();
}

template <int K, int CM, bool EXACT, bool FT>
hipError_t launch_ft(const BlurIterArgs& a, hipStream_t stream) {
    const auto al16 = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 == 0; };
    if (a.Wp % 4 == 0 && al16(a.qbar) && al16(a.pcol) && (!FT || al16(a.sfeat)))
        return launch_vec<K, CM, EXACT, true, FT>(a, stream);
    return launch_vec<K, CM, EXACT, false, FT>(a, stream);
}

template <int K, int CM, bool EXACT>
hipError_t launch_one(const BlurIterArgs& a, hipStream_t stream) {
    if (a.D > 0) return launch_ft<K, CM, EXACT, true>(a, stream);
    return launch_ft<K, CM, EXACT, false>(a, stream);
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
            a.B > 65535 || a.Hp > 65535 * kNC || a.D < 0 || a.D > kMaxFeat ||
            (a.D > 0 && !a.sfeat) || (!a.q_full && !a.qbar_out))
            return hipErrorInvalidValue;
        switch (a.C) {
            case 19: return launch_one<K, 19, true>(a, stream);
            case 21: return launch_one<K, 21, true>(a, stream);
            default: break;
        }
        if (a.C <= 8) return launch_one<K, 8, false>(a, stream);
        return launch_one<K, 24, false>(a, stream);
    }
}

}  // namespace convcrf
