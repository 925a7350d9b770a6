// iter.hip -- one mean-field iteration of a Convolutional CRF on gfx950.
//
// Compiled once per window side k (-DCRF_K=k).  One work-group owns a tile
// of 32 x rows output pixels of one image; it stages Q_t (or softmax(U) on the
// first iteration, Alg. 1 initialisation) and the colour planes of the tile
// plus an r-pixel halo in LDS, with zeros outside the image, so that
// neighbours outside the image contribute nothing to the message.  Each
// thread owns 4 horizontally adjacent pixels and keeps their C-class
// messages in registers.  For every window row it
//   1. recomputes the merged Gaussian weights K(p, p + d) of its 4 pixels
//      (Eq. 4, merged as in Sec. 4.1) from the staged colours -- the kernel
//      matrix of Eq. 5 is never written to memory -- and
//   2. for each class, reads the 4 + k - 1 staged Q values of that row once
//      and applies them to all 4 pixels (the locally-connected,
//      channel-constant filter of Eq. 6), one FMA per (pixel, tap, class).
// The epilogue applies the compatibility transform, adds the unary and
// normalises with a softmax (Alg. 1), writing Q_{t+1}; in message mode (the
// pooled message of the blur path, Sec. 4.2) it writes the raw message.
//
// The materialised variant reads the weights from a precomputed kernel
// matrix instead of step 1 (the two-stage structure of Sec. 4.1).

#include "crf_internal.h"

#ifndef CRF_K
#error "compile with -DCRF_K=<odd window side>"
#endif

namespace convcrf {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

// N consecutive floats from a 16-byte aligned LDS address (N even).
template <int N>
__device__ __forceinline__ void lds_row(const float* p, float (&v)[N]) {
    static_assert(N % 2 == 0, "row length must be even");
#pragma unroll
    for (int j = 0; j + 4 <= N; j += 4) {
        const float4 t = *reinterpret_cast<const float4*>(p + j);
        v[j] = t.x;
        v[j + 1] = t.y;
        v[j + 2] = t.z;
        v[j + 3] = t.w;
    }
    if constexpr (N % 4 == 2) {
        const float2 t = *reinterpret_cast<const float2*>(p + N - 2);
        v[N - 2] = t.x;
        v[N - 1] = t.y;
    }
}

// In-register softmax over the first C of CM values (max subtracted).
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

template <int K, int CM, bool EXACT, bool MAT>
__global__ __launch_bounds__(256) void iter_kernel(const IterArgs a) {
    constexpr int R = (K - 1) / 2;
    constexpr int LW = kTileW + 2 * R;
    constexpr int LS = (LW + 3) & ~3;
    constexpr int NW = kPix + K - 1;          // staged values per window row
    constexpr int KK = K * K;
    constexpr int CTR = R * K + R;            // centre tap index

    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);

    const int C = EXACT ? CM : a.C;
    const int H = a.H, W = a.W;
    const int nthreads = blockDim.x;
    const int rows = nthreads / kThreadsPerRow;
    const int LH = rows + 2 * R;
    const int plane = LH * LS;

    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * rows;
    const int x0 = (trem - tyi * a.tiles_x) * kTileW;

    const size_t HW = (size_t)H * W;
    const float* __restrict__ src = a.src + (size_t)b * C * HW;
    const float* __restrict__ feat = a.feat + (size_t)b * 3 * HW;

    float* const Qs = smem;                   // [C][LH][LS]
    float* const Cs = smem + C * plane;       // [3][LH][LS]

    // ---- stage Q_t (or softmax(U)) and colours, tile + halo, zero outside
    const int tid = threadIdx.x;
    const int nstage = LH * LW;
    for (int idx = tid; idx < nstage; idx += nthreads) {
        const int r = idx / LW;
        const int cc = idx - r * LW;
        const int gy = y0 - R + r;
        const int gx = x0 - R + cc;
        const bool inb = gy >= 0 && gy < H && gx >= 0 && gx < W;
        const size_t g = inb ? (size_t)gy * W + gx : 0;
        const int l = r * LS + cc;
        if (a.first) {
            float v[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c)
                v[c] = (inb && (EXACT || c < C)) ? src[c * HW + g] : 0.f;
            if (inb) softmax_regs<CM, EXACT>(v, C);
#pragma unroll
            for (int c = 0; c < CM; ++c)
                if (EXACT || c < C) Qs[c * plane + l] = v[c];
        } else {
#pragma unroll 4
            for (int c = 0; c < C; ++c) Qs[c * plane + l] = inb ? src[c * HW + g] : 0.f;
        }
        if constexpr (!MAT) {
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) Cs[ch * plane + l] = inb ? feat[ch * HW + g] : 0.f;
        }
    }
    __syncthreads();

    // ---- message: acc[i][c] = sum_d K(p_i, p_i + d) Q_t(p_i + d, c)
    const int tx = tid % kThreadsPerRow;
    const int ty = tid / kThreadsPerRow;
    const int col0 = tx * kPix;               // first staged column read
    const int y = y0 + ty;
    const int xb = x0 + col0;

    float acc[kPix][CM];
#pragma unroll
    for (int i = 0; i < kPix; ++i)
#pragma unroll
        for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;

    float own[3][kPix];
    if constexpr (!MAT) {
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            const float* p = Cs + ch * plane + (ty + R) * LS + col0 + R;
#pragma unroll
            for (int i = 0; i < kPix; ++i) own[ch][i] = p[i];
        }
    }
    const float* __restrict__ kmat =
        MAT ? a.kmat + (size_t)b * (KK - 1) * HW : nullptr;
    const bool pix_ok = y < H;

    // one window row of the message; unrolled over rows on the fused exact-C
    // path, rolled where the fully unrolled body would exceed the registers
    constexpr bool kUnrollRows = !MAT && (EXACT || CM <= 16) && K <= 9;
    auto window_row = [&](const int dy) {
        const int row = ty + dy;
        float w[kPix][K];
        if constexpr (!MAT) {
            float nc[3][NW];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) lds_row<NW>(Cs + ch * plane + row * LS + col0, nc[ch]);
#pragma unroll
            for (int i = 0; i < kPix; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    const int t = dy * K + dx;
                    if (t == CTR) { w[i][dx] = 0.f; continue; }
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    w[i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[t])) +
                               a.taps.smooth[t];
                }
            }
        } else {
#pragma unroll
            for (int dx = 0; dx < K; ++dx) {
                const int t = dy * K + dx;
                if (t == CTR) {
#pragma unroll
                    for (int i = 0; i < kPix; ++i) w[i][dx] = 0.f;
                    continue;
                }
                const int pl = t < CTR ? t : t - 1;
                const float* kp = kmat + (size_t)pl * HW + (size_t)y * W + xb;
                if (a.vec4 && pix_ok && xb + kPix <= W) {
                    const float4 v = *reinterpret_cast<const float4*>(kp);
                    w[0][dx] = v.x;
                    w[1][dx] = v.y;
                    w[2][dx] = v.z;
                    w[3][dx] = v.w;
                } else {
#pragma unroll
                    for (int i = 0; i < kPix; ++i)
                        w[i][dx] = (pix_ok && xb + i < W) ? kp[i] : 0.f;
                }
            }
        }
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            if (EXACT || c < C) {
                float q[NW];
                lds_row<NW>(Qs + c * plane + row * LS + col0, q);
#pragma unroll
                for (int i = 0; i < kPix; ++i)
#pragma unroll
                    for (int dx = 0; dx < K; ++dx)
                        // the centre weight is 0; unrolled rows skip its FMA outright
                        if (!kUnrollRows || dy * K + dx != CTR)
                            acc[i][c] = fmaf(w[i][dx], q[i + dx], acc[i][c]);
            }
        }
    };
    if constexpr (kUnrollRows) {
#pragma unroll
        for (int dy = 0; dy < K; ++dy) window_row(dy);
    } else {
#pragma unroll 1
        for (int dy = 0; dy < K; ++dy) window_row(dy);
    }
    if (a.include_center) {
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            if (EXACT || c < C) {
                const float* p = Qs + c * plane + (ty + R) * LS + col0 + R;
#pragma unroll
                for (int i = 0; i < kPix; ++i) acc[i][c] = fmaf(a.center_w, p[i], acc[i][c]);
            }
        }
    }

    if (!pix_ok) return;
    const bool full4 = a.vec4 && xb + kPix <= W;
    float* __restrict__ dst = a.dst + (size_t)b * C * HW + (size_t)y * W + xb;

    if (a.mode == kModeUpdate) {
        // compatibility transform: acc <- -mu * M  (Potts: +M, which differs
        // from -(sum M - M) by a per-pixel constant the softmax removes)
        if (a.mu != nullptr) {
            const float* __restrict__ mu = a.mu;
#pragma unroll
            for (int i = 0; i < kPix; ++i) {
                float z[CM];
#pragma unroll
                for (int l = 0; l < CM; ++l) {
                    float t = 0.f;
                    if (EXACT || l < C) {
#pragma unroll
                        for (int lp = 0; lp < CM; ++lp)
                            if (EXACT || lp < C) t = fmaf(mu[l * C + lp], acc[i][lp], t);
                    }
                    z[l] = -t;
                }
#pragma unroll
                for (int l = 0; l < CM; ++l) acc[i][l] = z[l];
            }
        }
        // + unary
        const float* __restrict__ u = a.unary + (size_t)b * C * HW + (size_t)y * W + xb;
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            if (!EXACT && c >= C) continue;
            if (full4) {
                const float4 v = *reinterpret_cast<const float4*>(u + c * HW);
                acc[0][c] += v.x;
                acc[1][c] += v.y;
                acc[2][c] += v.z;
                acc[3][c] += v.w;
            } else {
#pragma unroll
                for (int i = 0; i < kPix; ++i)
                    if (xb + i < W) acc[i][c] += u[c * HW + i];
            }
        }
#pragma unroll
        for (int i = 0; i < kPix; ++i) softmax_regs<CM, EXACT>(acc[i], C);
    }

#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        if (full4) {
            *reinterpret_cast<float4*>(dst + c * HW) =
                make_float4(acc[0][c], acc[1][c], acc[2][c], acc[3][c]);
        } else {
#pragma unroll
            for (int i = 0; i < kPix; ++i)
                if (xb + i < W) dst[c * HW + i] = acc[i][c];
        }
    }
}

// Opt a kernel into the full 160 KB of LDS once per device.
template <typename Fn>
hipError_t allow_full_lds(Fn fn) {
    static unsigned long long done = 0;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const unsigned long long bit = 1ull << (dev & 63);
    if (done & bit) return hipSuccess;
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                            hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
    if (e == hipSuccess) done |= bit;
    return e;
}

template <int K, int CM, bool EXACT, bool MAT>
hipError_t launch_one(const IterArgs& a, int rows, size_t lds, hipStream_t stream) {
    auto fn = iter_kernel<K, CM, EXACT, MAT>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(kThreadsPerRow * rows), lds, stream, a);
    return hipGetLastError();
}

template <int K, int CM, bool EXACT>
hipError_t launch_cm(const IterArgs& a, bool mat, int rows, size_t lds, hipStream_t stream) {
    return mat ? launch_one<K, CM, EXACT, true>(a, rows, lds, stream)
               : launch_one<K, CM, EXACT, false>(a, rows, lds, stream);
}

}  // namespace

#define CRF_CAT2(a, b) a##b
#define CRF_CAT(a, b) CRF_CAT2(a, b)

hipError_t CRF_CAT(launch_iter_k, CRF_K)(const IterArgs& a, bool materialised, int rows,
                                         size_t lds, hipStream_t stream) {
    constexpr int K = CRF_K;
    switch (a.C) {
        case 19: return launch_cm<K, 19, true>(a, materialised, rows, lds, stream);
        case 21: return launch_cm<K, 21, true>(a, materialised, rows, lds, stream);
        default: break;
    }
    if (a.C <= 4) return launch_cm<K, 4, false>(a, materialised, rows, lds, stream);
    if (a.C <= 8) return launch_cm<K, 8, false>(a, materialised, rows, lds, stream);
    if (a.C <= 16) return launch_cm<K, 16, false>(a, materialised, rows, lds, stream);
    return launch_cm<K, 24, false>(a, materialised, rows, lds, stream);
}

}  // namespace convcrf
