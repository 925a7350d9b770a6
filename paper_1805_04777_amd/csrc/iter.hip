// iter.hip -- one mean-field iteration of a Convolutional CRF on gfx950.
//
// Compiled once per window side k (-DCRF_K=k).  One work-group owns a tile
// of 32 x rows output pixels of one image; it stages Q_t (or softmax(U) on the
// first iteration, Alg. 1 initialisation) and the colour planes of the tile
// plus an r-pixel halo in LDS, with zeros outside the image, so that
// neighbours outside the image contribute nothing to the message.  Each
// thread owns P (2 or 4) horizontally adjacent pixels and keeps their C-class
// messages in registers.  For every window row it
//   1. recomputes the merged Gaussian weights K(p, p + d) of its P pixels
//      (Eq. 4, merged as in Sec. 4.1) from the staged colours -- the kernel
//      matrix of Eq. 5 is never written to memory -- and
//   2. for each class, reads the P + k - 1 staged Q values of that row once
//      and applies them to all P pixels (the locally-connected,
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

// P floats as one vector (P = 2 or 4).
template <int P>
struct Vec;
template <>
struct Vec<2> {
    using T = float2;
    __device__ static void get(const T& v, float* o) { o[0] = v.x; o[1] = v.y; }
    __device__ static T make(const float* i) { return make_float2(i[0], i[1]); }
};
template <>
struct Vec<4> {
    using T = float4;
    __device__ static void get(const T& v, float* o) {
        o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
    }
    __device__ static T make(const float* i) { return make_float4(i[0], i[1], i[2], i[3]); }
};

// N consecutive floats from an LDS address aligned to 4*A bytes (A = 2 or
// 4, N even): A-wide vector reads plus a 2-wide tail.
template <int N, int A>
__device__ __forceinline__ void lds_row(const float* p, float (&v)[N]) {
    static_assert(N % 2 == 0, "row length must be even");
    if constexpr (A == 4) {
#pragma unroll
        for (int j = 0; j + 4 <= N; j += 4) {
            const float4 t = *reinterpret_cast<const float4*>(p + j);
            v[j] = t.x;
            v[j + 1] = t.y;
            v[j + 2] = t.z;
            v[j + 3] = t.w;
        }
    }
    constexpr int done = A == 4 ? N / 4 * 4 : 0;
#pragma unroll
    for (int j = done; j < N; j += 2) {
        const float2 t = *reinterpret_cast<const float2*>(p + j);
        v[j] = t.x;
        v[j + 1] = t.y;
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

template <int K, int CM, bool EXACT, bool MAT, int P>
// P = 4: 256 threads and a 146 KB tile, one wave per SIMD; P = 2: 512
// threads, two waves per SIMD.  Declaring that occupancy lets the scheduler
// spend registers on keeping LDS reads in flight.
__global__ __launch_bounds__(P == 4 ? 256 : 512)
__attribute__((amdgpu_waves_per_eu(P == 4 ? 1 : 2, P == 4 ? 1 : 2)))
void iter_kernel(const IterArgs a) {
    constexpr int R = (K - 1) / 2;
    constexpr int LW = kTileW + 2 * R;        // staged columns
    constexpr int LS = iter_lds_stride(K, P);
    constexpr int NW = P + K - 1;             // staged values per window row
    constexpr int KK = K * K;
    constexpr int CTR = R * K + R;            // centre tap index
    constexpr int TPR = kTileW / P;           // threads per tile row
    constexpr int kStagePix = 3;
    using V = Vec<P>;

    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);

    const int C = EXACT ? CM : a.C;
    const int H = a.H, W = a.W;
    const int nthreads = blockDim.x;
    const int rows = nthreads / TPR;
    const int LH = rows + 2 * R;
    const int plane = LH * LS;

    // the C planes of this thread's P pixels, zero beyond the right edge
    auto load_pixels = [&](float (&v)[P][CM], const float* g, int xb, bool fullv) {
        const size_t hw = (size_t)a.H * a.W;
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            if (!EXACT && c >= C) continue;
            if (fullv) {
                float tmp[P];
                V::get(*reinterpret_cast<const typename V::T*>(g + c * hw), tmp);
#pragma unroll
                for (int i = 0; i < P; ++i) v[i][c] = tmp[i];
            } else {
#pragma unroll
                for (int i = 0; i < P; ++i) v[i][c] = (xb + i < a.W) ? g[c * hw + i] : 0.f;
            }
        }
    };

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
    // compatibility matrix [C][C] (only when given; read back as broadcasts)
    float* const Ms = smem + (C + (MAT ? 0 : 3)) * plane;

    // ---- stage Q_t (or softmax(U)) and colours, tile + halo, zero outside.
    // kStagePix halo pixels per thread and round; every plane of all of them
    // is loaded into registers before any LDS store, so the loads overlap
    // (one round covers the whole halo tile at 512 threads).
    const int tid = threadIdx.x;
    const int nstage = LH * LW;
    auto stage_load = [&](int idx, float (&v)[CM], float (&f)[3]) {
        const int r = idx / LW;
        const int cc = idx - r * LW;
        const int gy = y0 - R + r;
        const int gx = x0 - R + cc;
        const bool inb = idx < nstage && gy >= 0 && gy < H && gx >= 0 && gx < W;
        const size_t g = inb ? (size_t)gy * W + gx : 0;
#pragma unroll
        for (int c = 0; c < CM; ++c)
            v[c] = (inb && (EXACT || c < C)) ? src[c * HW + g] : 0.f;
        if constexpr (!MAT) {
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) f[ch] = inb ? feat[ch * HW + g] : 0.f;
        }
        return inb;
    };
    auto stage_store = [&](int idx, float (&v)[CM], const float (&f)[3], bool inb) {
        if (idx >= nstage) return;
        const int r = idx / LW;
        const int l = r * LS + (idx - r * LW);
        if (a.first && inb) softmax_regs<CM, EXACT>(v, C);
#pragma unroll
        for (int c = 0; c < CM; ++c)
            if (EXACT || c < C) Qs[c * plane + l] = v[c];
        if constexpr (!MAT) {
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) Cs[ch * plane + l] = f[ch];
        }
    };
    const int tx = tid % TPR;
    const int ty = tid / TPR;
    const int col0 = tx * P;                  // first staged column read
    const int y = y0 + ty;
    const int xb = x0 + col0;
    const bool pix_ok = y < H;
    const bool fullv = a.vec && xb + P <= W;
    const bool general_compat = a.mode == kModeUpdate && a.mu != nullptr;

    // With Potts the update is softmax(U + M) (the compatibility transform
    // -(sum M - M) differs from +M by a per-pixel constant), so the message
    // accumulates straight onto the unary, which is loaded here and arrives
    // while the tile is being staged.
    const bool unary_first = a.mode == kModeUpdate && !general_compat;
    float acc[P][CM];
#pragma unroll
    for (int i = 0; i < P; ++i)
#pragma unroll
        for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;
    if (unary_first && pix_ok) load_pixels(acc, a.unary + (size_t)b * C * HW + (size_t)y * W + xb, xb, fullv);

    if (general_compat)
        for (int i = tid; i < C * C; i += nthreads) Ms[i] = a.mu[i];
    for (int idx = tid; idx < nstage; idx += kStagePix * nthreads) {
        float v[kStagePix][CM], f[kStagePix][3];
        bool in[kStagePix];
#pragma unroll
        for (int j = 0; j < kStagePix; ++j) in[j] = stage_load(idx + j * nthreads, v[j], f[j]);
#pragma unroll
        for (int j = 0; j < kStagePix; ++j) stage_store(idx + j * nthreads, v[j], f[j], in[j]);
    }
    __syncthreads();

    // ---- message: acc[i][c] = sum_d K(p_i, p_i + d) Q_t(p_i + d, c)

    float own[3][P];
    if constexpr (!MAT) {
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            const float* p = Cs + ch * plane + (ty + R) * LS + col0 + R;
#pragma unroll
            for (int i = 0; i < P; ++i) own[ch][i] = p[i];
        }
    }
    const float* __restrict__ kmat =
        MAT ? a.kmat + (size_t)b * (KK - 1) * HW : nullptr;

    // one window row of the message; unrolled over rows on the fused exact-C
    // path, rolled where the fully unrolled body would exceed the registers
    constexpr bool kUnrollRows = !MAT && (EXACT || CM <= 16) && K <= 9;
    auto window_row = [&](const int dy) {
        const int row = ty + dy;
        float w[P][K];
        if constexpr (!MAT) {
            float nc[3][NW];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch)
                lds_row<NW, P>(Cs + ch * plane + row * LS + col0, nc[ch]);
#pragma unroll
            for (int i = 0; i < P; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    const int t = dy * K + dx;
                    if (t == CTR) { w[i][dx] = 0.f; continue; }
                    const int n = (dx - R) * (dx - R) + (dy - R) * (dy - R);
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    w[i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[n])) +
                               a.taps.smooth[n];
                }
            }
        } else {
#pragma unroll
            for (int dx = 0; dx < K; ++dx) {
                const int t = dy * K + dx;
                if (t == CTR) {
#pragma unroll
                    for (int i = 0; i < P; ++i) w[i][dx] = 0.f;
                    continue;
                }
                const int pl = t < CTR ? t : t - 1;
                const float* kp = kmat + (size_t)pl * HW + (size_t)y * W + xb;
                if (pix_ok && fullv) {
                    float tmp[P];
                    V::get(*reinterpret_cast<const typename V::T*>(kp), tmp);
#pragma unroll
                    for (int i = 0; i < P; ++i) w[i][dx] = tmp[i];
                } else {
#pragma unroll
                    for (int i = 0; i < P; ++i)
                        w[i][dx] = (pix_ok && xb + i < W) ? kp[i] : 0.f;
                }
            }
        }
        // classes two at a time, the next row of Q read while the current
        // one is applied
        auto apply = [&](const float (&q)[NW], int c) {
#pragma unroll
            for (int i = 0; i < P; ++i)
#pragma unroll
                for (int dx = 0; dx < K; ++dx)
                    // the centre weight is 0; unrolled rows skip its FMA outright
                    if (!kUnrollRows || dy * K + dx != CTR)
                        acc[i][c] = fmaf(w[i][dx], q[i + dx], acc[i][c]);
        };
        const float* qrow = Qs + row * LS + col0;
        float qa[NW], qb[NW];
        lds_row<NW, P>(qrow, qa);
#pragma unroll
        for (int c = 0; c < CM; c += 2) {
            if (EXACT || c < C) {
                const bool has1 = c + 1 < CM && (EXACT || c + 1 < C);
                if (has1) lds_row<NW, P>(qrow + (c + 1) * plane, qb);
                apply(qa, c);
                if (has1) {
                    if (c + 2 < CM && (EXACT || c + 2 < C)) lds_row<NW, P>(qrow + (c + 2) * plane, qa);
                    apply(qb, c + 1);
                }
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
                for (int i = 0; i < P; ++i) acc[i][c] = fmaf(a.center_w, p[i], acc[i][c]);
            }
        }
    }

    if (!pix_ok) return;
    float* __restrict__ dst = a.dst + (size_t)b * C * HW + (size_t)y * W + xb;

    if (a.mode == kModeUpdate) {
        // compatibility transform: acc <- -mu * M (general mu only; with
        // Potts acc already holds U + M)
        if (general_compat) {
            // Z = U - mu M, one row of mu at a time (a scheduling barrier per
            // row keeps the broadcast reads of mu from all being hoisted);
            // the unary is loaded first so that it arrives meanwhile
            float u[P][CM];
            load_pixels(u, a.unary + (size_t)b * C * HW + (size_t)y * W + xb, xb, fullv);
            float z[P][CM];
#pragma unroll
            for (int l = 0; l < CM; ++l) {
                if (EXACT || l < C) {
                    float t[P];
#pragma unroll
                    for (int i = 0; i < P; ++i) t[i] = 0.f;
#pragma unroll
                    for (int lp = 0; lp < CM; ++lp) {
                        if (EXACT || lp < C) {
                            const float m = Ms[l * C + lp];
#pragma unroll
                            for (int i = 0; i < P; ++i) t[i] = fmaf(m, acc[i][lp], t[i]);
                        }
                    }
#pragma unroll
                    for (int i = 0; i < P; ++i) z[i][l] = u[i][l] - t[i];
                } else {
#pragma unroll
                    for (int i = 0; i < P; ++i) z[i][l] = 0.f;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int i = 0; i < P; ++i)
#pragma unroll
                for (int c = 0; c < CM; ++c) acc[i][c] = z[i][c];
        }
#pragma unroll
        for (int i = 0; i < P; ++i) softmax_regs<CM, EXACT>(acc[i], C);
    }

#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (!EXACT && c >= C) continue;
        if (fullv) {
            float tmp[P];
#pragma unroll
            for (int i = 0; i < P; ++i) tmp[i] = acc[i][c];
            *reinterpret_cast<typename V::T*>(dst + c * HW) = V::make(tmp);
        } else {
#pragma unroll
            for (int i = 0; i < P; ++i)
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

template <int K, int CM, bool EXACT, bool MAT, int P>
hipError_t launch_one(const IterArgs& a, TileConfig t, size_t lds, hipStream_t stream) {
    auto fn = iter_kernel<K, CM, EXACT, MAT, P>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(t.threads()), lds, stream, a);
    return hipGetLastError();
}

template <int K, int CM, bool EXACT>
hipError_t launch_cm(const IterArgs& a, bool mat, TileConfig t, size_t lds, hipStream_t stream) {
    if (t.pix == 2)
        return mat ? launch_one<K, CM, EXACT, true, 2>(a, t, lds, stream)
                   : launch_one<K, CM, EXACT, false, 2>(a, t, lds, stream);
    return mat ? launch_one<K, CM, EXACT, true, 4>(a, t, lds, stream)
               : launch_one<K, CM, EXACT, false, 4>(a, t, lds, stream);
}

}  // namespace

#define CRF_CAT2(a, b) a##b
#define CRF_CAT(a, b) CRF_CAT2(a, b)

hipError_t CRF_CAT(launch_iter_k, CRF_K)(const IterArgs& a, bool materialised, TileConfig tile,
                                         size_t lds, hipStream_t stream) {
    constexpr int K = CRF_K;
    if (tile.pix != 2 && tile.pix != 4) return hipErrorInvalidValue;
    if (tile.threads() > (tile.pix == 4 ? 256 : 512) || tile.threads() % 64 != 0)
        return hipErrorInvalidValue;
    switch (a.C) {
        case 19: return launch_cm<K, 19, true>(a, materialised, tile, lds, stream);
        case 21: return launch_cm<K, 21, true>(a, materialised, tile, lds, stream);
        default: break;
    }
    if (a.C <= 4) return launch_cm<K, 4, false>(a, materialised, tile, lds, stream);
    if (a.C <= 8) return launch_cm<K, 8, false>(a, materialised, tile, lds, stream);
    if (a.C <= 16) return launch_cm<K, 16, false>(a, materialised, tile, lds, stream);
    return launch_cm<K, 24, false>(a, materialised, tile, lds, stream);
}

}  // namespace convcrf
