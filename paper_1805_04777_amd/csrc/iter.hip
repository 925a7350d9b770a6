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
// normalises with a softmax (Alg. 1), writing Q_{t+1}.
//
// The materialised variant reads the weights from a precomputed kernel
// matrix instead of step 1 (the two-stage structure of Sec. 4.1).
//
// Also here: stream_kernel, the same update with the staging streamed under
// the computation; rstream_kernel, its resident form (all iterations in one
// launch); and pmsg_kernel, the message of the blur path on the pooled grid
// (Sec. 4.2).

#include "crf_internal.h"
#include "lds_dma.h"

#ifndef CRF_K
#error "compile with -DCRF_K=<odd window side>"
#endif

namespace convcrf {
namespace {


// P floats as one vector (P = 1, 2 or 4).
template <int P>
struct Vec;
template <>
struct Vec<1> {
    using T = float;
    __device__ static void get(const T& v, float* o) { o[0] = v; }
    __device__ static T make(const float* i) { return i[0]; }
};
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


// Neighbour synchronisation of a resident launch (every work-group
// co-resident).  A work-group depends only on the border rings of the up to
// eight tiles around it, so instead of a grid barrier each tile publishes
// how many rings it has written (flags[tile] = value) and waits until each
// neighbour has published `value`.  Ordering: every wave waits until its
// own ring stores are acknowledged by L2 (the work-group barrier alone does
// not wait for them), so that after the barrier one agent-scope release by
// thread 0 (an L2 write-back, for the tiles on other XCDs) covers the stores
// of the whole work-group before its flag store; the waiting lanes (one per
// neighbour) poll with relaxed loads and one agent-scope acquire drops stale
// cache lines before the work-group reads the rings.  With the rings double-buffered this also keeps a tile from
// overwriting a buffer a neighbour still reads: that neighbour publishes
// value + 1 only after its read.  The wait is bounded: past kSpinLimit polls
// the lane records an error in *flag_err and goes on (wrong results, never a
// hang).
constexpr unsigned int kSpinLimit = 1u << 22;
// s_waitcnt operand for vmcnt(0) alone on gfx9-family targets: vmcnt in bits
// 3:0 and 15:14 zero, expcnt (6:4) and lgkmcnt (11:8) at their maxima
constexpr int kWaitVmem = 0x0F70;

__device__ __forceinline__ void neighbour_sync(unsigned int* flags, unsigned int* flag_err,
                                               int tile, int tiles_x, int tiles_y,
                                               unsigned int value) {
    __builtin_amdgcn_s_waitcnt(kWaitVmem);
    __syncthreads();
    if (threadIdx.x == 0) {
        // the write-back must have finished before the flag is visible; the
        // compiler's own wait after it is dropped when no store is pending
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __builtin_amdgcn_s_waitcnt(kWaitVmem);
        __hip_atomic_store(flags + tile, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (threadIdx.x < 9) {
        const int per_img = tiles_x * tiles_y;
        const int ti = tile % per_img;
        const int ty = ti / tiles_x + (int)threadIdx.x / 3 - 1;
        const int tx = ti % tiles_x + (int)threadIdx.x % 3 - 1;
        if (threadIdx.x != 4 && ty >= 0 && ty < tiles_y && tx >= 0 && tx < tiles_x) {
            const unsigned int* f = flags + (tile - ti) + ty * tiles_x + tx;
            unsigned int polls = 0;
            while (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < value) {
                __builtin_amdgcn_s_sleep(1);
                if (++polls == kSpinLimit) {
                    __hip_atomic_store(flag_err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        __builtin_amdgcn_s_waitcnt(kWaitVmem);   // invalidation done before the barrier
    }
    __syncthreads();
}

// The same wait for data that every work-group writes and reads with
// agent-scope atomic accesses (coherent across the XCDs' L2 caches, written
// through): each wave waits until its stores are performed, the work-group
// barrier orders thread 0's flag store after all of them, and the readers'
// own atomic loads need no cache invalidation -- no L2 write-back or
// invalidate of the XCD, which the release/acquire fences of neighbour_sync
// cost.  Bounded like neighbour_sync.
__device__ __forceinline__ void neighbour_sync_coherent(unsigned int* flags, unsigned int* flag_err,
                                                        int tile, int tiles_x, int tiles_y,
                                                        unsigned int value) {
    __builtin_amdgcn_s_waitcnt(kWaitVmem);
    __syncthreads();
    if (threadIdx.x == 0)
        __hip_atomic_store(flags + tile, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (threadIdx.x < 9) {
        const int per_img = tiles_x * tiles_y;
        const int ti = tile % per_img;
        const int ty = ti / tiles_x + (int)threadIdx.x / 3 - 1;
        const int tx = ti % tiles_x + (int)threadIdx.x % 3 - 1;
        if (threadIdx.x != 4 && ty >= 0 && ty < tiles_y && tx >= 0 && tx < tiles_x) {
            const unsigned int* f = flags + (tile - ti) + ty * tiles_x + tx;
            unsigned int polls = 0;
            while (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < value) {
                __builtin_amdgcn_s_sleep(1);
                if (++polls == kSpinLimit) {
                    __hip_atomic_store(flag_err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
            }
        }
    }
    __syncthreads();
}

// Threads = (32 / P) * rows: at the 146 KB tile of k = 7 that gives 1
// (P = 4) or 2 (P = 2) waves per SIMD; declaring it lets the scheduler size
// registers.  RES: resident launch running all a.iters iterations; the tile
// stays in LDS and between iterations the work-groups only exchange the
// r-pixel border rings of their tiles through a.ring[], synchronised with
// their neighbours.
template <int K, int CM, bool EXACT, bool MAT, int P, bool RES>
__global__ __launch_bounds__(P == 4 ? 256 : 512)
__attribute__((amdgpu_waves_per_eu(P == 4 ? 1 : 2, P == 4 ? 1 : 2)))
void iter_kernel(const IterArgs a) {
    constexpr int TW = 32;
    constexpr int R = (K - 1) / 2;
    constexpr int LW = TW + 2 * R;            // staged columns
    constexpr int LS = iter_lds_stride(K, P, TW);
    constexpr int NW = P + K - 1;             // staged values per window row
    constexpr int KK = K * K;
    constexpr int CTR = R * K + R;            // centre tap index
    constexpr int TPR = TW / P;               // threads per tile row
    constexpr int kStagePix = 3;
    static_assert(!RES || !MAT, "resident launches are fused");
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
    const int x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t cbase = (size_t)b * C;       // this image's first plane

    const size_t HW = (size_t)H * W;
    const float* __restrict__ src = a.src + cbase * HW;
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
    // (resident launches are built for Potts only)
    const bool general_compat = !RES && a.mu != nullptr;

    // With Potts the update is softmax(U + M) (the compatibility transform
    // -(sum M - M) differs from +M by a per-pixel constant), so the message
    // accumulates straight onto the unary, which is loaded here and arrives
    // while the tile is being staged.
    const bool unary_first = !general_compat;
    const float* const unary_px = a.unary + cbase * HW + (size_t)y * W + xb;
    float acc[P][CM];
#pragma unroll
    for (int i = 0; i < P; ++i)
#pragma unroll
        for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;
    if (unary_first && pix_ok) load_pixels(acc, unary_px, xb, fullv);

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
    for (int it = 0;; ++it) {
    if (it > 0) {  // resident launch: the next iteration starts from U again
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;
        if (unary_first && pix_ok) load_pixels(acc, unary_px, xb, fullv);
    }

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
        // classes in order, the rows of the next kDepth - 1 classes read from
        // LDS while the current one is applied (a rolling pipeline)
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
        constexpr int kDepth = 3;
        float qr[kDepth][NW];
#pragma unroll
        for (int j = 0; j < kDepth - 1; ++j)
            if (j < CM && (EXACT || j < C)) lds_row<NW, P>(qrow + j * plane, qr[j]);
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            if (EXACT || c < C) {
                const int nx = c + kDepth - 1;
                if (nx < CM && (EXACT || nx < C)) lds_row<NW, P>(qrow + nx * plane, qr[nx % kDepth]);
                apply(qr[c % kDepth], c);
                // one class per scheduling region: its reads are issued
                // kDepth - 1 classes ahead and are not batched with later ones
                if constexpr (kUnrollRows) __builtin_amdgcn_sched_barrier(0);
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

    float (&fin)[P][CM] = acc;
    const int xf = xb;
    const bool fullf = fullv;

    {
        // compatibility transform: fin <- U - mu * M (general mu only; with
        // Potts fin already holds U + M)
        if (general_compat) {
            // one row of mu at a time (a scheduling barrier per row keeps the
            // broadcast reads of mu from all being hoisted); the unary is
            // loaded first so that it arrives meanwhile
            float u[P][CM];
            {
                const float* ug = a.unary + cbase * HW + (size_t)y * W + xf;
#pragma unroll
                for (int c = 0; c < CM; ++c) {
                    if (!EXACT && c >= C) continue;
                    if (fullf && pix_ok) {
                        float tmp[P];
                        V::get(*reinterpret_cast<const typename V::T*>(ug + c * HW), tmp);
#pragma unroll
                        for (int j = 0; j < P; ++j) u[j][c] = tmp[j];
                    } else {
#pragma unroll
                        for (int j = 0; j < P; ++j)
                            u[j][c] = (pix_ok && xf + j < W) ? ug[c * HW + j] : 0.f;
                    }
                }
            }
            float z[P][CM];
#pragma unroll
            for (int l = 0; l < CM; ++l) {
                if (EXACT || l < C) {
                    float t[P];
#pragma unroll
                    for (int j = 0; j < P; ++j) t[j] = 0.f;
#pragma unroll
                    for (int lp = 0; lp < CM; ++lp) {
                        if (EXACT || lp < C) {
                            const float m = Ms[l * C + lp];
#pragma unroll
                            for (int j = 0; j < P; ++j) t[j] = fmaf(m, fin[j][lp], t[j]);
                        }
                    }
#pragma unroll
                    for (int j = 0; j < P; ++j) z[j][l] = u[j][l] - t[j];
                } else {
#pragma unroll
                    for (int j = 0; j < P; ++j) z[j][l] = 0.f;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int j = 0; j < P; ++j)
#pragma unroll
                for (int c = 0; c < CM; ++c) fin[j][c] = z[j][c];
        }
#pragma unroll
        for (int j = 0; j < P; ++j) softmax_regs<CM, EXACT>(fin[j], C);
    }

    if (!RES || it == a.iters - 1) {
        if (pix_ok) {
            float* __restrict__ dst = a.dst + cbase * HW + (size_t)y * W + xf;
#pragma unroll
            for (int c = 0; c < CM; ++c) {
                if (!EXACT && c >= C) continue;
                if (fullf) {
                    float tmp[P];
#pragma unroll
                    for (int j = 0; j < P; ++j) tmp[j] = fin[j][c];
                    *reinterpret_cast<typename V::T*>(dst + c * HW) = V::make(tmp);
                } else {
#pragma unroll
                    for (int j = 0; j < P; ++j)
                        if (xf + j < W) dst[c * HW + j] = fin[j][c];
                }
            }
        }
        break;
    }

    if constexpr (RES) {
        // Q_{t+1} of this tile into the LDS interior (in-image pixels; the
        // rest stays zero), its r-pixel border ring into the exchange buffer
        __syncthreads();                      // every read of Q_t is done
        float* __restrict__ ring = a.ring[(it + 1) & 1] + cbase * HW;
#pragma unroll
        for (int i = 0; i < P; ++i) {
            const int col = col0 + i;
            if (!pix_ok || xb + i >= W) continue;
            float* q = Qs + (ty + R) * LS + col + R;
#pragma unroll
            for (int c = 0; c < CM; ++c)
                if (EXACT || c < C) q[c * plane] = fin[i][c];
            if (ty < R || ty >= rows - R || col < R || col >= TW - R) {
                float* g = ring + (size_t)y * W + xb + i;
#pragma unroll
                for (int c = 0; c < CM; ++c)
                    if (EXACT || c < C) g[c * HW] = fin[i][c];
            }
        }
        neighbour_sync(a.sync + 1, a.sync, tile, a.tiles_x, a.tiles_per_img / a.tiles_x,
                       (unsigned int)(it + 1));
        // the halo of Q_{t+1}: the neighbouring tiles' rings (positions
        // outside the image keep the zero staged at the start)
        const float* __restrict__ nb = a.ring[(it + 1) & 1] + cbase * HW;
        const int band = R * LW, side = R * (LH - 2 * R);
        for (int idx = tid; idx < 2 * band + 2 * side; idx += nthreads) {
            int r, cc;
            if (idx < 2 * band) {
                const int k2 = idx - (idx >= band ? band : 0);
                r = (idx >= band ? LH - R : 0) + k2 / LW;
                cc = k2 - (k2 / LW) * LW;
            } else {
                const int j = idx - 2 * band;
                const int k2 = j - (j >= side ? side : 0);
                r = R + k2 / R;
                cc = (j >= side ? LW - R : 0) + (k2 - (k2 / R) * R);
            }
            const int gy = y0 - R + r, gx = x0 - R + cc;
            if (gy < 0 || gy >= H || gx < 0 || gx >= W) continue;
            const float* g = nb + (size_t)gy * W + gx;
            float v[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c) v[c] = (EXACT || c < C) ? g[c * HW] : 0.f;
            float* q = Qs + r * LS + cc;
#pragma unroll
            for (int c = 0; c < CM; ++c)
                if (EXACT || c < C) q[c * plane] = v[c];
        }
        __syncthreads();
    }
    }  // iterations
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
    auto fn = iter_kernel<K, CM, EXACT, MAT, P, false>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(t.threads()), lds, stream, a);
    return hipGetLastError();
}

// Resident launch: cooperative, so that the runtime refuses it (rather than
// the grid barrier waiting forever) unless every work-group is co-resident;
// hipErrorCooperativeLaunchTooLarge also when the occupancy query says the
// tiles do not fit at once, so the caller falls back to one launch per
// iteration.
template <int K, int CM, bool EXACT>
hipError_t launch_res(const IterArgs& a, TileConfig t, size_t lds, int num_cus,
                      hipStream_t stream, bool probe) {
    auto fn = iter_kernel<K, CM, EXACT, false, 2, true>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(fn),
                                                     t.threads(), lds);
    if (e != hipSuccess) return e;
    if ((long long)per_cu * num_cus < a.ntiles) return hipErrorCooperativeLaunchTooLarge;
    if (probe) return hipSuccess;
    IterArgs args = a;
    void* params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(fn), dim3(a.ntiles),
                                      dim3(t.threads()), params, (unsigned int)lds, stream);
}

// ------------------------------------------------------------ streamed update
// f(integral_constant<int, 0>), ..., f(integral_constant<int, N - 1>)
template <typename F, int... I>
__device__ __forceinline__ void static_for(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}

// Fused update with the staging streamed under the computation (iterations
// after the first; two pixels per thread on 64 x 16 tiles, all classes,
// k <= 7).  Instead
// of loading the whole halo'd tile before the message, every wave issues
// buffer loads that write straight into LDS (no registers held): the three
// colour planes and the first two chunks of class planes of Q_t.  As soon
// as the colours have landed the work-group computes all of its pixels'
// window weights (Eq. 4) into registers; then it applies them to the classes
// chunk by chunk, each chunk starting when its planes have landed and
// issuing the loads of the chunk two ahead, so that at most two chunks are
// in flight and the early ones do not queue behind the late ones.  The
// unary tile is loaded the same way, into the planes of chunks already
// applied, and added in the epilogue (compatibility, softmax, store).
//
// Each staged plane is padded to whole 64-float DMA rows and every wave
// issues the same number of loads per plane (a load past the plane goes to
// a dummy LDS row), so that a wave waits for a chunk with one constant
// vmcnt.  Pixels outside the image get an out-of-range buffer offset, which
// reads as zero: neighbours outside the image contribute nothing.
// Loads per wave of chunk k (classes [k CH, min((k + 1) CH, C))), 0 past
// the last chunk.
constexpr int stream_chunk_loads(int k, int C, int CH, int NJ) {
    return k * CH >= C ? 0 : NJ * (((k + 1) * CH < C ? (k + 1) * CH : C) - k * CH);
}

template <int K>
struct StreamShape {
    static constexpr int R = (K - 1) / 2;
    static constexpr int TW = kStreamTW, ROWS = kStreamRows;
    static constexpr int LW = TW + 2 * R, LH = ROWS + 2 * R;
    static constexpr int LS = iter_lds_stride(K, 2, TW);
    static constexpr int PLANE = stream_plane(K);
    static constexpr int NI = PLANE / 64;        // 64-float loads per plane
    static constexpr int NJ = (NI + 7) / 8;      // per wave and plane
};

// One chunk of the message, classes [C_LO, C_HI): for every (class, window
// row) step, the row of P + K - 1 staged values is read from LDS two steps
// ahead of the one being applied (a rolling pipeline, one scheduling region
// per step), and applied to both pixels with the weights held in registers.
// Qs points at plane 0 of the staged Q; the tile row of the thread is ty and
// its first staged column col0.
template <int K, int P, int LS, int PLANE, int CM, int C_LO, int C_HI>
__device__ __forceinline__ void message_chunk(const float* Qs, int ty, int col0,
                                              const float (&w)[K][P][K], float (&acc)[P][CM]) {
    constexpr int R = (K - 1) / 2, CTR = R * K + R, NW = P + K - 1;
    constexpr int kDepth = 3;
    constexpr int NC = C_HI - C_LO;
    constexpr int nsteps = NC * K;
    float qr[kDepth][NW];
    // per class one base offset the compiler cannot merge with the row
    // offsets, so that those fold into the LDS reads' immediates
    const float* qb[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        unsigned off = (unsigned)((C_LO + i) * PLANE + ty * LS + col0);
        asm volatile("" : "+v"(off));
        qb[i] = Qs + off;
    }
#pragma unroll
    for (int t = 0; t < kDepth - 1; ++t)
        if (t < nsteps) lds_row<NW, P>(qb[t / K] + (t % K) * LS, qr[t]);
#pragma unroll
    for (int t = 0; t < nsteps; ++t) {
        const int nx = t + kDepth - 1;
        if (nx < nsteps) lds_row<NW, P>(qb[nx / K] + (nx % K) * LS, qr[nx % kDepth]);
        const int c = C_LO + t / K, dy = t % K;
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int dx = 0; dx < K; ++dx)
                if (dy * K + dx != CTR)
                    acc[i][c] = fmaf(w[dy][i][dx], qr[t % kDepth][i + dx], acc[i][c]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// FIRST: the first iteration, whose source is U itself: all planes are
// loaded at once, each thread keeps the unary of its own pixels in
// registers, and the staged halo tile is turned into softmax(U) in place
// (Alg. 1 initialisation) before the message.
template <int K, int CM, int CH, bool FIRST>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void stream_kernel(const IterArgs a) {
    using SS = StreamShape<K>;
    constexpr int R = SS::R, LW = SS::LW, LH = SS::LH, LS = SS::LS;
    constexpr int PLANE = SS::PLANE, NI = SS::NI, NJ = SS::NJ;
    constexpr int P = 2, TW = SS::TW, ROWS = SS::ROWS, TPR = TW / P;
    static_assert(TPR * ROWS == 512 && TW * ROWS == 1024, "512 threads, two pixels each");
    constexpr int NW = P + K - 1;
    constexpr int CTR = R * K + R;
    constexpr int NCH = (CM + CH - 1) / CH;
    constexpr unsigned kOob = 0x80000000u;   // offset past any buffer: reads 0

    constexpr int MUP = (CM * CM + 63) / 64 * 64;   // compatibility, whole rows
    // the unary tile [CM][ROWS x TW] goes to the planes of chunks 0 .. UCH - 1
    // once they have been applied (the first chunk whose start frees enough)
    constexpr int UCH = (CM * 1024 + CH * PLANE - 1) / (CH * PLANE);
    static_assert(UCH < NCH, "the unary tile fits in the planes of the chunks before the last");
    constexpr int NU = (CM * 4 + 7) / 8;         // 16-byte loads of 8 rows, per wave
    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qs = smem;                      // [CM][PLANE]
    float* const Cs = smem + CM * PLANE;         // [3][PLANE]
    float* const Ms = Cs + 3 * PLANE;            // [CM][CM] (+ padding) when given
    float* const dummy = Ms + (a.mu ? MUP : 0);  // one 256-float row
    const unsigned lds0 = (unsigned)(size_t)(__attribute__((address_space(3))) float*)smem;
    auto lds_addr = [&](const float* p) { return lds0 + (unsigned)((p - smem) * 4); };

    const int H = a.H, W = a.W;
    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * ROWS;
    const int x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t HW = (size_t)H * W;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;

    // ---- issue every load into LDS: colours, then Q_t class by class
    unsigned voff[NJ];
    int dst[NJ];                                 // float offset in a plane, or -1: dummy
#pragma unroll
    for (int s = 0; s < NJ; ++s) {
        const int j = wave + 8 * s;
        const int f = j * 64 + lane;
        const int r = f / LS, col = f - (f / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        const bool in = j < NI && f < LH * LS && col < LW && gy >= 0 && gy < H && gx >= 0 && gx < W;
        voff[s] = in ? (unsigned)((gy * W + gx) * 4) : kOob;
        dst[s] = j < NI ? j * 64 : -1;
    }
    const rsrc_t rf = buffer_rsrc(a.feat + (size_t)b * 3 * HW, (unsigned)(3 * HW * 4));
    const rsrc_t rq = buffer_rsrc(a.src + (size_t)b * CM * HW, (unsigned)(CM * HW * 4));
    // the compatibility matrix rides with the colours: MUP / 64 rows, one
    // per wave in turn (the same count on every wave: wave-uniform loads
    // past the matrix go to the dummy row)
    constexpr int NMU = (MUP / 64 + 7) / 8;
    const int nmu = a.mu ? NMU : 0;
    const rsrc_t rm = buffer_rsrc(a.mu ? a.mu : a.feat, (unsigned)(CM * CM * 4));
    for (int s = 0; s < nmu; ++s) {
        const int j = wave + 8 * s;
        lds_dma(rm, (unsigned)((j * 64 + lane) * 4), 0, lds_addr(j < MUP / 64 ? Ms + j * 64 : dummy));
    }
#pragma unroll
    for (int ch = 0; ch < 3; ++ch)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rf, voff[s], (int)(ch * HW * 4),
                    lds_addr(dst[s] >= 0 ? Cs + ch * PLANE + dst[s] : dummy));
    auto issue_chunk = [&](int k) {
        const int c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        for (int c = k * CH; c < c_hi; ++c)
#pragma unroll
            for (int s = 0; s < NJ; ++s)
                lds_dma(rq, voff[s], (int)(c * HW * 4),
                        lds_addr(dst[s] >= 0 ? Qs + c * PLANE + dst[s] : dummy));
    };
    if constexpr (FIRST) {
        for (int k = 0; k < NCH; ++k) issue_chunk(k);
    } else {
        issue_chunk(0);
        if (NCH > 1) issue_chunk(1);
    }

    const int tx = tid % TPR, ty = tid / TPR;
    const int col0 = tx * P;
    const int y = y0 + ty, xb = x0 + col0;
    const bool pix_ok = y < H && xb < W;        // W even: both pixels or neither

    // ---- colours landed: the window weights of both pixels, all rows
    // (a wait beyond the 63 loads a wave can have outstanding is clamped:
    // the loads before the last 63 issued have completed by then)
    __builtin_amdgcn_s_waitcnt(vm_wait(FIRST ? NJ * CM
                                             : stream_chunk_loads(0, CM, CH, NJ) +
                                                   stream_chunk_loads(1, CM, CH, NJ)));
    __syncthreads();
    float w[K][P][K];
    {
        float own[3][P];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
#pragma unroll
            for (int i = 0; i < P; ++i) own[ch][i] = Cs[ch * PLANE + (ty + R) * LS + col0 + R + i];
#pragma unroll
        for (int dy = 0; dy < K; ++dy) {
            float nc[3][NW];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) lds_row<NW, P>(Cs + ch * PLANE + (ty + dy) * LS + col0, nc[ch]);
#pragma unroll
            for (int i = 0; i < P; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    if (dy * K + dx == CTR) { w[dy][i][dx] = 0.f; continue; }
                    const int n = (dx - R) * (dx - R) + (dy - R) * (dy - R);
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    w[dy][i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[n])) +
                                   a.taps.smooth[n];
                }
            }
        }
    }

    float u[P][CM];
    if constexpr (FIRST) {
        // every plane landed: keep this thread's unary, then softmax(U) over
        // the staged in-image positions (outside the image stays zero)
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
        __syncthreads();
#pragma unroll
        for (int c = 0; c < CM; ++c)
#pragma unroll
            for (int i = 0; i < P; ++i) u[i][c] = Qs[c * PLANE + (ty + R) * LS + col0 + R + i];
        __syncthreads();
        for (int pos = tid; pos < LH * LS; pos += 512) {
            const int r = pos / LS, col = pos - (pos / LS) * LS;
            const int gy = y0 - R + r, gx = x0 - R + col;
            if (col >= LW || gy < 0 || gy >= H || gx < 0 || gx >= W) continue;
            float z[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c) z[c] = Qs[c * PLANE + pos];
            softmax_regs<CM, true>(z, CM);
#pragma unroll
            for (int c = 0; c < CM; ++c) Qs[c * PLANE + pos] = z[c];
        }
        __syncthreads();
    }

    // ---- the message, chunk by chunk as the planes land
    float acc[P][CM];
#pragma unroll
    for (int i = 0; i < P; ++i)
#pragma unroll
        for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;
    float* const Us = Qs;                        // [CM][ROWS x TW], from chunk UCH on
    const rsrc_t ru = buffer_rsrc(a.unary + (size_t)b * CM * HW, (unsigned)(CM * HW * 4));
    static_for([&](auto kc) {
        constexpr int k = decltype(kc)::value;
        constexpr int c_lo = k * CH;
        constexpr int c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        // chunk k landed.  Issued after its loads (at chunk k - 2) and
        // before this wait: chunk k + 1 (at chunk k - 1), and the unary if
        // it went out at chunk k - 2 or k - 1.
        if constexpr (!FIRST) {
            __builtin_amdgcn_s_waitcnt(vm_wait(stream_chunk_loads(k + 1, CM, CH, NJ) +
                                               (UCH < k && k <= UCH + 2 ? NU : 0)));
            __syncthreads();
        }
        if constexpr (!FIRST && k + 2 < NCH) issue_chunk(k + 2);
        if constexpr (!FIRST && k == UCH) {
            // every wave is past the chunks before k: their planes take the
            // unary tile, plane c at Us + 1024 c, 256 / TW rows per load
#pragma unroll
            for (int s = 0; s < NU; ++s) {
                const int j = wave + 8 * s;          // (plane, band of 256 / TW rows)
                constexpr int LPR = TW / 4;          // lanes per row
                const int c = j / 4, r = (j % 4) * (256 / TW) + lane / LPR, col = (lane % LPR) * 4;
                const bool in = j < CM * 4 && y0 + r < H && x0 + col < W;
                lds_dma16(ru, in ? (unsigned)(((y0 + r) * W + x0 + col) * 4) : kOob,
                          (int)((j < CM * 4 ? c : 0) * HW * 4),
                          lds_addr(j < CM * 4 ? Us + j * 256 : dummy));
            }
        }
        message_chunk<K, P, LS, PLANE, CM, c_lo, c_hi>(Qs, ty, col0, w, acc);
        if (a.include_center) {
#pragma unroll
            for (int c = c_lo; c < c_hi; ++c)
#pragma unroll
                for (int i = 0; i < P; ++i)
                    acc[i][c] = fmaf(a.center_w, Qs[c * PLANE + (ty + R) * LS + col0 + R + i],
                                     acc[i][c]);
        }
    }, std::make_integer_sequence<int, NCH>{});
    if constexpr (!FIRST) {
        __builtin_amdgcn_s_waitcnt(vm_wait(0));
        __syncthreads();
#pragma unroll
        for (int c = 0; c < CM; ++c) {
            const float2 t = *reinterpret_cast<const float2*>(Us + c * 1024 + ty * TW + col0);
            u[0][c] = t.x;
            u[1][c] = t.y;
        }
    }
    if (!pix_ok) return;

    // ---- compatibility, unary, softmax (Alg. 1), store Q_{t+1}
    if (a.mu) {
        float z[P][CM];
#pragma unroll
        for (int l = 0; l < CM; ++l) {
            float t[P];
#pragma unroll
            for (int i = 0; i < P; ++i) t[i] = 0.f;
#pragma unroll
            for (int lp = 0; lp < CM; ++lp) {
                const float m = Ms[l * CM + lp];
#pragma unroll
                for (int i = 0; i < P; ++i) t[i] = fmaf(m, acc[i][lp], t[i]);
            }
#pragma unroll
            for (int i = 0; i < P; ++i) z[i][l] = u[i][l] - t[i];
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] = z[i][c];
    } else {
        // Potts: softmax(U + M)
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] += u[i][c];
    }
#pragma unroll
    for (int i = 0; i < P; ++i) softmax_regs<CM, true>(acc[i], CM);
    float* __restrict__ qd = a.dst + (size_t)b * CM * HW + (size_t)y * W + xb;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        float tmp[P];
#pragma unroll
        for (int i = 0; i < P; ++i) tmp[i] = acc[i][c];
        *reinterpret_cast<typename Vec<P>::T*>(qd + c * HW) = Vec<P>::make(tmp);
    }
}

template <int K, int CM, int CH>
hipError_t launch_stream(const IterArgs& a, size_t lds, hipStream_t stream) {
    auto fn = a.first ? stream_kernel<K, CM, CH, true> : stream_kernel<K, CM, CH, false>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(512), lds, stream, a);
    return hipGetLastError();
}

// ---------------------------------------------------------- ring update
// The later iterations on half-height tiles (kStreamTW x kRingRows, 256
// threads, two pixels each) so that two work-groups share a CU and one's
// waits overlap the other's arithmetic.  As stream_kernel, but the class
// chunks cycle through kRingSlots LDS slots (chunk k in slot k mod
// kRingSlots; one chunk per slot is issued at the start, then chunk
// k + kRingSlots - 1 goes into the slot of chunk k - 1 once every wave is
// past it) and each thread's unary comes straight into registers, issued
// once the first chunk has landed.
// FD > 0: learnable smoothness features (the "+T" variant of Sec. 4.2): the
// FD feature planes are staged beside the colours and the smoothness Gaussian
// of each weight is taken on the feature distance.
template <int K, int CM, int CH, int FD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void ring_kernel(const IterArgs a) {
    constexpr int R = (K - 1) / 2;
    constexpr int P = 2, TW = kStreamTW, ROWS = kRingRows, TPR = TW / P, NWAVE = 4;
    static_assert(TPR * ROWS == 256, "256 threads, two pixels each");
    constexpr int LW = TW + 2 * R, LH = ROWS + 2 * R;
    constexpr int LS = iter_lds_stride(K, 2, TW);
    constexpr int PLANE = ring_plane(K);
    constexpr int NI = PLANE / 64;               // 64-float loads per plane
    constexpr int NJ = (NI + NWAVE - 1) / NWAVE; // per wave and plane
    constexpr int NW = P + K - 1;
    constexpr int CTR = R * K + R;
    constexpr int NCH = (CM + CH - 1) / CH;
    constexpr unsigned kOob = 0x80000000u;
    constexpr int MUP = (CM * CM + 63) / 64 * 64;
    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    constexpr bool FT = FD > 0;
    constexpr int D = FD;
    float* const Qs = smem;                              // [3][CH][PLANE]
    float* const Cs = smem + kRingSlots * CH * PLANE;    // [3][PLANE]
    float* const Ms = Cs + 3 * PLANE;                    // [CM][CM] (+ padding) when given
    float* const dummy = Ms + (a.mu ? MUP : 0);          // one 256-float row
    float* const Fs = dummy + 256;                       // [FD][PLANE]
    const unsigned lds0 = (unsigned)(size_t)(__attribute__((address_space(3))) float*)smem;
    auto lds_addr = [&](const float* p) { return lds0 + (unsigned)((p - smem) * 4); };

    const int H = a.H, W = a.W;
    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * ROWS;
    const int x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t HW = (size_t)H * W;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int tx = tid % TPR, ty = tid / TPR;
    const int col0 = tx * P;
    const int y = y0 + ty, xb = x0 + col0;
    const bool pix_ok = y < H && xb < W;        // W even: both pixels or neither

    // ---- colours, then the first two chunks of Q_t
    unsigned voff[NJ];
    int dst[NJ];                                 // float offset in a plane, or -1: dummy
#pragma unroll
    for (int s = 0; s < NJ; ++s) {
        const int j = wave + NWAVE * s;
        const int f = j * 64 + lane;
        const int r = f / LS, col = f - (f / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        const bool in = j < NI && f < LH * LS && col < LW && gy >= 0 && gy < H && gx >= 0 && gx < W;
        voff[s] = in ? (unsigned)((gy * W + gx) * 4) : kOob;
        dst[s] = j < NI ? j * 64 : -1;
    }
    const rsrc_t rf = buffer_rsrc(a.feat + (size_t)b * 3 * HW, (unsigned)(3 * HW * 4));
    const rsrc_t rq = buffer_rsrc(a.src + (size_t)b * CM * HW, (unsigned)(CM * HW * 4));
    constexpr int NMU = (MUP / 64 + NWAVE - 1) / NWAVE;
    const int nmu = a.mu ? NMU : 0;
    const rsrc_t rm = buffer_rsrc(a.mu ? a.mu : a.feat, (unsigned)(CM * CM * 4));
    for (int s = 0; s < nmu; ++s) {
        const int j = wave + NWAVE * s;
        lds_dma(rm, (unsigned)((j * 64 + lane) * 4), 0, lds_addr(j < MUP / 64 ? Ms + j * 64 : dummy));
    }
#pragma unroll
    for (int ch = 0; ch < 3; ++ch)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rf, voff[s], (int)(ch * HW * 4),
                    lds_addr(dst[s] >= 0 ? Cs + ch * PLANE + dst[s] : dummy));
    if constexpr (FT) {
        const rsrc_t rs = buffer_rsrc(a.sfeat + (size_t)b * D * HW, (unsigned)(D * HW * 4));
#pragma unroll
        for (int ch = 0; ch < D; ++ch)
#pragma unroll
            for (int s = 0; s < NJ; ++s)
                lds_dma(rs, voff[s], (int)(ch * HW * 4),
                        lds_addr(dst[s] >= 0 ? Fs + ch * PLANE + dst[s] : dummy));
    }
    // chunk k goes to slot k % kRingSlots
    auto issue_chunk = [&](int k) {
        const int c_lo = k * CH, c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        float* const slot = Qs + (k % kRingSlots) * CH * PLANE;
        for (int c = c_lo; c < c_hi; ++c)
#pragma unroll
            for (int s = 0; s < NJ; ++s)
                lds_dma(rq, voff[s], (int)(c * HW * 4),
                        lds_addr(dst[s] >= 0 ? slot + (c - c_lo) * PLANE + dst[s] : dummy));
    };
    // one chunk per slot now (A0 of them); from then on AHEAD = kRingSlots - 1
    // chunks ahead: chunk k + AHEAD is issued at chunk k, into the slot of
    // chunk k - 1
    constexpr int A0 = kRingSlots, AHEAD = kRingSlots - 1;
    static_for([&](auto kc) {
        if constexpr (decltype(kc)::value < NCH) issue_chunk(decltype(kc)::value);
    }, std::make_integer_sequence<int, A0>{});
    // loads of chunks [k0, k0 + n) per wave
    auto chunk_loads = [](int k0, int n) {
        int t = 0;
        for (int j = k0; j < k0 + n; ++j) t += stream_chunk_loads(j, CM, CH, NJ);
        return t;
    };

    // ---- colours landed: the window weights of both pixels, all rows
    __builtin_amdgcn_s_waitcnt(vm_wait(chunk_loads(0, A0)));
    __syncthreads();
    float w[K][P][K];
    {
        float own[3][P];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
#pragma unroll
            for (int i = 0; i < P; ++i) own[ch][i] = Cs[ch * PLANE + (ty + R) * LS + col0 + R + i];
#pragma unroll
        for (int dy = 0; dy < K; ++dy) {
            // FT: the squared feature distance accumulates in w first, one
            // plane at a time, to keep the register footprint of a row small
            if constexpr (FT) {
#pragma unroll
                for (int i = 0; i < P; ++i)
#pragma unroll
                    for (int dx = 0; dx < K; ++dx) w[dy][i][dx] = 0.f;
#pragma unroll
                for (int ch = 0; ch < D; ++ch) {
                    const float* const fp = Fs + ch * PLANE;
                    float fo[P], nf[NW];
#pragma unroll
                    for (int i = 0; i < P; ++i) fo[i] = fp[(ty + R) * LS + col0 + R + i];
                    lds_row<NW, P>(fp + (ty + dy) * LS + col0, nf);
#pragma unroll
                    for (int i = 0; i < P; ++i)
#pragma unroll
                        for (int dx = 0; dx < K; ++dx) {
                            const float e = fo[i] - nf[i + dx];
                            w[dy][i][dx] = fmaf(e, e, w[dy][i][dx]);
                        }
                }
            }
            float nc[3][NW];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) lds_row<NW, P>(Cs + ch * PLANE + (ty + dy) * LS + col0, nc[ch]);
#pragma unroll
            for (int i = 0; i < P; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    if (dy * K + dx == CTR) { w[dy][i][dx] = 0.f; continue; }
                    const int n = (dx - R) * (dx - R) + (dy - R) * (dy - R);
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    const float smo = FT ? a.w_smooth * __builtin_amdgcn_exp2f(a.neg_gamma * w[dy][i][dx])
                                         : a.taps.smooth[n];
                    w[dy][i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[n])) +
                                   smo;
                }
            }
        }
    }

    float acc[P][CM];
#pragma unroll
    for (int i = 0; i < P; ++i)
#pragma unroll
        for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;
    // the unary of this thread's pixels goes straight into registers; it is
    // needed only by the epilogue, so its loads are issued once chunk UK = 0
    // has landed, which keeps them out of the launch's opening burst of
    // colour and class-plane loads
    constexpr int UK = 0;
    float u[P][CM];
    static_for([&](auto kc) {
        constexpr int k = decltype(kc)::value;
        constexpr int c_lo = k * CH;
        constexpr int c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        // chunk k landed (the chunks issued after it, up to chunk `last`,
        // and the unary when it went out after chunk k, may not have); every
        // wave is past chunk k - 1, whose slot chunk k + AHEAD takes.  Chunk
        // k was issued at chunk `sk` (-1: at the start).
        constexpr int last0 = k == 0 ? A0 - 1 : (A0 - 1 > k - 1 + AHEAD ? A0 - 1 : k - 1 + AHEAD);
        constexpr int last = last0 < NCH - 1 ? last0 : NCH - 1;
        constexpr int sk = k < A0 ? -1 : k - AHEAD;
        __builtin_amdgcn_s_waitcnt(vm_wait(chunk_loads(k + 1, last - k) +
                                           (sk <= UK && UK < k ? CM : 0)));
        __syncthreads();
        if constexpr (k + AHEAD < NCH && k + AHEAD > last) issue_chunk(k + AHEAD);
        if constexpr (k == UK) {
            const float* up = a.unary + (size_t)b * CM * HW + (size_t)(pix_ok ? y : 0) * W +
                              (pix_ok ? xb : 0);
#pragma unroll
            for (int c = 0; c < CM; ++c) {
                const float2 t = *reinterpret_cast<const float2*>(up + c * HW);
                u[0][c] = t.x;
                u[1][c] = t.y;
            }
        }
        // the slot seen as planes c_lo .. c_hi - 1 of Q_t
        const float* const qk = Qs + (k % kRingSlots) * CH * PLANE - c_lo * PLANE;
        message_chunk<K, P, LS, PLANE, CM, c_lo, c_hi>(qk, ty, col0, w, acc);
        if (a.include_center) {
#pragma unroll
            for (int c = c_lo; c < c_hi; ++c)
#pragma unroll
                for (int i = 0; i < P; ++i)
                    acc[i][c] = fmaf(a.center_w, qk[c * PLANE + (ty + R) * LS + col0 + R + i],
                                     acc[i][c]);
        }
    }, std::make_integer_sequence<int, NCH>{});
    __builtin_amdgcn_s_waitcnt(vm_wait(0));     // the unary
    if (!pix_ok) return;

    // ---- compatibility, unary, softmax (Alg. 1), store Q_{t+1}
    if (a.mu) {
        float z[P][CM];
#pragma unroll
        for (int l = 0; l < CM; ++l) {
            float t[P];
#pragma unroll
            for (int i = 0; i < P; ++i) t[i] = 0.f;
#pragma unroll
            for (int lp = 0; lp < CM; ++lp) {
                const float m = Ms[l * CM + lp];
#pragma unroll
                for (int i = 0; i < P; ++i) t[i] = fmaf(m, acc[i][lp], t[i]);
            }
#pragma unroll
            for (int i = 0; i < P; ++i) z[i][l] = u[i][l] - t[i];
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] = z[i][c];
    } else {
        // Potts: softmax(U + M)
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] += u[i][c];
    }
#pragma unroll
    for (int i = 0; i < P; ++i) softmax_regs<CM, true>(acc[i], CM);
    float* __restrict__ qd = a.dst + (size_t)b * CM * HW + (size_t)y * W + xb;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        float tmp[P];
#pragma unroll
        for (int i = 0; i < P; ++i) tmp[i] = acc[i][c];
        *reinterpret_cast<typename Vec<P>::T*>(qd + c * HW) = Vec<P>::make(tmp);
    }
}

template <int K, int CM, int CH>
hipError_t launch_ring(const IterArgs& a, hipStream_t stream) {
    auto fn = ring_kernel<K, CM, CH, 0>;
    switch (a.sfeat ? a.D : 0) {
        case 0: break;
        case 1: fn = ring_kernel<K, CM, CH, 1>; break;
        case 2: fn = ring_kernel<K, CM, CH, 2>; break;
        case 3: fn = ring_kernel<K, CM, CH, 3>; break;
        case 4: fn = ring_kernel<K, CM, CH, 4>; break;
        default: return hipErrorNotSupported;
    }
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(256),
                       ring_lds_bytes(K, CM, CH, a.mu != nullptr, a.sfeat ? a.D : 0), stream, a);
    return hipGetLastError();
}

// ------------------------------------------------- quad update (k = 7, Potts)
// Rounds 2..T of the k = 7 update with Potts compatibility, on the ring's
// tiles, staging and class-chunk ring, with a thread layout that cuts the
// LDS bytes of the message (which bound ring_kernel's message loop): a pair
// of lanes shares four horizontally adjacent pixels.  The even lane applies
// window rows 0, 1, 2 and the left half of row 3, the odd lane rows 4, 5, 6
// and the right half of row 3: 24 taps each, the centre excluded; each lane
// picks its per-offset constants once per tap.  Per (class, window row) a
// lane reads 10 staged floats (rows
// padded to 16 bytes: two 16-byte reads and an 8-byte one) for 28 FMAs,
// where the two-pixel layout reads 8 for 14.  After each chunk the pair adds
// its two partial messages with one DPP lane swap per class and pixel: the
// even lane keeps pixels 0 and 1, the odd lane pixels 2 and 3, and each then
// runs ring_kernel's epilogue on its two.
template <int N>
__device__ __forceinline__ void lds_row16(const float* p, float (&v)[N]) {
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

// x from the other lane of the pair (lanes 2m and 2m + 1)
__device__ __forceinline__ float pair_swap(float x) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
}

// One chunk of the quad message, classes [C_LO, C_HI): step t applies window
// row t % 4 of class C_LO + t / 4 (rows 0..2 full, 3 the half row), read
// from LDS two steps ahead, to the lane's four pixels.
template <int PLANE, int LS, int C_LO, int C_HI>
__device__ __forceinline__ void quad_chunk(const float* Qs, unsigned rbase, unsigned hbase,
                                           const float (&w)[4][4][7], float (&acc)[4][C_HI - C_LO]) {
    constexpr int NC = C_HI - C_LO, nsteps = NC * 4, kDepth = 3;
    float qr[kDepth][10];
    // per class one base for the full rows (rows at immediate offsets from
    // it) and one for the half row, opaque to the compiler so that it does
    // not fold them into per-step address registers
    const float* qb[NC];
    const float* hb[NC];
#pragma unroll
    for (int i = 0; i < NC; ++i) {
        unsigned off = (unsigned)((C_LO + i) * PLANE) + rbase;
        unsigned hoff = (unsigned)((C_LO + i) * PLANE) + hbase;
        asm volatile("" : "+v"(off), "+v"(hoff));
        qb[i] = Qs + off;
        hb[i] = Qs + hoff;
    }
    auto rd = [&](int t, float (&v)[10]) {
        const float* const q = t % 4 == 3 ? hb[t / 4] : qb[t / 4] + (t % 4) * LS;
        if (t % 4 == 3) {
            float h[6];
            lds_row16<6>(q, h);
#pragma unroll
            for (int j = 0; j < 6; ++j) v[j] = h[j];
        } else {
            lds_row16<10>(q, v);
        }
    };
#pragma unroll
    for (int t = 0; t < kDepth - 1; ++t)
        if (t < nsteps) rd(t, qr[t]);
#pragma unroll
    for (int t = 0; t < nsteps; ++t) {
        const int nx = t + kDepth - 1;
        if (nx < nsteps) rd(nx, qr[nx % kDepth]);
        const int c = t / 4, j = t % 4;
        const int ntap = j == 3 ? 3 : 7;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int d = 0; d < ntap; ++d) acc[i][c] = fmaf(w[j][i][d], qr[t % kDepth][i + d], acc[i][c]);
        __builtin_amdgcn_sched_barrier(0);
    }
}

template <int CM, int CH>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void quad_kernel(const IterArgs a) {
    constexpr int K = 7, R = 3;
    constexpr int TW = kStreamTW, ROWS = kRingRows, NWAVE = 4;
    constexpr int LW = TW + 2 * R, LH = ROWS + 2 * R;
    constexpr int LS = kQuadStride;
    constexpr int PLANE = quad_plane();
    constexpr int NI = PLANE / 64;               // 64-float loads per plane
    constexpr int NJ = (NI + NWAVE - 1) / NWAVE; // per wave and plane
    constexpr int NCH = (CM + CH - 1) / CH;
    constexpr unsigned kOob = 0x80000000u;
    static_assert(4 * 16 == TW && 2 * 16 * ROWS == 256, "16 pixel quads per row, a lane pair each");
    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qs = smem;                              // [kRingSlots][CH][PLANE]
    float* const Cs = smem + kRingSlots * CH * PLANE;    // [3][PLANE]
    float* const dummy = Cs + 3 * PLANE;                 // one 256-float row
    const unsigned lds0 = (unsigned)(size_t)(__attribute__((address_space(3))) float*)smem;
    auto lds_addr = [&](const float* p) { return lds0 + (unsigned)((p - smem) * 4); };

    const int H = a.H, W = a.W;
    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * ROWS;
    const int x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t HW = (size_t)H * W;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int half = tid & 1, ty = tid >> 5;
    const int cq = 4 * ((tid >> 1) & 15);        // staged column of pixel 0's window
    const int y = y0 + ty, xo = x0 + cq + 2 * half;   // the lane's two output pixels
    const bool pix_ok = y < H && x0 + cq < W;    // W % 4 == 0: all four or none

    // ---- colours, then the first chunks of Q_t (as ring_kernel)
    unsigned voff[NJ];
    int dst[NJ];
#pragma unroll
    for (int s = 0; s < NJ; ++s) {
        const int j = wave + NWAVE * s;
        const int f = j * 64 + lane;
        const int r = f / LS, col = f - (f / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        const bool in = j < NI && f < LH * LS && col < LW && gy >= 0 && gy < H && gx >= 0 && gx < W;
        voff[s] = in ? (unsigned)((gy * W + gx) * 4) : kOob;
        dst[s] = j < NI ? j * 64 : -1;
    }
    const rsrc_t rf = buffer_rsrc(a.feat + (size_t)b * 3 * HW, (unsigned)(3 * HW * 4));
    const rsrc_t rq = buffer_rsrc(a.src + (size_t)b * CM * HW, (unsigned)(CM * HW * 4));
#pragma unroll
    for (int ch = 0; ch < 3; ++ch)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rf, voff[s], (int)(ch * HW * 4),
                    lds_addr(dst[s] >= 0 ? Cs + ch * PLANE + dst[s] : dummy));
    auto issue_chunk = [&](int k) {
        const int c_lo = k * CH, c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        float* const slot = Qs + (k % kRingSlots) * CH * PLANE;
        for (int c = c_lo; c < c_hi; ++c)
#pragma unroll
            for (int s = 0; s < NJ; ++s)
                lds_dma(rq, voff[s], (int)(c * HW * 4),
                        lds_addr(dst[s] >= 0 ? slot + (c - c_lo) * PLANE + dst[s] : dummy));
    };
    constexpr int A0 = kRingSlots, AHEAD = kRingSlots - 1;
    static_for([&](auto kc) {
        if constexpr (decltype(kc)::value < NCH) issue_chunk(decltype(kc)::value);
    }, std::make_integer_sequence<int, A0>{});
    auto chunk_loads = [](int k0, int n) {
        int t = 0;
        for (int j = k0; j < k0 + n; ++j) t += stream_chunk_loads(j, CM, CH, NJ);
        return t;
    };

    // this lane's window rows: full rows R (half + 1) + j, j < R, at
    // rbase + j LS, and the half row R at hbase
    const unsigned rbase = (unsigned)((ty + (R + 1) * half) * LS + cq);
    const unsigned hbase = (unsigned)((ty + R) * LS + cq + (R + 1) * half);

    // ---- colours landed: the weights of the lane's 4 x 24 taps
    __builtin_amdgcn_s_waitcnt(vm_wait(chunk_loads(0, A0)));
    __syncthreads();
    float w[4][4][K];
    {
        float own[3][4];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            float r[10];
            lds_row16<10>(Cs + ch * PLANE + (ty + R) * LS + cq, r);
#pragma unroll
            for (int i = 0; i < 4; ++i) own[ch][i] = r[R + i];
        }
#pragma unroll
        for (int j = 0; j < R; ++j) {
            float nc[3][10];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) lds_row16<10>(Cs + ch * PLANE + rbase + j * LS, nc[ch]);
#pragma unroll
            for (int dx = 0; dx < K; ++dx) {
                // |d|^2 of the tap for the even lane (row j) and the odd one (row R + 1 + j)
                const int ne = (dx - R) * (dx - R) + (R - j) * (R - j);
                const int no = (dx - R) * (dx - R) + (j + 1) * (j + 1);
                float ae = a.taps.app_log2[ne], ao = a.taps.app_log2[no];
                float se = a.taps.smooth[ne], so = a.taps.smooth[no];
                asm volatile("" : "+s"(ae), "+s"(ao), "+s"(se), "+s"(so));
                const float ca = half ? ao : ae;
                const float cs = half ? so : se;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    w[j][i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, ca)) + cs;
                }
            }
        }
        // the half row: taps dx = d (even lane) or R + 1 + d (odd lane)
        float hc[3][6];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) lds_row16<6>(Cs + ch * PLANE + hbase, hc[ch]);
#pragma unroll
        for (int d = 0; d < R; ++d) {
            const int nl = (R - d) * (R - d), nr = (d + 1) * (d + 1);
            // both constants as scalars first, then the lane's choice
            float al = a.taps.app_log2[nl], ar = a.taps.app_log2[nr];
            float sl = a.taps.smooth[nl], sr = a.taps.smooth[nr];
            asm volatile("" : "+s"(al), "+s"(ar), "+s"(sl), "+s"(sr));
            const float ca = half ? ar : al;
            const float cs = half ? sr : sl;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float d0 = own[0][i] - hc[0][i + d];
                const float d1 = own[1][i] - hc[1][i + d];
                const float d2 = own[2][i] - hc[2][i + d];
                const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                w[3][i][d] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, ca)) + cs;
            }
        }
    }

    // keep the weights' arithmetic above the chunk loop, where the unary's
    // registers are not yet live
    __builtin_amdgcn_sched_barrier(0);
    // the message of the lane's two pixels, completed chunk by chunk; the
    // unary (Potts: Z = U + M) is loaded at the last chunk, where it first
    // has registers to land in
    float fin[2][CM];
    float u[2][CM];
    constexpr int UK = NCH - 1;
    static_for([&](auto kc) {
        constexpr int k = decltype(kc)::value;
        constexpr int c_lo = k * CH;
        constexpr int c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        constexpr int last0 = k == 0 ? A0 - 1 : (A0 - 1 > k - 1 + AHEAD ? A0 - 1 : k - 1 + AHEAD);
        constexpr int last = last0 < NCH - 1 ? last0 : NCH - 1;
        constexpr int sk = k < A0 ? -1 : k - AHEAD;
        __builtin_amdgcn_s_waitcnt(vm_wait(chunk_loads(k + 1, last - k) +
                                           (sk <= UK && UK < k ? CM : 0)));
        __syncthreads();
        if constexpr (k + AHEAD < NCH && k + AHEAD > last) issue_chunk(k + AHEAD);
        if constexpr (k == UK) {
            // buffer loads: one lane offset and a scalar offset per class, so
            // that no 64-bit address is held per class
            const __amdgpu_buffer_rsrc_t ru = __builtin_amdgcn_make_buffer_rsrc(
                (void*)(a.unary + (size_t)b * CM * HW), (short)0, (int)(CM * HW * 4), 0x00020000);
            const int uoff = pix_ok ? (y * W + xo) * 4 : 0;
#pragma unroll
            for (int c = 0; c < CM; ++c) {
                const auto t = __builtin_amdgcn_raw_buffer_load_b64(ru, uoff, (int)(c * HW * 4), 0);
                u[0][c] = __int_as_float((int)t[0]);
                u[1][c] = __int_as_float((int)t[1]);
            }
        }
        float acc[4][c_hi - c_lo];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < c_hi - c_lo; ++c) acc[i][c] = 0.f;
        const float* const qk = Qs + (k % kRingSlots) * CH * PLANE;
        quad_chunk<PLANE, LS, c_lo, c_hi>(qk - c_lo * PLANE, rbase, hbase, w, acc);
#pragma unroll
        for (int c = 0; c < c_hi - c_lo; ++c)
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float mine = half ? acc[2 + i][c] : acc[i][c];
                const float send = half ? acc[i][c] : acc[2 + i][c];
                fin[i][c_lo + c] = mine + pair_swap(send);
                // materialised here: sunk to the epilogue, the add would keep
                // both of its operands live through the remaining chunks
                asm volatile("" : "+v"(fin[i][c_lo + c]));
            }
    }, std::make_integer_sequence<int, NCH>{});
    __builtin_amdgcn_s_waitcnt(vm_wait(0));     // the unary
    if (!pix_ok) return;

    // ---- Potts: softmax(U + M), store Q_{t+1}
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int c = 0; c < CM; ++c) fin[i][c] += u[i][c];
        softmax_regs<CM, true>(fin[i], CM);
    }
    float* __restrict__ qd = a.dst + (size_t)b * CM * HW + (size_t)y * W + xo;
#pragma unroll
    for (int c = 0; c < CM; ++c)
        *reinterpret_cast<float2*>(qd + c * HW) = make_float2(fin[0][c], fin[1][c]);
}

// The first round of the k = 7 Potts update in the quad layout, on the
// tiles of stream_kernel<..., FIRST> (64 x 16 pixels, 512 threads, all planes
// of U staged at once, softmax(U) applied to the staged halo tile in LDS).
// Everything is on chip before the message, so its loop runs at the LDS
// rate, which the quad layout lowers; each lane keeps the unary of its two
// pixels, read from LDS before the softmax.
template <int CM, int CH>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void quad_first_kernel(const IterArgs a) {
    constexpr int K = 7, R = 3;
    constexpr int TW = kStreamTW, ROWS = kStreamRows, NWAVE = 8;
    constexpr int LW = TW + 2 * R, LH = ROWS + 2 * R;
    constexpr int LS = kQuadStride;
    constexpr int PLANE = quad_first_plane();
    constexpr int NI = PLANE / 64;               // 64-float loads per plane
    constexpr int NJ = (NI + NWAVE - 1) / NWAVE; // per wave and plane
    constexpr int NCH = (CM + CH - 1) / CH;
    constexpr unsigned kOob = 0x80000000u;
    static_assert(2 * 16 * ROWS == 512, "16 pixel quads per row, a lane pair each");
    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qs = smem;                      // [CM][PLANE]
    float* const Cs = smem + CM * PLANE;         // [3][PLANE]
    float* const dummy = Cs + 3 * PLANE;         // one 256-float row
    const unsigned lds0 = (unsigned)(size_t)(__attribute__((address_space(3))) float*)smem;
    auto lds_addr = [&](const float* p) { return lds0 + (unsigned)((p - smem) * 4); };

    const int H = a.H, W = a.W;
    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * ROWS;
    const int x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t HW = (size_t)H * W;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int half = tid & 1, ty = tid >> 5;
    const int cq = 4 * ((tid >> 1) & 15);
    const int y = y0 + ty, xo = x0 + cq + 2 * half;
    const bool pix_ok = y < H && x0 + cq < W;

    // ---- every load into LDS: the colours, then U class by class
    unsigned voff[NJ];
    int dst[NJ];
#pragma unroll
    for (int s = 0; s < NJ; ++s) {
        const int j = wave + NWAVE * s;
        const int f = j * 64 + lane;
        const int r = f / LS, col = f - (f / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        const bool in = j < NI && f < LH * LS && col < LW && gy >= 0 && gy < H && gx >= 0 && gx < W;
        voff[s] = in ? (unsigned)((gy * W + gx) * 4) : kOob;
        dst[s] = j < NI ? j * 64 : -1;
    }
    const rsrc_t rf = buffer_rsrc(a.feat + (size_t)b * 3 * HW, (unsigned)(3 * HW * 4));
    const rsrc_t rq = buffer_rsrc(a.src + (size_t)b * CM * HW, (unsigned)(CM * HW * 4));
#pragma unroll
    for (int ch = 0; ch < 3; ++ch)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rf, voff[s], (int)(ch * HW * 4),
                    lds_addr(dst[s] >= 0 ? Cs + ch * PLANE + dst[s] : dummy));
    for (int c = 0; c < CM; ++c)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rq, voff[s], (int)(c * HW * 4),
                    lds_addr(dst[s] >= 0 ? Qs + c * PLANE + dst[s] : dummy));

    const unsigned rbase = (unsigned)((ty + (R + 1) * half) * LS + cq);
    const unsigned hbase = (unsigned)((ty + R) * LS + cq + (R + 1) * half);

    // ---- colours landed (the class planes may not have): the weights
    // (a wait beyond the 63 loads a wave can have outstanding is clamped:
    // the loads before the last 63 issued have completed by then)
    __builtin_amdgcn_s_waitcnt(vm_wait(NJ * CM));
    __syncthreads();
    float w[4][4][K];
    {
        float own[3][4];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            float r[10];
            lds_row16<10>(Cs + ch * PLANE + (ty + R) * LS + cq, r);
#pragma unroll
            for (int i = 0; i < 4; ++i) own[ch][i] = r[R + i];
        }
#pragma unroll
        for (int j = 0; j < R; ++j) {
            float nc[3][10];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) lds_row16<10>(Cs + ch * PLANE + rbase + j * LS, nc[ch]);
#pragma unroll
            for (int dx = 0; dx < K; ++dx) {
                const int ne = (dx - R) * (dx - R) + (R - j) * (R - j);
                const int no = (dx - R) * (dx - R) + (j + 1) * (j + 1);
                float ae = a.taps.app_log2[ne], ao = a.taps.app_log2[no];
                float se = a.taps.smooth[ne], so = a.taps.smooth[no];
                asm volatile("" : "+s"(ae), "+s"(ao), "+s"(se), "+s"(so));
                const float ca = half ? ao : ae;
                const float cs = half ? so : se;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    w[j][i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, ca)) + cs;
                }
            }
        }
        float hc[3][6];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) lds_row16<6>(Cs + ch * PLANE + hbase, hc[ch]);
#pragma unroll
        for (int d = 0; d < R; ++d) {
            const int nl = (R - d) * (R - d), nr = (d + 1) * (d + 1);
            float al = a.taps.app_log2[nl], ar = a.taps.app_log2[nr];
            float sl = a.taps.smooth[nl], sr = a.taps.smooth[nr];
            asm volatile("" : "+s"(al), "+s"(ar), "+s"(sl), "+s"(sr));
            const float ca = half ? ar : al;
            const float cs = half ? sr : sl;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float d0 = own[0][i] - hc[0][i + d];
                const float d1 = own[1][i] - hc[1][i + d];
                const float d2 = own[2][i] - hc[2][i + d];
                const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                w[3][i][d] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, ca)) + cs;
            }
        }
    }
    __builtin_amdgcn_sched_barrier(0);

    // ---- every plane landed: the lane's unary (Z = U + M, Potts), then
    // softmax(U) over the staged in-image positions (outside stays zero)
    __builtin_amdgcn_s_waitcnt(vm_wait(0));
    __syncthreads();
    float fin[2][CM];
    // staged column of the lane's first pixel: cq + 2 half + R (odd: two
    // dword reads)
    const int upos = (ty + R) * LS + cq + 2 * half + R;
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        fin[0][c] = Qs[c * PLANE + upos];
        fin[1][c] = Qs[c * PLANE + upos + 1];
    }
    __syncthreads();
    for (int pos = tid; pos < LH * LS; pos += 512) {
        const int r = pos / LS, col = pos - (pos / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        if (col >= LW || gy < 0 || gy >= H || gx < 0 || gx >= W) continue;
        float z[CM];
#pragma unroll
        for (int c = 0; c < CM; ++c) z[c] = Qs[c * PLANE + pos];
        softmax_regs<CM, true>(z, CM);
#pragma unroll
        for (int c = 0; c < CM; ++c) Qs[c * PLANE + pos] = z[c];
    }
    __syncthreads();

    // ---- the message, chunk by chunk, each chunk's pair sums added to fin
    static_for([&](auto kc) {
        constexpr int k = decltype(kc)::value;
        constexpr int c_lo = k * CH;
        constexpr int c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
        float acc[4][c_hi - c_lo];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int c = 0; c < c_hi - c_lo; ++c) acc[i][c] = 0.f;
        quad_chunk<PLANE, LS, c_lo, c_hi>(Qs, rbase, hbase, w, acc);
#pragma unroll
        for (int c = 0; c < c_hi - c_lo; ++c)
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float mine = half ? acc[2 + i][c] : acc[i][c];
                const float send = half ? acc[i][c] : acc[2 + i][c];
                fin[i][c_lo + c] += mine + pair_swap(send);
                asm volatile("" : "+v"(fin[i][c_lo + c]));
            }
    }, std::make_integer_sequence<int, NCH>{});
    if (!pix_ok) return;

#pragma unroll
    for (int i = 0; i < 2; ++i) softmax_regs<CM, true>(fin[i], CM);
    float* __restrict__ qd = a.dst + (size_t)b * CM * HW + (size_t)y * W + xo;
#pragma unroll
    for (int c = 0; c < CM; ++c)
        *reinterpret_cast<float2*>(qd + c * HW) = make_float2(fin[0][c], fin[1][c]);
}

template <int CM, int CH>
hipError_t launch_quad_first(const IterArgs& a, hipStream_t stream) {
    auto fn = quad_first_kernel<CM, CH>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(512), stream_lds_bytes(7, CM, false), stream, a);
    return hipGetLastError();
}

template <int CM, int CH>
hipError_t launch_quad(const IterArgs& a, hipStream_t stream) {
    auto fn = quad_kernel<CM, CH>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles), dim3(256), ring_lds_bytes(7, CM, CH, false, 0), stream, a);
    return hipGetLastError();
}

// ---------------------------------------------------- resident streamed form
// All T iterations in one cooperative launch on the tiles of stream_kernel
// (every tile's work-group co-resident).  The window weights (the colours do
// not change) and the unary of each thread's pixels stay in registers for
// the whole call; Q_t of the tile stays in LDS.  Between iterations a tile
// writes only its r-pixel border ring to an exchange buffer (agent-scope
// atomic stores), synchronises with its up to eight neighbours
// (neighbour_sync_coherent) and reads the r-pixel frame around it back from
// theirs (agent-scope atomic loads).  Potts compatibility only.
template <int K, int CM, int CH>
__global__ __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(2, 2)))
void rstream_kernel(const IterArgs a) {
    using SS = StreamShape<K>;
    constexpr int R = SS::R, LW = SS::LW, LH = SS::LH, LS = SS::LS;
    constexpr int PLANE = SS::PLANE, NI = SS::NI, NJ = SS::NJ;
    constexpr int P = 2, TW = SS::TW, ROWS = SS::ROWS, TPR = TW / P;
    constexpr int NW = P + K - 1, CTR = R * K + R;
    constexpr int NCH = (CM + CH - 1) / CH;
    constexpr unsigned kOob = 0x80000000u;
    static_assert(ROWS >= 2 * R && TW >= 2 * R, "border rings of a tile do not overlap");

    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qs = smem;                      // [CM][PLANE]
    float* const Cs = smem + CM * PLANE;         // [3][PLANE]
    float* const dummy = Cs + 3 * PLANE;         // one 256-float row
    const unsigned lds0 = (unsigned)(size_t)(__attribute__((address_space(3))) float*)smem;
    auto lds_addr = [&](const float* q) { return lds0 + (unsigned)((q - smem) * 4); };

    const int H = a.H, W = a.W;
    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * ROWS;
    const int x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t HW = (size_t)H * W;
    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;

    // ---- stage the colours and U (the source of the first iteration)
    unsigned voff[NJ];
    int dst[NJ];
#pragma unroll
    for (int s = 0; s < NJ; ++s) {
        const int j = wave + 8 * s;
        const int f = j * 64 + lane;
        const int r = f / LS, col = f - (f / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        const bool in = j < NI && f < LH * LS && col < LW && gy >= 0 && gy < H && gx >= 0 && gx < W;
        voff[s] = in ? (unsigned)((gy * W + gx) * 4) : kOob;
        dst[s] = j < NI ? j * 64 : -1;
    }
    const rsrc_t rf = buffer_rsrc(a.feat + (size_t)b * 3 * HW, (unsigned)(3 * HW * 4));
    const rsrc_t rq = buffer_rsrc(a.src + (size_t)b * CM * HW, (unsigned)(CM * HW * 4));
#pragma unroll
    for (int ch = 0; ch < 3; ++ch)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rf, voff[s], (int)(ch * HW * 4),
                    lds_addr(dst[s] >= 0 ? Cs + ch * PLANE + dst[s] : dummy));
    for (int c = 0; c < CM; ++c)
#pragma unroll
        for (int s = 0; s < NJ; ++s)
            lds_dma(rq, voff[s], (int)(c * HW * 4),
                    lds_addr(dst[s] >= 0 ? Qs + c * PLANE + dst[s] : dummy));

    const int tx = tid % TPR, ty = tid / TPR;
    const int col0 = tx * P;
    const int y = y0 + ty, xb = x0 + col0;
    const bool pix_ok = y < H && xb < W;        // W even: both pixels or neither

    // ---- the window weights, once for all iterations
    __builtin_amdgcn_s_waitcnt(vm_wait(NJ * CM));   // (clamped: see stream_kernel)
    __syncthreads();
    float w[K][P][K];
    {
        float own[3][P];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch)
#pragma unroll
            for (int i = 0; i < P; ++i) own[ch][i] = Cs[ch * PLANE + (ty + R) * LS + col0 + R + i];
#pragma unroll
        for (int dy = 0; dy < K; ++dy) {
            float nc[3][NW];
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) lds_row<NW, P>(Cs + ch * PLANE + (ty + dy) * LS + col0, nc[ch]);
#pragma unroll
            for (int i = 0; i < P; ++i) {
#pragma unroll
                for (int dx = 0; dx < K; ++dx) {
                    if (dy * K + dx == CTR) { w[dy][i][dx] = 0.f; continue; }
                    const int n = (dx - R) * (dx - R) + (dy - R) * (dy - R);
                    const float d0 = own[0][i] - nc[0][i + dx];
                    const float d1 = own[1][i] - nc[1][i + dx];
                    const float d2 = own[2][i] - nc[2][i + dx];
                    const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                    w[dy][i][dx] = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[n])) +
                                   a.taps.smooth[n];
                }
            }
        }
    }
    // ---- the unary of this thread's pixels, then softmax(U) in place
    __builtin_amdgcn_s_waitcnt(vm_wait(0));
    __syncthreads();
    float u[P][CM];
#pragma unroll
    for (int c = 0; c < CM; ++c)
#pragma unroll
        for (int i = 0; i < P; ++i) u[i][c] = Qs[c * PLANE + (ty + R) * LS + col0 + R + i];
    __syncthreads();
    for (int pos = tid; pos < LH * LS; pos += 512) {
        const int r = pos / LS, col = pos - (pos / LS) * LS;
        const int gy = y0 - R + r, gx = x0 - R + col;
        if (col >= LW || gy < 0 || gy >= H || gx < 0 || gx >= W) continue;
        float z[CM];
#pragma unroll
        for (int c = 0; c < CM; ++c) z[c] = Qs[c * PLANE + pos];
        softmax_regs<CM, true>(z, CM);
#pragma unroll
        for (int c = 0; c < CM; ++c) Qs[c * PLANE + pos] = z[c];
    }
    __syncthreads();

    for (int it = 0;; ++it) {
        float acc[P][CM];
#pragma unroll
        for (int i = 0; i < P; ++i)
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] = 0.f;
        static_for([&](auto kc) {
            constexpr int k = decltype(kc)::value;
            constexpr int c_lo = k * CH;
            constexpr int c_hi = (k + 1) * CH < CM ? (k + 1) * CH : CM;
            message_chunk<K, P, LS, PLANE, CM, c_lo, c_hi>(Qs, ty, col0, w, acc);
        }, std::make_integer_sequence<int, NCH>{});
        if (a.include_center) {
#pragma unroll
            for (int c = 0; c < CM; ++c)
#pragma unroll
                for (int i = 0; i < P; ++i)
                    acc[i][c] = fmaf(a.center_w, Qs[c * PLANE + (ty + R) * LS + col0 + R + i], acc[i][c]);
        }
        // Potts: Q_{t+1} = softmax(U + M)
#pragma unroll
        for (int i = 0; i < P; ++i) {
#pragma unroll
            for (int c = 0; c < CM; ++c) acc[i][c] += u[i][c];
            softmax_regs<CM, true>(acc[i], CM);
        }
        if (it == a.iters - 1) {
            if (pix_ok) {
                float* __restrict__ qd = a.dst + (size_t)b * CM * HW + (size_t)y * W + xb;
#pragma unroll
                for (int c = 0; c < CM; ++c)
                    *reinterpret_cast<float2*>(qd + c * HW) = make_float2(acc[0][c], acc[1][c]);
            }
            break;
        }
        // Q_{t+1}: the interior back into LDS, the border ring to the
        // exchange buffer of this parity
        __syncthreads();                          // every read of Q_t is done
        float* __restrict__ ring = a.ring[(it + 1) & 1] + (size_t)b * CM * HW;
        if (pix_ok) {
            const bool border = ty < R || ty >= ROWS - R || col0 < R || col0 + 1 >= TW - R;
#pragma unroll
            for (int c = 0; c < CM; ++c) {
                // (an odd offset when r is odd: two single stores)
                float* q = Qs + c * PLANE + (ty + R) * LS + col0 + R;
                q[0] = acc[0][c];
                q[1] = acc[1][c];
                if (border) {
                    float* g = ring + c * HW + (size_t)y * W + xb;
                    __hip_atomic_store(g, acc[0][c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(g + 1, acc[1][c], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
        neighbour_sync_coherent(a.sync + 1, a.sync, tile, a.tiles_x, a.tiles_per_img / a.tiles_x,
                                (unsigned int)(it + 1));
        // the frame around the tile from the neighbours' rings (outside the
        // image stays zero)
        const float* __restrict__ nb = a.ring[(it + 1) & 1] + (size_t)b * CM * HW;
        constexpr int band = R * LW, side = R * (LH - 2 * R);
        for (int idx = tid; idx < 2 * band + 2 * side; idx += 512) {
            int r, cc;
            if (idx < 2 * band) {
                const int k2 = idx - (idx >= band ? band : 0);
                r = (idx >= band ? LH - R : 0) + k2 / LW;
                cc = k2 - (k2 / LW) * LW;
            } else {
                const int j = idx - 2 * band;
                const int k2 = j - (j >= side ? side : 0);
                r = R + k2 / R;
                cc = (j >= side ? LW - R : 0) + (k2 - (k2 / R) * R);
            }
            const int gy = y0 - R + r, gx = x0 - R + cc;
            if (gy < 0 || gy >= H || gx < 0 || gx >= W) continue;
            const float* g = nb + (size_t)gy * W + gx;
            float v[CM];
#pragma unroll
            for (int c = 0; c < CM; ++c)
                v[c] = __hip_atomic_load(g + c * HW, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
            for (int c = 0; c < CM; ++c) Qs[c * PLANE + r * LS + cc] = v[c];
        }
        __syncthreads();
    }
}

// Cooperative: the runtime refuses the launch (rather than a neighbour wait
// never ending) unless every work-group is co-resident; the occupancy query
// refuses it first when the tiles cannot all be resident at once.
template <int K, int CM, int CH>
hipError_t launch_rstream(const IterArgs& a, size_t lds, int num_cus, hipStream_t stream,
                          bool probe) {
    auto fn = rstream_kernel<K, CM, CH>;
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(fn), 512, lds);
    if (e != hipSuccess) return e;
    if ((long long)per_cu * num_cus < a.ntiles) return hipErrorCooperativeLaunchTooLarge;
    if (probe) return hipSuccess;
    IterArgs args = a;
    void* params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void*>(fn), dim3(a.ntiles), dim3(512),
                                      params, (unsigned int)lds, stream);
}

// ------------------------------------------------------------ pooled message
// The message of the blur path (Sec. 4.2) on the s x s pooled grid, which is
// small (128 x 128 cells at 512^2, s = 4), so parallelism comes from the
// window: one wavefront per window row.  A work-group owns a tile of 16 x 8
// cells and a chunk of at most CM classes; it stages the chunk's planes and
// the pooled colours with their r-cell halo (zeros outside the grid), every
// wave computes the weights of its window row once (2 cells per lane) and
// applies them to all classes of the chunk, and the k row partials are
// summed in LDS, each wave finalising every k-th class.  Output: the raw
// message M (no compatibility, unary or softmax).  FD > 0: learnable
// smoothness features (the "+T" variant of Sec. 4.2) pooled to the cells
// like the colours, staged beside them; the smoothness Gaussian of each
// weight is taken on the pooled feature distance.
template <int K>
struct PmsgShape {
    static constexpr int R = (K - 1) / 2, P = 2, TW = 16, TH = 8;
    static constexpr int LW = TW + 2 * R, LH = TH + 2 * R, LS = (LW + 1) / 2 * 2;
    static constexpr int PLANE = LH * LS, NPX = TW * TH;
};

template <int K, int CM, int FD>
__global__ __launch_bounds__(64 * K) void pmsg_kernel(const IterArgs a) {
    using PS = PmsgShape<K>;
    constexpr int R = PS::R, P = PS::P, TW = PS::TW, TH = PS::TH, LW = PS::LW, LH = PS::LH;
    constexpr int LS = PS::LS, PLANE = PS::PLANE, NPX = PS::NPX;
    constexpr int TPR = TW / P, NW = P + K - 1;
    static_assert(TPR * TH == 64, "one wavefront per window row");

    extern __shared__ float4 smem4[];
    float* const smem = reinterpret_cast<float*>(smem4);
    float* const Qs = smem;                      // [CM][PLANE]
    float* const Cs = smem + CM * PLANE;         // [3][PLANE]
    float* const Fs = Cs + 3 * PLANE;            // [FD][PLANE] pooled features
    float* const Ps = Fs + FD * PLANE;           // [K][CM][NPX] row partials

    const int C = min(a.C, a.planes - (int)blockIdx.y * a.C);
    const int H = a.H, W = a.W;
    const int tile = xcd_tile(blockIdx.x, a.ntiles);
    const int b = tile / a.tiles_per_img;
    const int trem = tile - b * a.tiles_per_img;
    const int tyi = trem / a.tiles_x;
    const int y0 = tyi * TH, x0 = (trem - tyi * a.tiles_x) * TW;
    const size_t HW = (size_t)H * W;
    const float* __restrict__ src = a.src + ((size_t)b * a.planes + (size_t)blockIdx.y * a.C) * HW;
    const float* __restrict__ feat = a.feat + (size_t)b * 3 * HW;
    const float* __restrict__ sfeat = FD > 0 ? a.sfeat + (size_t)b * FD * HW : nullptr;

    // ---- stage the chunk's planes, the colours and the features, zero
    // outside the grid; every load of a thread is issued before its LDS stores
    constexpr int NT = 64 * K;
    constexpr int PER = ((CM + 3 + FD) * LH * LW + NT - 1) / NT;
    const int tid = threadIdx.x;
    const int nstage = (C + 3 + FD) * LH * LW;
    float v[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int idx = tid + j * NT;
        const int pl = idx / (LH * LW), rem = idx - pl * (LH * LW);
        const int r = rem / LW, cc = rem - (rem / LW) * LW;
        const int gy = y0 - R + r, gx = x0 - R + cc;
        const bool in = idx < nstage && gy >= 0 && gy < H && gx >= 0 && gx < W;
        const size_t g = in ? (size_t)gy * W + gx : 0;
        v[j] = in ? (pl < C       ? src[(size_t)pl * HW + g]
                     : pl < C + 3 ? feat[(size_t)(pl - C) * HW + g]
                                  : sfeat[(size_t)(pl - C - 3) * HW + g])
                  : 0.f;
    }
#pragma unroll
    for (int j = 0; j < PER; ++j) {
        const int idx = tid + j * NT;
        if (idx >= nstage) continue;
        const int pl = idx / (LH * LW), rem = idx - pl * (LH * LW);
        const int r = rem / LW, cc = rem - (rem / LW) * LW;
        (pl < C ? Qs + pl * PLANE : pl < C + 3 ? Cs + (pl - C) * PLANE : Fs + (pl - C - 3) * PLANE)
            [r * LS + cc] = v[j];
    }
    __syncthreads();

    // ---- window row g of both cells of this lane
    const int grp = tid >> 6, lane = tid & 63;
    const int tx = lane % TPR, ty = lane / TPR, col0 = tx * P;
    float w[P][K];
    {
        float own[3][P], nc[3][NW];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
#pragma unroll
            for (int i = 0; i < P; ++i) own[ch][i] = Cs[ch * PLANE + (ty + R) * LS + col0 + R + i];
            lds_row<NW, P>(Cs + ch * PLANE + (ty + grp) * LS + col0, nc[ch]);
        }
        // FD: the squared feature distance of every tap of the row
        float fd2[P][K];
        if constexpr (FD > 0) {
#pragma unroll
            for (int i = 0; i < P; ++i)
#pragma unroll
                for (int dx = 0; dx < K; ++dx) fd2[i][dx] = 0.f;
#pragma unroll
            for (int ch = 0; ch < FD; ++ch) {
                float fo[P], nf[NW];
#pragma unroll
                for (int i = 0; i < P; ++i) fo[i] = Fs[ch * PLANE + (ty + R) * LS + col0 + R + i];
                lds_row<NW, P>(Fs + ch * PLANE + (ty + grp) * LS + col0, nf);
#pragma unroll
                for (int i = 0; i < P; ++i)
#pragma unroll
                    for (int dx = 0; dx < K; ++dx) {
                        const float e = fo[i] - nf[i + dx];
                        fd2[i][dx] = fmaf(e, e, fd2[i][dx]);
                    }
            }
        }
        const int dy = grp - R;
#pragma unroll
        for (int i = 0; i < P; ++i) {
#pragma unroll
            for (int dx = 0; dx < K; ++dx) {
                const int n = (dx - R) * (dx - R) + dy * dy;
                const float d0 = own[0][i] - nc[0][i + dx];
                const float d1 = own[1][i] - nc[1][i + dx];
                const float d2 = own[2][i] - nc[2][i + dx];
                const float col2 = fmaf(d2, d2, fmaf(d1, d1, d0 * d0));
                const float smo = FD > 0 ? a.w_smooth * __builtin_amdgcn_exp2f(a.neg_gamma * fd2[i][dx])
                                         : a.taps.smooth[n];
                const float v = __builtin_amdgcn_exp2f(fmaf(col2, a.neg_beta, a.taps.app_log2[n])) +
                                smo;
                // the centre: excluded, or K(p, p) when it is included
                w[i][dx] = (n == 0) ? (a.include_center ? a.center_w : 0.f) : v;
            }
        }
    }
    float acc[P][CM];
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (c >= C) {
#pragma unroll
            for (int i = 0; i < P; ++i) acc[i][c] = 0.f;
            continue;
        }
        float q[NW];
        lds_row<NW, P>(Qs + c * PLANE + (ty + grp) * LS + col0, q);
#pragma unroll
        for (int i = 0; i < P; ++i) {
            float t = 0.f;
#pragma unroll
            for (int dx = 0; dx < K; ++dx) t = fmaf(w[i][dx], q[i + dx], t);
            acc[i][c] = t;
        }
    }
    // ---- sum the K row partials; wave g finalises classes g, g + K, ...
#pragma unroll
    for (int c = 0; c < CM; ++c) {
        if (c >= C) continue;
        *reinterpret_cast<float2*>(Ps + (grp * CM + c) * NPX + ty * TW + col0) =
            make_float2(acc[0][c], acc[1][c]);
    }
    __syncthreads();
    const int y = y0 + ty, xb = x0 + col0;
    if (y >= H) return;
    float* __restrict__ dst = a.dst + ((size_t)b * a.planes + (size_t)blockIdx.y * a.C) * HW +
                              (size_t)y * W + xb;
    for (int c = grp; c < C; c += K) {
        float m0 = 0.f, m1 = 0.f;
        for (int gg = 0; gg < K; ++gg) {
            const float2 t = *reinterpret_cast<const float2*>(Ps + (gg * CM + c) * NPX + ty * TW + col0);
            m0 += t.x;
            m1 += t.y;
        }
        if (xb < W) dst[(size_t)c * HW] = m0;
        if (xb + 1 < W) dst[(size_t)c * HW + 1] = m1;
    }
}

template <int K>
hipError_t launch_pmsg_cm(const IterArgs& a, int nchunks, size_t lds, hipStream_t stream) {
    auto fn = pmsg_kernel<K, kPmsgClasses, 0>;
    switch (a.sfeat ? a.D : 0) {
        case 0: break;
        case 1: fn = pmsg_kernel<K, kPmsgClasses, 1>; break;
        case 2: fn = pmsg_kernel<K, kPmsgClasses, 2>; break;
        case 3: fn = pmsg_kernel<K, kPmsgClasses, 3>; break;
        case 4: fn = pmsg_kernel<K, kPmsgClasses, 4>; break;
        default: return hipErrorInvalidValue;
    }
    hipError_t e = allow_full_lds(fn);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(fn, dim3(a.ntiles, nchunks), dim3(64 * K), lds, stream, a);
    return hipGetLastError();
}

// The built tile shapes: P = 2 or 4 pixels per thread, width 32.
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
    if (tile.width != 32) return hipErrorInvalidValue;
    if ((tile.width / tile.pix) * tile.rows % 64 != 0) return hipErrorInvalidValue;  // whole waves
    if (tile.threads() > (tile.pix == 4 ? 256 : 512)) return hipErrorInvalidValue;
    if (a.mode != kModeUpdate || a.planes != a.C) return hipErrorInvalidValue;
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

// Resident streamed form: k = 3, 5, 7, C = 19 or 21, Potts, vector path.
hipError_t CRF_CAT(launch_rstream_k, CRF_K)(const IterArgs& a, size_t lds, int num_cus,
                                            hipStream_t stream, bool probe) {
    constexpr int K = CRF_K;
    if constexpr (K < 3 || K > 7) {
        return hipErrorNotSupported;
    } else {
        if (a.mode != kModeUpdate || a.planes != a.C || !a.vec || (a.W & 3) || a.mu != nullptr ||
            a.iters < 2 || reinterpret_cast<uintptr_t>(a.src) % 16 != 0 ||
            (size_t)a.C * a.H * a.W * 4 >= (1ull << 31))
            return hipErrorNotSupported;
        switch (a.C) {
            case 19: return launch_rstream<K, 19, 4>(a, lds, num_cus, stream, probe);
            case 21: return launch_rstream<K, 21, 3>(a, lds, num_cus, stream, probe);
            default: return hipErrorNotSupported;
        }
    }
}

// Pooled message of the blur path, any k, chunks of at most kPmsgClasses.
hipError_t CRF_CAT(launch_pmsg_k, CRF_K)(const IterArgs& a, int nchunks, size_t lds,
                                         hipStream_t stream) {
    if (a.mode != kModeMessage || a.C < 1 || a.C > kPmsgClasses || nchunks < 1 ||
        nchunks * a.C < a.planes || (nchunks - 1) * a.C >= a.planes)
        return hipErrorInvalidValue;
    return launch_pmsg_cm<CRF_K>(a, nchunks, lds, stream);
}

// Streamed updates are built for k = 3, 5, 7 and the class counts 19 and 21.
hipError_t CRF_CAT(launch_stream_k, CRF_K)(const IterArgs& a, size_t lds, hipStream_t stream) {
    constexpr int K = CRF_K;
    if constexpr (K < 3 || K > 7) {
        return hipErrorNotSupported;
    } else {
        if (a.mode != kModeUpdate || a.planes != a.C || !a.vec || (a.W & 3) ||
            reinterpret_cast<uintptr_t>(a.unary) % 16 != 0 ||
            (size_t)a.C * a.H * a.W * 4 >= (1ull << 31))
            return hipErrorNotSupported;
        switch (a.C) {
            case 19: return launch_stream<K, 19, 4>(a, lds, stream);
            case 21: return launch_stream<K, 21, 3>(a, lds, stream);
            default: return hipErrorNotSupported;
        }
    }
}

// Ring updates: as the streamed ones, later iterations only (the source is
// Q_t), on kStreamTW x kRingRows tiles.
hipError_t CRF_CAT(launch_ring_k, CRF_K)(const IterArgs& a, hipStream_t stream) {
    constexpr int K = CRF_K;
    if constexpr (K < 3 || K > 7) {
        return hipErrorNotSupported;
    } else {
        if (a.mode != kModeUpdate || a.first || a.planes != a.C || !a.vec || (a.W & 3) ||
            (size_t)a.C * a.H * a.W * 4 >= (1ull << 31) ||
            (a.sfeat && (a.D < 1 || a.D > kMaxFeat || (size_t)a.D * a.H * a.W * 4 >= (1ull << 31))))
            return hipErrorNotSupported;
        switch (a.C) {
            case 19: return launch_ring<K, 19, 4>(a, stream);
            case 21: return launch_ring<K, 21, 3>(a, stream);
            default: return hipErrorNotSupported;
        }
    }
}

#if CRF_K == 7
// Quad updates: the ring's rounds 2..T at k = 7 with Potts compatibility,
// no centre tap and no learnable features.
hipError_t launch_quad_k7(const IterArgs& a, hipStream_t stream) {
    if (a.mode != kModeUpdate || a.first || a.planes != a.C || !a.vec || (a.W & 3) || a.mu ||
        a.include_center || a.sfeat || (size_t)a.C * a.H * a.W * 4 >= (1ull << 31))
        return hipErrorNotSupported;
    switch (a.C) {
        case 19: return launch_quad<19, 4>(a, stream);
        case 21: return launch_quad<21, 3>(a, stream);
        default: return hipErrorNotSupported;
    }
}

// The first round in the quad layout on the streamed tiles (a.first, the
// source U; the unary 16-byte aligned as for stream_kernel).
hipError_t launch_quad_first_k7(const IterArgs& a, hipStream_t stream) {
    if (a.mode != kModeUpdate || !a.first || a.planes != a.C || !a.vec || (a.W & 3) || a.mu ||
        a.include_center || a.sfeat || reinterpret_cast<uintptr_t>(a.unary) % 16 != 0 ||
        (size_t)a.C * a.H * a.W * 4 >= (1ull << 31))
        return hipErrorNotSupported;
    switch (a.C) {
        case 19: return launch_quad_first<19, 4>(a, stream);
        case 21: return launch_quad_first<21, 3>(a, stream);
        default: return hipErrorNotSupported;
    }
}
#endif

// Resident launches are built for the two-pixel, one-group tile of k <= 7
// and Potts compatibility.
hipError_t CRF_CAT(launch_resident_k, CRF_K)(const IterArgs& a, TileConfig tile, size_t lds,
                                             int num_cus, hipStream_t stream, bool probe) {
    constexpr int K = CRF_K;
    if constexpr (K > 7) {
        return hipErrorNotSupported;
    } else {
        if (tile.pix != 2 || tile.width != 32 || tile.threads() > 512 ||
            a.mode != kModeUpdate || a.iters < 2 || a.planes != a.C || a.mu != nullptr)
            return hipErrorNotSupported;
        switch (a.C) {
            case 19: return launch_res<K, 19, true>(a, tile, lds, num_cus, stream, probe);
            case 21: return launch_res<K, 21, true>(a, tile, lds, num_cus, stream, probe);
            default: break;
        }
        if (a.C <= 4) return launch_res<K, 4, false>(a, tile, lds, num_cus, stream, probe);
        if (a.C <= 8) return launch_res<K, 8, false>(a, tile, lds, num_cus, stream, probe);
        if (a.C <= 16) return launch_res<K, 16, false>(a, tile, lds, num_cus, stream, probe);
        return launch_res<K, 24, false>(a, tile, lds, num_cus, stream, probe);
    }
}

}  // namespace convcrf
