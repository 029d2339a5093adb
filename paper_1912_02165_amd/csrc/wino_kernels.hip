// HIP kernels of the Winograd F(m x m, 3 x 3) convolution on gfx950 other than the
// fused kernel (wino_ws.h, instantiated per blocking by wino_fused_inst.hip): the
// kernel transform, the three-stage pipeline, and the host-side choice and launch
// of the fused kernel's blocking.
#include "wino_ws.h"

#include <cstdio>

namespace wino {

// The fused kernel's instantiations live in their own objects.
#define WINO_EXTERN_WS(m, R, kit, tb, fs, csp)                                                              \
    extern template hipError_t launch_ws_t<m, tb, fs, csp>(const Geometry &, const float *, const float *, \
                                                           float *, bool, int, int, const SplitBuffers &,  \
                                                           hipStream_t);
WINO_FUSED_BLOCKINGS(WINO_EXTERN_WS)
#undef WINO_EXTERN_WS

// Load the T x T input tile of (tile, channel c) with implicit zero padding
// (Sec. 2.1): rows ty*M - 1 + a, columns tx*M - 1 + b.  Reads use clamped,
// always in-bounds addresses; out-of-image elements are then replaced by 0.
template <int M>
struct TileLoader {
    static constexpr int T = M + 2;
    int rowoff[T];
    int colc[T];
    unsigned rowok;  // bit a: row a inside the image (and the tile exists)
    unsigned colok;  // bit b: column b inside the image

    __device__ __forceinline__ void init(const Geometry &g, const TileIdx &t) {
        rowok = 0u;
        colok = 0u;
#pragma unroll
        for (int a = 0; a < T; ++a) {
            int h = t.ty * M - 1 + a;
            if (t.ok && h >= 0 && h < g.H) rowok |= 1u << a;
            rowoff[a] = clampi(h, 0, g.H - 1) * g.W;
        }
#pragma unroll
        for (int b = 0; b < T; ++b) {
            int w = t.tx * M - 1 + b;
            if (w >= 0 && w < g.W) colok |= 1u << b;
            colc[b] = clampi(w, 0, g.W - 1);
        }
    }

    // xc points at channel plane (n, c); cok says whether c < C.
    __device__ __forceinline__ void load(const float *__restrict__ xc, bool cok, float *d) const {
#pragma unroll
        for (int a = 0; a < T; ++a) {
            const float *xr = xc + rowoff[a];
            bool rok = cok && ((rowok >> a) & 1u);
#pragma unroll
            for (int b = 0; b < T; ++b) {
                float v = xr[colc[b]];
                d[a * T + b] = (rok && ((colok >> b) & 1u)) ? v : 0.0f;
            }
        }
    }
};

// ---------------------------------------------------------------------------
// Kernel transform (Sec. 3, step 2: right-hand matrices transformed ahead of
// time).  Thread (kb, cs, lane) transforms kernel (k, c) with k = 16 kb + lane%16,
// c = 4 cs + lane/16 and stores the T^2 values in matrix-core operand order:
// wt[((kb * Cs + cs) * Q + f/4) * 64 + lane][f % 4], Q = ceil(T^2/4).  Channels
// >= C, output channels >= K and frequencies >= T^2 are stored as zeros.
template <int M>
__global__ void __launch_bounds__(256) weight_transform_kernel(const float *__restrict__ w,
                                                               floatx4 *__restrict__ wt, Geometry g,
                                                               unsigned *zero, int nzero) {
    constexpr int T = M + 2, T2 = T * T;
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < nzero; i += blockDim.x) zero[i] = 0u;
    const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long total = (long long)g.Kb_alloc * g.Cs * 64;
    if (gid >= total) return;
    const int lane = (int)(gid & 63);
    const long long grp = gid >> 6;
    const int cs = (int)(grp % g.Cs);
    const int kb = (int)(grp / g.Cs);
    const int c = cs * 4 + (lane >> 4);
    const int k = kb * 16 + (lane & 15);
    float gk[9];
    const bool ok = (c < g.C) && (k < g.K);
    const float *src = w + ((long long)(ok ? k : 0) * g.C + (ok ? c : 0)) * 9;
#pragma unroll
    for (int i = 0; i < 9; ++i) gk[i] = ok ? src[i] : 0.0f;
    constexpr int Q = freq_quads<M>();
    float t[4 * Q];
    kernel_tile_transform<M>(gk, t);
#pragma unroll
    for (int f = T2; f < 4 * Q; ++f) t[f] = 0.0f;
    floatx4 *dst = wt + grp * Q * 64 + lane;
#pragma unroll
    for (int f4 = 0; f4 < Q; ++f4) {
        floatx4 v = {t[4 * f4], t[4 * f4 + 1], t[4 * f4 + 2], t[4 * f4 + 3]};
        dst[f4 * 64] = v;
    }
}

// ---------------------------------------------------------------------------
// Three-stage pipeline (Sec. 3): stage 1 writes U[f][c][tile] for all tiles,
// stage 2 forms M[f][k][tile] = sum_c W'[f][c][k] U[f][c][tile] for each f,
// stage 3 inverse-transforms M into y.  Padded rows (c >= C, k >= K, tile >= ntiles)
// of U and M hold zeros.

template <int M>
__global__ void __launch_bounds__(256) input_transform_kernel(const float *__restrict__ x,
                                                              float *__restrict__ U, Geometry g) {
    constexpr int T = M + 2, T2 = T * T;
    const int tile = blockIdx.x * blockDim.x + threadIdx.x;
    const int c = blockIdx.y;
    if (tile >= g.tiles_p) return;
    const TileIdx ti = decode_tile(g, tile);
    TileLoader<M> ld;
    ld.init(g, ti);
    const long long HW = (long long)g.H * g.W;
    const bool cok = c < g.C;
    float d[T2];
    ld.load(x + ((long long)ti.n * g.C + (cok ? c : 0)) * HW, cok, d);
    float u[T2];
    input_tile_transform<M>(d, u);
    const long long Cp = (long long)g.Cs * 4;
#pragma unroll
    for (int f = 0; f < T2; ++f) U[((long long)f * Cp + c) * g.tiles_p + tile] = u[f];
}

// Stage 2: per frequency f (blockIdx.z), each wave computes 64 output channels x
// 32 tiles with 4 x 2 matrix-core blocks.
template <int M>
__global__ void __launch_bounds__(256) frequency_gemm_kernel(const float *__restrict__ U,
                                                             const float *__restrict__ wt,
                                                             float *__restrict__ Mout, Geometry g) {
    constexpr int T = M + 2, T2 = T * T;
    constexpr int KBW = 4, TBW = 2;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int waves = blockDim.x >> 6;
    const int f = blockIdx.z;
    const int t0 = (blockIdx.x * waves + wave) * (16 * TBW);
    if (t0 >= g.tiles_p) return;
    const int kb0 = blockIdx.y * KBW;
    const long long Cp = (long long)g.Cs * 4;
    const long long Kp = (long long)g.Kb_alloc * 16;
    floatx4 acc[KBW][TBW];
#pragma unroll
    for (int i = 0; i < KBW; ++i)
#pragma unroll
        for (int j = 0; j < TBW; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const float *ub = U + ((long long)f * Cp + (lane >> 4)) * g.tiles_p + t0 + (lane & 15);
    const float *wb = wt + (long long)(f >> 2) * 256 + lane * 4 + (f & 3);
    for (int cs = 0; cs < g.Cs; ++cs) {
        float a[KBW], b[TBW];
#pragma unroll
        for (int i = 0; i < KBW; ++i) a[i] = wb[((long long)(kb0 + i) * g.Cs + cs) * (4 * freq_quads<M>()) * 64];
#pragma unroll
        for (int j = 0; j < TBW; ++j) b[j] = ub[(long long)cs * 4 * g.tiles_p + j * 16];
#pragma unroll
        for (int i = 0; i < KBW; ++i)
#pragma unroll
            for (int j = 0; j < TBW; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i], b[j], acc[i][j], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < KBW; ++i)
#pragma unroll
        for (int j = 0; j < TBW; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const long long k = (kb0 + i) * 16 + (lane >> 4) * 4 + v;
                Mout[((long long)f * Kp + k) * g.tiles_p + t0 + j * 16 + (lane & 15)] = acc[i][j][v];
            }
}

template <int M>
__global__ void __launch_bounds__(256) output_transform_kernel(const float *__restrict__ Min,
                                                               float *__restrict__ y, Geometry g) {
    constexpr int T = M + 2, T2 = T * T;
    const int tile = blockIdx.x * blockDim.x + threadIdx.x;
    const int k = blockIdx.y;
    if (tile >= g.ntiles) return;
    const TileIdx ti = decode_tile(g, tile);
    const long long Kp = (long long)g.Kb_alloc * 16;
    float mm[T2];
#pragma unroll
    for (int f = 0; f < T2; ++f) mm[f] = Min[((long long)f * Kp + k) * g.tiles_p + tile];
    float yy[M * M];
    output_tile_transform<M>(mm, yy);
    const long long HW = (long long)g.H * g.W;
    float *yp = y + ((long long)ti.n * g.K + k) * HW;
#pragma unroll
    for (int i = 0; i < M; ++i) {
        const int h = ti.ty * M + i;
        if (h < g.H) {
#pragma unroll
            for (int j = 0; j < M; ++j) {
                const int w = ti.tx * M + j;
                if (w < g.W) yp[(long long)h * g.W + w] = yy[i * M + j];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Launchers.

#define WINO_DISPATCH_M(m, CALL)          \
    switch (m) {                          \
        case 2: { constexpr int MM = 2; CALL; } break; \
        case 4: { constexpr int MM = 4; CALL; } break; \
        case 5: { constexpr int MM = 5; CALL; } break; \
        case 6: { constexpr int MM = 6; CALL; } break; \
        default: return hipErrorInvalidValue; \
    }

hipError_t launch_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s,
                                   unsigned *zero, int nzero) {
    const long long total = (long long)g.Kb_alloc * g.Cs * 64;
    dim3 block(256), grid((unsigned)((total + 255) / 256));
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(weight_transform_kernel<MM>, grid, block, 0, s, w,
                                            reinterpret_cast<floatx4 *>(wt), g, zero, nzero));
    return hipGetLastError();
}

bool fused_blocking_built(int m, int R, int kit) {
    for (const FusedBlocking &b : kFusedBlockings)
        if (b.m == m && b.R == R && b.kit == kit) return true;
    return false;
}

// Default blocking of a layer, from the capacity bounds of Sec. 4.1 and the
// number of work-item rounds.
//  * Capacity: a task's result matrices (R tiles x Kit output channels x T^2
//    frequencies) live in the consumer waves' registers, at most 144 per lane of
//    four waves: R * Kit * T^2 <= 36864.  F(2), F(4): R = 16 or 32 with Kit <= 64;
//    F(5), F(6): R = 16, Kit <= 32.
//  * Reuse: every transformed input tile is multiplied by the Kit output
//    channels' kernels (the input-transform cost per product falls as 1 / Kit),
//    and every transformed-kernel operand read from L2 by the R tiles (the
//    paper's task arithmetic intensity against the shared cache, R / 2).  So the
//    largest R and Kit that fit are preferred ...
//  * ... unless the layer has too few items to fill the compute units: the
//    estimated time of a blocking is its item cost (products plus input
//    transforms, in SIMD cycles) times the rounds of items the persistent grid
//    runs, including the split of a last, partly filled round; a smaller Kit is
//    taken when it is estimated at least 10 % faster.
FusedCfg fused_cfg_default(const Geometry &g, int num_cus, int want_R, int want_kit) {
    const int T2 = (g.m + 2) * (g.m + 2);
    // vector instructions of one input-tile transform (B^T d B), per tile and channel
    const double in_ops = g.m == 2 ? 32.0 : g.m == 4 ? 150.0 : g.m == 5 ? 270.0 : 390.0;
    FusedCfg best{};
    double best_t = 0.0;
    const int Rs[2] = {32, 16};
    const int kits[3] = {64, 32, 16};
    for (int R : Rs) {
        for (int kit : kits) {
            if (!fused_blocking_built(g.m, R, kit) || (want_R && R != want_R) || (want_kit && kit != want_kit))
                continue;
            FusedCfg c{R, kit, num_cus, 0};
            const SplitInfo si = fused_split_info(g, c);
            // SIMD cycles per item: products (32 multiply-adds per cycle) and
            // input transforms (16 lane-operations per cycle), over 4 SIMDs
            const double per_tc = (double)kit * T2 / 32.0 + in_ops / 16.0;
            const double item = (double)R * g.C * per_tc / 4.0;
            double rounds = (double)si.nfull;
            if (si.n_tail > 0) {
                rounds += (double)((si.n_units + num_cus - 1) / num_cus) / si.maxc;
            } else if (si.n_items > si.nfull * num_cus) {
                rounds += 1.0;
            }
            const double t = rounds * item;
            if (best.R == 0 || t < 0.9 * best_t) {
                best = c;
                best_t = t;
            }
        }
    }
    return best;
}

SplitInfo fused_split_info(const Geometry &g, const FusedCfg &cfg) {
#define WINO_SPLIT_WS(m_, R_, kit_, tb, fs, csp) \
    if (g.m == m_ && cfg.R == R_ && cfg.kit == kit_) return ws_split_info<m_, tb, fs, csp>(g, cfg.num_cus, cfg.csplit);
    WINO_FUSED_BLOCKINGS(WINO_SPLIT_WS)
#undef WINO_SPLIT_WS
    return SplitInfo{};
}

void describe_fused(const Geometry &g, const FusedCfg &cfg, char *buf, size_t len) {
    const SplitInfo si = fused_split_info(g, cfg);
    int tb = 0, fs = 0, csp = 0;
    for (const FusedBlocking &b : kFusedBlockings)
        if (b.m == g.m && b.R == cfg.R && b.kit == cfg.kit) {
            tb = b.tb;
            fs = b.fs;
            csp = b.csp;
        }
    snprintf(buf, len,
             "fused_ws_kernel<M=%d,TB=%d,FS=%d,CSP=%d,VX,SPLIT=%d> R=%d tiles x Kit=%d output channels per "
             "item, %d input channels per stage, %d items (%d tile groups x %d channel groups), %d stages per "
             "item, grid %d, split items %d x %d pieces",
             g.m, tb, fs, csp, si.n_tail > 0 ? 1 : 0, cfg.R, cfg.kit, 256 / cfg.R, si.n_items,
             si.n_kgroups > 0 ? si.n_items / si.n_kgroups : 0, si.n_kgroups, si.stages, si.grid, si.n_tail, si.maxc);
}

hipError_t launch_fused(const Geometry &g, const FusedCfg &cfg, const float *x, const float *wt,
                        float *y, const SplitBuffers &sb, hipStream_t s) {
    if (!fused_blocking_built(g.m, cfg.R, cfg.kit)) return hipErrorInvalidValue;
    const uintptr_t ya = reinterpret_cast<uintptr_t>(y);
    // rows of whole tiles stored as vectors: 16-byte aligned for m = 4, 8-byte for m =
    // 2, 6; m = 5 uses buffer stores that need only 4-byte alignment
    const bool vec = (g.m == 5) ? true
                     : (g.m == 4) ? (g.W % 4 == 0 && ya % 16 == 0) : (g.W % 2 == 0 && ya % 8 == 0);
#define WINO_LAUNCH_WS(m_, R_, kit_, tb, fs, csp)                                                         \
    if (g.m == m_ && cfg.R == R_ && cfg.kit == kit_)                                                        \
        return launch_ws_t<m_, tb, fs, csp>(g, x, wt, y, vec, cfg.num_cus, cfg.csplit, sb, s);
    WINO_FUSED_BLOCKINGS(WINO_LAUNCH_WS)
#undef WINO_LAUNCH_WS
    return hipErrorInvalidValue;
}

void describe_three_stage(const Geometry &g, char *buf, size_t len) {
    snprintf(buf, len, "input_transform_kernel<M=%d>, frequency_gemm_kernel<M=%d>, output_transform_kernel<M=%d>: "
             "%d tiles, U and M of %d frequencies in device memory", g.m, g.m, g.m, g.ntiles, g.T2);
}

hipError_t launch_input_transform(const Geometry &g, const float *x, float *U, hipStream_t s) {
    dim3 block(256), grid((unsigned)((g.tiles_p + 255) / 256), (unsigned)(g.Cs * 4));
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(input_transform_kernel<MM>, grid, block, 0, s, x, U, g));
    return hipGetLastError();
}

hipError_t launch_frequency_gemm(const Geometry &g, const float *U, const float *wt, float *Mout,
                                 hipStream_t s) {
    const int waves = 4, tiles_per_wave = 32;
    dim3 block(64 * waves);
    dim3 grid((unsigned)((g.tiles_p + waves * tiles_per_wave - 1) / (waves * tiles_per_wave)),
              (unsigned)(g.Kb_alloc / 4), (unsigned)g.T2);
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(frequency_gemm_kernel<MM>, grid, block, 0, s, U, wt, Mout, g));
    return hipGetLastError();
}

hipError_t launch_output_transform(const Geometry &g, const float *Min, float *y, hipStream_t s) {
    dim3 block(256), grid((unsigned)((g.ntiles + 255) / 256), (unsigned)g.K);
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(output_transform_kernel<MM>, grid, block, 0, s, Min, y, g));
    return hipGetLastError();
}

}  // namespace wino
