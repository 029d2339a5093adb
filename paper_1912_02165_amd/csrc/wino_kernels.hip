// HIP kernels for the Winograd F(m x m, 3 x 3) convolution on gfx950.
//
// Matrix-core mapping (v_mfma_f32_16x16x4_f32, one 64-lane wave):
//   D[16 x 16] += A[16 x 4] * B[4 x 16]
//   lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] and holds
//   D[4 * (l / 16) + v][l % 16], v = 0..3.
// Every product here is, for one frequency f, D[k][tile] += sum_c W'[f][c][k] U[f][c][tile]
// (Sec. 3, step 2), so A is a 16 (k) x 4 (c) slice of the transformed kernels and
// B a 4 (c) x 16 (tile) slice of the transformed input.  Lane l therefore works
// on tile l % 16 and channel l / 16 of each 4-channel step: it can build its own
// B operand for all T^2 frequencies from one input tile held in registers, and
// after the channel loop it holds, for its tile, all T^2 frequencies of four
// output channels, so the output transform also runs in registers.
#include "wino_internal.h"
#include "wino_transforms.h"

namespace wino {

typedef float floatx4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int clampi(int v, int lo, int hi) { return v < lo ? lo : (v > hi ? hi : v); }

// Index arithmetic of one tile: image n, tile row ty, tile column tx.
struct TileIdx {
    int n, ty, tx;
    bool ok;
};

__device__ __forceinline__ TileIdx decode_tile(const Geometry &g, int tile) {
    TileIdx t;
    t.ok = tile < g.ntiles;
    int tt = t.ok ? tile : 0;
    int per_img = g.TH * g.TW;
    t.n = tt / per_img;
    int rem = tt - t.n * per_img;
    t.ty = rem / g.TW;
    t.tx = rem - t.ty * g.TW;
    return t;
}

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
// wt[((kb * Cs + cs) * T^2/4 + f/4) * 64 + lane][f % 4].  Channels >= C and
// output channels >= K are stored as zeros.
template <int M>
__global__ void __launch_bounds__(256) weight_transform_kernel(const float *__restrict__ w,
                                                               floatx4 *__restrict__ wt, Geometry g) {
    constexpr int T = M + 2, T2 = T * T;
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
    float t[T2];
    kernel_tile_transform<M>(gk, t);
    floatx4 *dst = wt + grp * (T2 / 4) * 64 + lane;
#pragma unroll
    for (int f4 = 0; f4 < T2 / 4; ++f4) {
        floatx4 v = {t[4 * f4], t[4 * f4 + 1], t[4 * f4 + 2], t[4 * f4 + 3]};
        dst[f4 * 64] = v;
    }
}

// ---------------------------------------------------------------------------
// Fused kernel (Sec. 4: a task of R tiles does input transform -> T^2 products
// against the hot kernel matrices -> output transform).  Here a task is a
// workgroup of `waves` waves; each wave owns 16 consecutive tiles and the same
// NKB blocks of 16 output channels.  Per 4-channel step a lane loads one input
// tile, transforms it in registers (B^T d B) and feeds each frequency to the
// matrix core against the matching transformed-kernel slice, which every wave
// of the workgroup reads from the same cached lines.  The accumulators (the
// paper's result matrices) never leave registers; after the last step each lane
// inverse-transforms its tile for its four output channels and writes y.
template <int M, int NKB>
__global__ void __launch_bounds__(256) fused_kernel(const float *__restrict__ x,
                                                    const floatx4 *__restrict__ wt,
                                                    float *__restrict__ y, Geometry g) {
    constexpr int T = M + 2, T2 = T * T;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int waves = blockDim.x >> 6;
    const int tile = (blockIdx.x * waves + wave) * 16 + (lane & 15);
    const int cq = lane >> 4;
    const int kb0 = blockIdx.y * NKB;
    const TileIdx ti = decode_tile(g, tile);
    TileLoader<M> ld;
    ld.init(g, ti);
    const long long HW = (long long)g.H * g.W;
    const float *xn = x + (long long)ti.n * g.C * HW;

    floatx4 acc[NKB][T2];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int f = 0; f < T2; ++f) acc[kb][f] = floatx4{0.f, 0.f, 0.f, 0.f};

    for (int cs = 0; cs < g.Cs; ++cs) {
        const int c = cs * 4 + cq;
        const bool cok = c < g.C;
        float d[T2];
        ld.load(xn + (cok ? c : 0) * HW, cok, d);
        float u[T2];
        input_tile_transform<M>(d, u);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
            const floatx4 *wp = wt + ((long long)(kb0 + kb) * g.Cs + cs) * (T2 / 4) * 64 + lane;
#pragma unroll
            for (int f4 = 0; f4 < T2 / 4; ++f4) {
                const floatx4 a = wp[f4 * 64];
                acc[kb][4 * f4 + 0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], u[4 * f4 + 0], acc[kb][4 * f4 + 0], 0, 0, 0);
                acc[kb][4 * f4 + 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], u[4 * f4 + 1], acc[kb][4 * f4 + 1], 0, 0, 0);
                acc[kb][4 * f4 + 2] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], u[4 * f4 + 2], acc[kb][4 * f4 + 2], 0, 0, 0);
                acc[kb][4 * f4 + 3] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], u[4 * f4 + 3], acc[kb][4 * f4 + 3], 0, 0, 0);
            }
        }
    }

    // Output transform Y = A^T Mm A per (output channel, tile), clipped to H x W.
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int k = (kb0 + kb) * 16 + cq * 4 + v;
            float mm[T2];
#pragma unroll
            for (int f = 0; f < T2; ++f) mm[f] = acc[kb][f][v];
            float yy[M * M];
            output_tile_transform<M>(mm, yy);
            if (ti.ok && k < g.K) {
                float *yp = y + ((long long)ti.n * g.K + k) * HW;
#pragma unroll
                for (int i = 0; i < M; ++i) {
                    const int h = ti.ty * M + i;
                    if (h < g.H) {
#pragma unroll
                        for (int j = 0; j < M; ++j) {
                            const int w = ti.tx * M + j;
                            if (w < g.W) __builtin_nontemporal_store(yy[i * M + j], yp + (long long)h * g.W + w);
                        }
                    }
                }
            }
        }
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
        for (int i = 0; i < KBW; ++i) a[i] = wb[((long long)(kb0 + i) * g.Cs + cs) * T2 * 64];
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
        case 6: { constexpr int MM = 6; CALL; } break; \
        default: return hipErrorInvalidValue; \
    }

hipError_t launch_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s) {
    const long long total = (long long)g.Kb_alloc * g.Cs * 64;
    dim3 block(256), grid((unsigned)((total + 255) / 256));
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(weight_transform_kernel<MM>, grid, block, 0, s, w,
                                            reinterpret_cast<floatx4 *>(wt), g));
    return hipGetLastError();
}

bool fused_cfg_supported(int m, const FusedCfg &cfg) {
    if (cfg.waves < 1 || cfg.waves > 4) return false;
    switch (m) {
        case 2: return cfg.nkb == 1 || cfg.nkb == 2 || cfg.nkb == 4;
        case 4: return cfg.nkb == 1 || cfg.nkb == 2;
        case 6: return cfg.nkb == 1;
        default: return false;
    }
}

FusedCfg fused_cfg_default(const Geometry &g) {
    FusedCfg c;
    c.waves = 4;
    switch (g.m) {
        case 2: c.nkb = g.Kb >= 4 ? 4 : (g.Kb >= 2 ? 2 : 1); break;
        case 4: c.nkb = g.Kb >= 2 ? 2 : 1; break;
        default: c.nkb = 1; break;
    }
    return c;
}

template <int M, int NKB>
static void launch_fused_t(const Geometry &g, int waves, const float *x, const float *wt, float *y,
                           hipStream_t s) {
    const int tiles_per_group = 16 * waves;
    dim3 block(64 * waves);
    dim3 grid((unsigned)((g.ntiles + tiles_per_group - 1) / tiles_per_group),
              (unsigned)((g.Kb + NKB - 1) / NKB));
    hipLaunchKernelGGL((fused_kernel<M, NKB>), grid, block, 0, s, x,
                       reinterpret_cast<const floatx4 *>(wt), y, g);
}

hipError_t launch_fused(const Geometry &g, const FusedCfg &cfg, const float *x, const float *wt,
                        float *y, hipStream_t s) {
    if (!fused_cfg_supported(g.m, cfg)) return hipErrorInvalidValue;
    switch (g.m) {
        case 2:
            if (cfg.nkb == 1) launch_fused_t<2, 1>(g, cfg.waves, x, wt, y, s);
            else if (cfg.nkb == 2) launch_fused_t<2, 2>(g, cfg.waves, x, wt, y, s);
            else launch_fused_t<2, 4>(g, cfg.waves, x, wt, y, s);
            break;
        case 4:
            if (cfg.nkb == 1) launch_fused_t<4, 1>(g, cfg.waves, x, wt, y, s);
            else launch_fused_t<4, 2>(g, cfg.waves, x, wt, y, s);
            break;
        case 6:
            launch_fused_t<6, 1>(g, cfg.waves, x, wt, y, s);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
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
