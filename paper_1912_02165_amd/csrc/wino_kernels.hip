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
// Three-stage pipeline (Sec. 3): stage 1 writes the transformed input tiles U of
// all tiles to device memory, stage 2 forms M[f][k][tile] = sum_c W'[f][c][k]
// U[f][c][tile] for every frequency f, stage 3 inverse-transforms M into y.
// The intermediates are stored in the matrix-core operand order, four
// consecutive frequencies per 16-byte element, so that every stage moves them
// with one coalesced 1 KB access per wave and instruction:
//   U [F4][TB][Cs][64][4]:    element (f, c, tile) at f4 = f/4, tb = tile/16,
//                             cs = c/4, lane (c%4)*16 + tile%16, slot f%4 (the B
//                             operand of v_mfma_f32_16x16x4f32 for 4 frequencies);
//   M [F4][TB][Kb][4][64][4]: element (f, k, tile) at f4, tb, kb = k/16, v = k%4,
//                             lane ((k%16)/4)*16 + tile%16, slot f%4 (the
//                             accumulator layout: lane l holds D[4(l/16)+v][l%16]).
// TB = tiles_p / 16, Cs = ceil(C/4), Kb = Kb_alloc; channels, output channels and
// tiles past the problem hold zeros.

// Workgroup b of a 1-D grid of n runs on XCD b % 8; the index returned numbers the
// workgroups so that each XCD takes one contiguous range of them.
__device__ __forceinline__ int xcd_contiguous_block(int b, int n) {
    const int xcd = b % 8, per = n / 8, extra = n % 8;
    return xcd * per + (xcd < extra ? xcd : extra) + b / 8;
}

// Input tile of F(7x7,3x3) (T = 9, too wide for the row-vector loader's halo
// exchange within 16 lanes): per row the lane's own 7 columns as 4-byte-aligned
// vector loads (4 + 2 + 1 floats) and its two halo columns as single loads; rows
// and halo columns outside the image read as zero through the buffer range check,
// own columns past W (the last tile of a row) are cleared.
template <int M>
struct WideRowTile {
    static constexpr int T = M + 2;
    static_assert(M == 7, "loader of the 9 x 9 input tiles");
    unsigned roff[T];
    unsigned own, left, right, ownok;

    __device__ __forceinline__ void init(const Geometry &g, const TileIdx &t, int lane_c) {
        const unsigned base = (unsigned)(((long long)t.n * g.C + lane_c) * g.H * g.W) * 4u;
#pragma unroll
        for (int a = 0; a < T; ++a) {
            const int h = t.ty * M - 1 + a;
            roff[a] = (t.ok && h >= 0 && h < g.H) ? base + (unsigned)(h * g.W) * 4u : kOutside;
        }
        own = (unsigned)(t.tx * M) * 4u;
        left = t.tx > 0 ? own - 4u : kOutside;
        right = t.tx * M + M < g.W ? own + 4u * M : kOutside;
        ownok = 0u;
#pragma unroll
        for (int j = 0; j < M; ++j)
            if (t.tx * M + j < g.W) ownok |= 1u << j;
    }

    __device__ __forceinline__ void load(int32x4 r, float *d) const {
#pragma unroll
        for (int a = 0; a < T; ++a) {
            const unsigned ro = roff[a];
            const floatx4 q4 = buffer_load_f32x4(r, __builtin_elementwise_add_sat(ro, own), 0, 0);
            const floatx2 q2 = buffer_load_f32x2(r, __builtin_elementwise_add_sat(ro, own + 16u), 0, 0);
            const float q1 = buffer_load_f32(r, __builtin_elementwise_add_sat(ro, own + 24u), 0, 0);
            d[a * T] = buffer_load_f32(r, __builtin_elementwise_add_sat(ro, left), 0, 0);
            d[a * T + T - 1] = buffer_load_f32(r, __builtin_elementwise_add_sat(ro, right), 0, 0);
#pragma unroll
            for (int j = 0; j < 4; ++j) d[a * T + 1 + j] = q4[j];
            d[a * T + 5] = q2[0];
            d[a * T + 6] = q2[1];
            d[a * T + 7] = q1;
        }
        if (ownok != (1u << M) - 1u) {
#pragma unroll
            for (int a = 0; a < T; ++a)
#pragma unroll
                for (int j = 0; j < M; ++j)
                    if (!((ownok >> j) & 1u)) d[a * T + 1 + j] = 0.0f;
        }
    }
};

// Stage 1: the workgroup's 256 threads are 16 tiles x 16 channels (the producer
// mapping of the fused kernel: lane%16 = tile, so the row-vector loader's DPP halo
// exchange applies); each transforms its tile and stores one float4 per four
// frequencies.  Workgroups are numbered tile block fastest within a channel group
// and XCD-contiguously, so the input rows shared by vertically adjacent tiles
// (the two overlap rows of the windows) are read from HBM once and then from L2.
template <int M, bool VX>
__global__ void __launch_bounds__(256) input_transform_kernel(const float *__restrict__ x,
                                                              floatx4 *__restrict__ U, Geometry g) {
    constexpr int T2 = (M + 2) * (M + 2);
    const int tid = threadIdx.x, lane = tid & 63;
    const int tr = tid & 15, cl = tid >> 4;
    const int TB = g.tiles_p / 16;
    const int lb = xcd_contiguous_block(blockIdx.x, gridDim.x);
    const int tb = lb % TB, c = (lb / TB) * 16 + cl;
    if (c >= g.Cs * 4) return;  // past the last 4-channel step
    const TileIdx ti = decode_tile(g, tb * 16 + tr);
    const long long HW = (long long)g.H * g.W;
    const int32x4 rs = make_rsrc(x, (unsigned)((long long)g.N * g.C * HW * 4));
    float d[T2];
    if constexpr (VX && M == 7) {
        WideRowTile<M> ld;
        ld.init(g, ti, c);
        ld.load(rs, d);
    } else if constexpr (VX) {
        RowTile<M> ld;
        TileIdx rf, rl;
        row_edges<1>(g, tb * 16, tr, rf, rl);
        ld.init(g, ti, rf, rl, c, tr);
        ld.issue(rs, d);
        RowTile<M>::finish(d, ld.flags(), (g.W % M) != 0);
    } else {
        BufTile<M, (M <= 2)> ld;
        ld.init(g, ti, c);
        ld.load(rs, d);
    }
    if (c >= g.C) {  // channel padding (its loads read another channel's plane)
#pragma unroll
        for (int f = 0; f < T2; ++f) d[f] = 0.0f;
    }
    floatx4 *dst = U + ((long long)tb * g.Cs + (c >> 2)) * 64 + lane;
    const long long fstride = (long long)TB * g.Cs * 64;
    input_tile_transform_emit<M>(d, [&](int f4, float a, float b, float cc, float e) {
        dst[f4 * fstride] = floatx4{a, b, cc, e};
    });
}

// Buffer-unit copy from memory straight into LDS (gfx950: `buffer_load_dwordx4 ...
// lds`): lane l's `size` bytes at voffset + soffset of the resource land at byte
// size * l of the wave-uniform LDS address lds.  No registers hold the data; its
// completion is counted by vmcnt like any load.
typedef __attribute__((address_space(3))) void *lds_void_ptr;
__device__ void buffer_load_lds(int32x4 rsrc, lds_void_ptr lds, int size, unsigned voffset, unsigned soffset,
                                int offset, int aux) __asm("llvm.amdgcn.raw.buffer.load.lds");
template <class P>
__device__ __forceinline__ lds_void_ptr lds_ptr(P *p) {
    return (lds_void_ptr)(p);
}
// Waits until at most N vector-memory accesses of this wave are outstanding (other
// counters untouched).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}
// Workgroup barrier with no memory wait of its own (the caller has waited for what
// it needs); also a compiler barrier, so no LDS access moves across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// LDS ring depth of the three-stage product kernel, in channel steps of 8 KB
// (measured: 3 steps is 1-6 % faster than 4-6 on the deep layers, equal on the
// others).
constexpr int kGemmSteps = 3;

// Stage 2: per workgroup four frequencies (one float4 of operands) x 4 tile blocks
// x 4 output blocks (64 tiles x 64 output channels); each of the 4 waves
// multiplies 2 tile blocks by 2 output blocks for the 4 frequencies (16 matrix
// products per 4-channel step).  A channel step's operands -- 4 KB of W' and 4 KB
// of U, each 1 KB block already in matrix-core lane order -- are copied straight
// from memory into an LDS ring of NS steps by the buffer unit (no registers), one
// W' block and one U block per wave, NS - 1 steps ahead of the products; each
// wave then reads its 2 + 2 blocks from LDS, so every operand crosses L2 once per
// workgroup.  Workgroups are numbered so that the output groups of one tile group
// are consecutive on one XCD (workgroup b runs on XCD b % 8), so the tile group's
// U is read from HBM once and then from that XCD's L2.
template <int M>
__global__ void __launch_bounds__(256) frequency_gemm_kernel(const floatx4 *__restrict__ U,
                                                             const floatx4 *__restrict__ wt,
                                                             floatx4 *__restrict__ Mout, Geometry g) {
    constexpr int Q = freq_quads<M>();
    constexpr int NS = kGemmSteps;
    __shared__ floatx4 ring[NS][8][64];  // per step: W' blocks 0..3, then U blocks 0..3
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int TB = g.tiles_p / 16, TG = TB / 4, KG = g.Kb_alloc / 4;
    const int lb = xcd_contiguous_block(blockIdx.x, gridDim.x);
    const int kg = lb % KG, rest = lb / KG;
    const int tg = rest % TG, f4 = rest / TG;
    const int Cs = g.Cs;
    // The blocks this wave copies: output block 4 kg + wave of W', tile block
    // 4 tg + wave of U; step cs at byte offset cs * Q KB (W') or cs KB (U).
    const floatx4 *abase = wt + ((long long)(kg * 4 + wave) * Cs * Q + f4) * 64;
    const floatx4 *bbase = U + (((long long)f4 * TB + tg * 4 + wave) * Cs) * 64;
    const int32x4 ar = make_rsrc_uniform(reinterpret_cast<const float *>(abase),
                                         (unsigned)(Cs - 1) * Q * 1024u + 1024u);
    const int32x4 br = make_rsrc_uniform(reinterpret_cast<const float *>(bbase), (unsigned)Cs * 1024u);
    const unsigned vo = (unsigned)lane * 16u;
    // Steps past the last are clamped to it (the copies stay in bounds and every
    // iteration issues the same number, which the vmcnt wait below relies on).
    auto issue = [&](int st) {
        const unsigned c = (unsigned)(st < Cs ? st : Cs - 1);
        floatx4 *slot = ring[st % NS][0];
        buffer_load_lds(ar, lds_ptr(slot + wave * 64), 16, vo, c * Q * 1024u, 0, 0);
        buffer_load_lds(br, lds_ptr(slot + (4 + wave) * 64), 16, vo, c * 1024u, 0, 0);
    };
    floatx4 acc[2][2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[i][j][q] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < NS - 1; ++st) issue(st);
    const int ai = (wave & 1) * 2, bj = 4 + (wave >> 1) * 2;
    for (int cs = 0; cs < Cs; ++cs) {
        // This wave's copies of step cs are complete once at most the 2 (NS - 2)
        // copies issued after them are outstanding; the barrier then makes every
        // wave's copies of step cs visible, and tells that every wave has read
        // step cs - 1, whose slot the next copies overwrite.
        wait_vmcnt<2 * (NS - 2)>();
        lds_barrier();
        issue(cs + NS - 1);
        const floatx4(*sl)[64] = ring[cs % NS];
        floatx4 a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) a[i] = sl[ai + i][lane];
#pragma unroll
        for (int j = 0; j < 2; ++j) b[j] = sl[bj + j][lane];
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j][q] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][q], b[j][q], acc[i][j][q], 0, 0, 0);
    }
    // The copies issued past the last step (clamped repeats of it) must land
    // before the workgroup ends and its LDS can be given to another workgroup.
    wait_vmcnt<0>();
    // M: one float4 (4 frequencies) per lane and (tile block, output block, v)
    const int kb0 = kg * 4 + (wave & 1) * 2, tb0 = tg * 4 + (wave >> 1) * 2;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                Mout[((((long long)f4 * TB + tb0 + j) * g.Kb_alloc + kb0 + i) * 4 + v) * 64 + lane] =
                    floatx4{acc[i][j][0][v], acc[i][j][1][v], acc[i][j][2][v], acc[i][j][3][v]};
}

// Stage 3: the workgroup's 4 waves are the four v of one (tile block, output
// block): lane = 16 * q + tile%16 with output channel k = 16 kb + 4 q + v, so a
// wave reads one 1 KB float4 row of M per four frequencies.
template <int M>
__global__ void __launch_bounds__(256) output_transform_kernel(const floatx4 *__restrict__ Min,
                                                               float *__restrict__ y, Geometry g) {
    constexpr int T2 = (M + 2) * (M + 2), Q = freq_quads<M>();
    const int lane = threadIdx.x & 63, v = threadIdx.x >> 6;
    const int tb = blockIdx.x, kb = blockIdx.y;
    const int TB = g.tiles_p / 16;
    const int tile = tb * 16 + (lane & 15), k = kb * 16 + (lane >> 4) * 4 + v;
    const floatx4 *src = Min + (((long long)tb * g.Kb_alloc + kb) * 4 + v) * 64 + lane;
    const long long fstride = (long long)TB * g.Kb_alloc * 4 * 64;
    float mm[4 * Q];
#pragma unroll
    for (int f4 = 0; f4 < Q; ++f4) {
        const floatx4 q4 = src[f4 * fstride];
#pragma unroll
        for (int e = 0; e < 4; ++e) mm[4 * f4 + e] = q4[e];
    }
    if (tile >= g.ntiles || k >= g.K) return;
    const TileIdx ti = decode_tile(g, tile);
    float yy[M * M];
    output_tile_transform<M>(mm, yy);
    (void)T2;
    if constexpr (M % 2 == 1) {
        // odd m: rows of tiles whose m columns lie inside the image are stored as
        // 4-byte-aligned vector pieces (y is below 2^31 bytes), rows below the
        // image skipped, the rows of tiles cut by the right edge element by element
        const int h0 = ti.ty * M, w0 = ti.tx * M;
        const bool fullw = w0 + M <= g.W;
        const int32x4 yrs = make_rsrc(y, (unsigned)((long long)g.N * g.K * g.H * g.W * 4));
        const unsigned vb = (unsigned)(((((long long)ti.n * g.K + k) * g.H + h0) * g.W + w0) * 4);
        float *yp = y + ((long long)ti.n * g.K + k) * g.H * g.W;
#pragma unroll
        for (int i = 0; i < M; ++i) {
            if (h0 + i >= g.H) break;
            if (fullw) {
                store_row_buf<M, false>(yrs, vb, (unsigned)i * (unsigned)g.W * 4u, yy + i * M);
            } else {
#pragma unroll
                for (int jj = 0; jj < M; ++jj)
                    if (w0 + jj < g.W) yp[(long long)(h0 + i) * g.W + w0 + jj] = yy[i * M + jj];
            }
        }
        return;
    }
    const bool vec = (M == 4) ? (g.W % 4 == 0 && (reinterpret_cast<uintptr_t>(y) & 15) == 0)
                              : (g.W % 2 == 0 && (reinterpret_cast<uintptr_t>(y) & 7) == 0);
    store_tile<M>(y + ((long long)ti.n * g.K + k) * g.H * g.W, yy, ti.ty * M, ti.tx * M, g, vec);
}

// ---------------------------------------------------------------------------
// Launchers.

// Tile sizes of the kernel transform and the three-stage kernels: the fused
// kernel's and F(7x7,3x3) (T = 9: its 21 float4s of frequencies per tile and
// channel exceed the fused kernel's LDS stage ring).
#define WINO_DISPATCH_M(m, CALL)          \
    switch (m) {                          \
        case 2: { constexpr int MM = 2; CALL; } break; \
        case 4: { constexpr int MM = 4; CALL; } break; \
        case 5: { constexpr int MM = 5; CALL; } break; \
        case 6: { constexpr int MM = 6; CALL; } break; \
        case 7: { constexpr int MM = 7; CALL; } break; \
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
// number of work items.
//  * Capacity: a task's result matrices (R tiles x Kit output channels x T^2
//    frequencies) live in the consumer waves' registers, at most 144 per lane of
//    four waves: R * Kit * T^2 <= 36864.  F(2), F(4): Kit <= 64 (R = 32 only for
//    F(2)); F(5), F(6): R = 16, Kit <= 32.
//  * Reuse: every transformed input tile is multiplied by the Kit output
//    channels' kernels (the input-transform work per product falls as 1 / Kit)
//    and every transformed-kernel operand read from L2 by the R tiles (the
//    paper's task arithmetic intensity against the shared cache, R / 2).  So the
//    largest task that fits is taken: Kit at its maximum; R = 32 for F(2) when C
//    <= 64 (measured: with more channels the 16-channel stages of R = 16 run
//    faster), else 16 ...
//  * ... as long as the layer has at least one task per compute unit.  A layer
//    with fewer takes the blocking with the most tasks instead (smaller Kit,
//    then smaller R): on the N=1, 56x56, C=K=64 layer at F(2) 196 tasks of 16 x
//    16 run in 8.4 us against 14.8 us for 25 tasks of 32 x 64.
// Measured on every layer (steady state, one MI355X): splitting a task's output
// channels among its consumer waves costs more than the transform reuse it gives
// up whenever the larger tasks already fill the compute units.
FusedCfg fused_cfg_default(const Geometry &g, int num_cus, int want_R, int want_kit) {
    FusedCfg best{};
    int best_items = -1;
    bool best_fills = false;
    const int pref_R = (g.m == 2 && g.C <= 64) ? 32 : 16;
    for (const FusedBlocking &b : kFusedBlockings) {
        if (b.m != g.m || (want_R && b.R != want_R) || (want_kit && b.kit != want_kit)) continue;
        const FusedCfg c{b.R, b.kit, num_cus, 0};
        const int items = fused_split_info(g, c).n_items;
        const bool fills = items >= num_cus;
        bool take;
        if (best.R == 0) take = true;
        else if (fills != best_fills) take = fills;
        else if (fills) {
            // both fill the units: the largest task, R = pref_R first
            const bool bp = best.R == pref_R, cp = b.R == pref_R;
            take = b.kit > best.kit || (b.kit == best.kit && cp && !bp);
        } else {
            // neither fills the units: the most tasks
            take = items > best_items;
        }
        if (take) {
            best = c;
            best_items = items;
            best_fills = fills;
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
    dim3 block(256), grid((unsigned)((long long)(g.tiles_p / 16) * ((g.Cs * 4 + 15) / 16)));
    // row-vector input loads need every row start aligned to the vector width
    // (m = 5, 7: 4-byte-aligned vector loads)
    const unsigned vw = (g.m == 4) ? 16u : (g.m == 5 || g.m == 7) ? 4u : 8u;
    const bool vx = (reinterpret_cast<uintptr_t>(x) % vw == 0) && ((unsigned)g.W * 4u) % vw == 0;
    floatx4 *u4 = reinterpret_cast<floatx4 *>(U);
    if (vx) {
        WINO_DISPATCH_M(g.m, hipLaunchKernelGGL((input_transform_kernel<MM, true>), grid, block, 0, s, x, u4, g));
    } else {
        WINO_DISPATCH_M(g.m, hipLaunchKernelGGL((input_transform_kernel<MM, false>), grid, block, 0, s, x, u4, g));
    }
    return hipGetLastError();
}

hipError_t launch_frequency_gemm(const Geometry &g, const float *U, const float *wt, float *Mout,
                                 hipStream_t s) {
    const long long nblk = (long long)(g.tiles_p / 64) * (g.Kb_alloc / 4) * ((g.T2 + 3) / 4);
    dim3 block(256), grid((unsigned)nblk);
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(frequency_gemm_kernel<MM>, grid, block, 0, s,
                                            reinterpret_cast<const floatx4 *>(U),
                                            reinterpret_cast<const floatx4 *>(wt),
                                            reinterpret_cast<floatx4 *>(Mout), g));
    return hipGetLastError();
}

hipError_t launch_output_transform(const Geometry &g, const float *Min, float *y, hipStream_t s) {
    dim3 block(256), grid((unsigned)(g.tiles_p / 16), (unsigned)g.Kb);
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(output_transform_kernel<MM>, grid, block, 0, s,
                                            reinterpret_cast<const floatx4 *>(Min), y, g));
    return hipGetLastError();
}

}  // namespace wino
