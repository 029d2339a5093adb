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
#include <type_traits>

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

// Frequencies are grouped in float4s (four consecutive f) for the matrix-core
// operands; T^2 = 49 (F(5)) ends with a partial group padded with zeros.
template <int M>
constexpr int freq_quads() { return ((M + 2) * (M + 2) + 3) / 4; }

// ---------------------------------------------------------------------------
// Kernel transform (Sec. 3, step 2: right-hand matrices transformed ahead of
// time).  Thread (kb, cs, lane) transforms kernel (k, c) with k = 16 kb + lane%16,
// c = 4 cs + lane/16 and stores the T^2 values in matrix-core operand order:
// wt[((kb * Cs + cs) * Q + f/4) * 64 + lane][f % 4], Q = ceil(T^2/4).  Channels
// >= C, output channels >= K and frequencies >= T^2 are stored as zeros.
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
// Buffer-resource loads of input tiles.  A raw buffer load whose byte offset is
// at or past the resource's size returns 0 without touching memory, which gives
// the implicit zero padding of Sec. 2.1 with unconditional loads: offsets of rows
// or columns outside the image are pushed to >= 2^31 (x is below 2^31 bytes) with
// a saturating add.
typedef int int32x4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

// Raw buffer loads, called through the LLVM intrinsics with an explicit 4-dword
// resource (base address, size in bytes, 32-bit data format).
__device__ float buffer_load_f32(int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.load.f32");
__device__ floatx2 buffer_load_f32x2(int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.load.v2f32");
__device__ floatx4 buffer_load_f32x4(int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.load.v4f32");
__device__ void buffer_store_f32x4(floatx4 v, int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.store.v4f32");
__device__ void buffer_store_f32x2(floatx2 v, int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.store.v2f32");
__device__ void buffer_store_f32(float v, int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.store.f32");
// Cache-policy bit of a buffer access that makes it coherent across the device
// (the coherence that device-scope atomic loads and stores use).
constexpr int kDeviceCoherent = 1 << 4;
// Cache-policy bit of a streaming (non-temporal) access.  An output larger than
// the Infinity Cache, written once, is stored this way so that it does not push
// input tiles that another output-channel group still needs, or the transformed
// kernels, out of L2; a smaller output is better left in the caches.
constexpr int kStream = 1 << 1;
constexpr long long kStreamOutputBytes = 128ll << 20;

__device__ __forceinline__ int32x4 make_rsrc(const float *base, unsigned bytes) {
    const unsigned long long p = reinterpret_cast<unsigned long long>(base);
    int32x4 r;
    r[0] = (int)(unsigned)(p & 0xffffffffull);
    r[1] = (int)(unsigned)((p >> 32) & 0xffffull);  // stride 0: raw buffer
    r[2] = (int)bytes;                                 // range-checked size
    r[3] = 0x00020000;                                 // 32-bit data format
    return r;
}

// The same resource held in scalar registers, for a base address the compiler
// cannot prove uniform (a per-lane resource would turn every access into a loop
// over distinct lane values).
__device__ __forceinline__ int32x4 make_rsrc_uniform(const float *base, unsigned bytes) {
    int32x4 r = make_rsrc(base, bytes);
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = __builtin_amdgcn_readfirstlane(r[i]);
    return r;
}

constexpr unsigned kOutside = 0x80000000u;

// Per-lane byte offsets of the T x T input tile (rows ty*M-1+a, columns tx*M-1+b)
// of one tile and channel lane_c, relative to the plane of channel 0 of the
// current channel step.  PRECOMP keeps all T^2 offsets in registers; otherwise
// each element costs one saturating add.
template <int M, bool PRECOMP>
struct BufTile {
    static constexpr int T = M + 2, T2 = T * T;
    unsigned off[PRECOMP ? T2 : 1];
    unsigned roff[PRECOMP ? 1 : T];
    unsigned coff[PRECOMP ? 1 : T];

    __device__ __forceinline__ void init(const Geometry &g, const TileIdx &t, int lane_c) {
        const unsigned base = (unsigned)(((long long)t.n * g.C + lane_c) * g.H * g.W) * 4u;
        unsigned ro[T], co[T];
#pragma unroll
        for (int a = 0; a < T; ++a) {
            const int h = t.ty * M - 1 + a;
            ro[a] = (t.ok && h >= 0 && h < g.H) ? base + (unsigned)(h * g.W) * 4u : kOutside;
        }
#pragma unroll
        for (int b = 0; b < T; ++b) {
            const int w = t.tx * M - 1 + b;
            co[b] = (w >= 0 && w < g.W) ? (unsigned)w * 4u : kOutside;
        }
        if constexpr (PRECOMP) {
#pragma unroll
            for (int a = 0; a < T; ++a)
#pragma unroll
                for (int b = 0; b < T; ++b) off[a * T + b] = __builtin_elementwise_add_sat(ro[a], co[b]);
        } else {
#pragma unroll
            for (int a = 0; a < T; ++a) roff[a] = ro[a];
#pragma unroll
            for (int b = 0; b < T; ++b) coff[b] = co[b];
        }
    }

    __device__ __forceinline__ unsigned offset(int a, int b) const {
        if constexpr (PRECOMP) return off[a * T + b];
        else return __builtin_elementwise_add_sat(roff[a], coff[b]);
    }

    __device__ __forceinline__ void load(int32x4 r, float *d) const {
#pragma unroll
        for (int a = 0; a < T; ++a)
#pragma unroll
            for (int b = 0; b < T; ++b)
                d[a * T + b] = buffer_load_f32(r, offset(a, b), 0, 0);
    }
};

// Row-vector loads of input tiles.  Lanes l and l+1 of a 16-lane DPP row hold
// horizontally adjacent tiles of the same channel (tiles are numbered along
// rows), and the T = m + 2 columns of a tile's row are its own m columns plus one
// halo column on each side, which are the neighbours' own edge columns.  So each
// lane loads only its own m columns of a row with vector loads and takes the
// halo columns from lanes l-1 and l+1 with DPP row shifts.  A tile in the first
// (last) column of tiles has zero padding on its left (right).
//
// The two halo columns that no lane of the DPP row owns (left of its first tile,
// right of its last) take 2T elements, which the row fetches with ONE load: lane
// 15-2a loads element a of the left column and lane 14-2a element a of the right
// one (a < T <= 8).  A rotation of the row by 2a+1 lanes then brings element a of
// the left column to lane 0 and of the right column to lane 15, where the row
// shifts (which leave the edge lane's own value in place) pass it on.
__device__ __forceinline__ float dpp_from_left(float v) {   // lane l gets lane l-1 (0 at row start)
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                 0x111, 0xf, 0xf, true));
}
__device__ __forceinline__ float dpp_from_right(float v) {  // lane l gets lane l+1 (0 at row end)
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                 0x101, 0xf, 0xf, true));
}
// lane l gets lane l-1; lane 0 of each row keeps `edge`
__device__ __forceinline__ float dpp_from_left_or(float edge, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, edge),
                                                                 __builtin_bit_cast(int, v), 0x111,
                                                                 0xf, 0xf, false));
}
// lane l gets lane l+1; lane 15 of each row keeps `edge`
__device__ __forceinline__ float dpp_from_right_or(float edge, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, edge),
                                                                 __builtin_bit_cast(int, v), 0x101,
                                                                 0xf, 0xf, false));
}
// lane l gets lane (l - S) mod 16 of its row
template <int S>
__device__ __forceinline__ float dpp_rotate(float v) {
    static_assert(S >= 1 && S <= 15, "row rotation by 1..15 lanes");
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                 0x120 + S, 0xf, 0xf, true));
}

// First and last tile of the 16-lane DPP row that holds tile t0 + tr of a task of
// 16*TB tiles starting at t0.  Each candidate is decoded from a wave-uniform
// index (on the scalar unit) and the lane picks its row's.
template <int TB>
__device__ __forceinline__ void row_edges(const Geometry &g, int t0, int tr, TileIdx &rf, TileIdx &rl) {
    rf = decode_tile(g, t0);
    rl = decode_tile(g, t0 + 15);
#pragma unroll
    for (int k = 1; k < TB; ++k) {
        const TileIdx f = decode_tile(g, t0 + 16 * k), l = decode_tile(g, t0 + 16 * k + 15);
        if ((tr >> 4) == k) {
            rf = f;
            rl = l;
        }
    }
}

template <int M>
struct RowTile {
    static constexpr int T = M + 2;
    static_assert(T <= 8, "2T halo elements per 16-lane row");
    unsigned roff[T];   // byte offset of column 0 of input row a (>= 2^31 if outside)
    unsigned own;       // byte offset of the tile's first own column, tx*M*4
    unsigned hoff;      // byte offset of the row's halo element this lane fetches
    bool first, last;   // tile in the first / last column of tiles: halo is padding
    unsigned ownok;     // bit j: own column j lies inside the image

    // Halo element of lane `lane16`: side (left for odd lanes) and row a.
    static __device__ __forceinline__ bool halo_left(int lane16) { return (lane16 & 1) != 0; }
    static __device__ __forceinline__ int halo_row(int lane16) {
        return halo_left(lane16) ? (15 - lane16) >> 1 : (14 - lane16) >> 1;
    }

    // t: this lane's tile; rfirst, rlast: the first and last tile of its DPP row.
    __device__ __forceinline__ void init(const Geometry &g, const TileIdx &t, const TileIdx &rfirst,
                                         const TileIdx &rlast, int lane_c, int lane16) {
        const unsigned base = (unsigned)(((long long)t.n * g.C + lane_c) * g.H * g.W) * 4u;
#pragma unroll
        for (int a = 0; a < T; ++a) {
            const int h = t.ty * M - 1 + a;
            roff[a] = (t.ok && h >= 0 && h < g.H) ? base + (unsigned)(h * g.W) * 4u : kOutside;
        }
        own = (unsigned)(t.tx * M) * 4u;
        first = t.tx == 0;
        last = t.tx == g.TW - 1;
        ownok = 0u;
#pragma unroll
        for (int j = 0; j < M; ++j)
            if (t.tx * M + j < g.W) ownok |= 1u << j;
        // column left of the first tile / right of the last; outside the image
        // (padding) it reads as 0
        const bool left = halo_left(lane16);
        const TileIdx edge = left ? rfirst : rlast;
        const int a = halo_row(lane16);
        const int h = edge.ty * M - 1 + a;
        const int w = left ? edge.tx * M - 1 : edge.tx * M + M;
        hoff = kOutside;
        if (a < T && edge.ok && h >= 0 && h < g.H && w >= 0 && w < g.W)
            hoff = (unsigned)((((long long)edge.n * g.C + lane_c) * g.H + h) * g.W + w) * 4u;
    }

    // Issues the loads of one tile without waiting for them: row a of d receives
    // [-, own columns, -] and d[0] the lane's halo element; the halo exchange and
    // the masks are applied by finish(), once the data has arrived, so that loads
    // can run several stages ahead.
    __device__ __forceinline__ void issue(int32x4 r, float *d) const {
#pragma unroll
        for (int a = 0; a < T; ++a) {
            // Own columns with one vector load for m = 2, 4 and two for m = 6 (4 + 2,
            // rows 8-byte aligned) and m = 5 (4 + 1).  roff is below 2^31 or exactly 2^31 and
            // own + 4*M is below 2^31, so the offsets never wrap.
            const unsigned base = roff[a] + own;
            if constexpr (M == 4) {
                const floatx4 q = buffer_load_f32x4(r, base, 0, 0);
#pragma unroll
                for (int j = 0; j < 4; ++j) d[a * T + 1 + j] = q[j];
            } else if constexpr (M == 6) {
                const floatx4 q = buffer_load_f32x4(r, base, 0, 0);
                const floatx2 q2 = buffer_load_f32x2(r, base + 16u, 0, 0);
#pragma unroll
                for (int j = 0; j < 4; ++j) d[a * T + 1 + j] = q[j];
                d[a * T + 5] = q2[0];
                d[a * T + 6] = q2[1];
            } else if constexpr (M == 5) {  // rows 4-byte aligned
                const floatx4 q = buffer_load_f32x4(r, base, 0, 0);
#pragma unroll
                for (int j = 0; j < 4; ++j) d[a * T + 1 + j] = q[j];
                d[a * T + 5] = buffer_load_f32(r, base + 16u, 0, 0);
            } else {
                static_assert(M == 2, "m = 2, 4, 5 or 6");
                const floatx2 q = buffer_load_f32x2(r, base, 0, 0);
                d[a * T + 1] = q[0];
                d[a * T + 2] = q[1];
            }
        }
        d[0] = buffer_load_f32(r, hoff, 0, 0);
    }

    // The per-tile facts finish() needs, packed so they can travel with the data
    // of a stage while the loader moves on to the next item.
    __device__ __forceinline__ unsigned flags() const {
        return (first ? 1u : 0u) | (last ? 2u : 0u) | (ownok << 8);
    }

    template <int A = 0>
    static __device__ __forceinline__ void finish_rows(float *d, float hf, unsigned fl) {
        if constexpr (A < T) {
            // element A of the row's outer halo columns, now in lanes 0 and 15
            const float hv = dpp_rotate<2 * A + 1>(hf);
            const float ln = dpp_from_left_or(hv, d[A * T + M]);  // left neighbour's last own column
            const float rn = dpp_from_right_or(hv, d[A * T + 1]);  // right neighbour's first own column
            d[A * T] = (fl & 1u) ? 0.0f : ln;
            d[A * T + T - 1] = (fl & 2u) ? 0.0f : rn;
            finish_rows<A + 1>(d, hf, fl);
        }
    }

    static __device__ __forceinline__ void finish(float *d, unsigned fl, bool maskcols) {
        finish_rows(d, d[0], fl);
        if (maskcols) {  // own columns past W (W % m != 0)
            asm volatile("");  // keeps this a branch instead of selects run by every tile
#pragma unroll
            for (int a = 0; a < T; ++a)
#pragma unroll
                for (int j = 0; j < M; ++j)
                    if (!((fl >> (8 + j)) & 1u)) d[a * T + 1 + j] = 0.0f;
        }
    }
};

// ---------------------------------------------------------------------------
// Fused kernel (Sec. 4: a task of R tiles does input transform -> T^2 products
// against the hot kernel matrices -> output transform).  Here a task is a
// workgroup of `waves` waves; each wave owns 16 consecutive tiles and the same
// NKB blocks of 16 output channels.  Per 4-channel step a lane loads one input
// tile, transforms it in registers (B^T d B) and feeds each frequency to the
// matrix core against the matching transformed-kernel slice, which every wave
// of the workgroup reads from the same cached lines.  The next step's input tile
// is loaded while the current one is transformed and multiplied.  The
// accumulators (the paper's result matrices) never leave registers; after the
// last step each lane inverse-transforms its tile for its four output channels
// and writes y.
template <int M, int NKB>
__device__ __forceinline__ void fused_step(floatx4 (&acc)[NKB][(M + 2) * (M + 2)], const float *d,
                                           const floatx4 *__restrict__ wt, const Geometry &g,
                                           int kb0, int cs, int lane, bool zero_u) {
    constexpr int T = M + 2, T2 = T * T;
    float u[T2];
    input_tile_transform<M>(d, u);
    if (zero_u) {  // channel past C in the last step (only when C % 4 != 0)
#pragma unroll
        for (int f = 0; f < T2; ++f) u[f] = 0.0f;
    }
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        const floatx4 *wp = wt + ((long long)(kb0 + kb) * g.Cs + cs) * (T2 / 4) * 64 + lane;
#pragma unroll
        for (int f4 = 0; f4 < T2 / 4; ++f4) {
            const floatx4 a = wp[f4 * 64];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                acc[kb][4 * f4 + q] =
                    __builtin_amdgcn_mfma_f32_16x16x4f32(a[q], u[4 * f4 + q], acc[kb][4 * f4 + q], 0, 0, 0);
        }
    }
}

template <int M, int NKB>
__global__ void __launch_bounds__(256) fused_kernel(const float *__restrict__ x,
                                                    const floatx4 *__restrict__ wt,
                                                    float *__restrict__ y, Geometry g) {
    constexpr int T = M + 2, T2 = T * T;
    constexpr bool PRECOMP = (M <= 2);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int waves = blockDim.x >> 6;
    const int tile = (blockIdx.x * waves + wave) * 16 + (lane & 15);
    const int cq = lane >> 4;
    const int kb0 = blockIdx.y * NKB;
    const TileIdx ti = decode_tile(g, tile);
    BufTile<M, PRECOMP> ld;
    ld.init(g, ti, cq);
    const long long HW = (long long)g.H * g.W;
    const unsigned xbytes = (unsigned)((long long)g.N * g.C * HW * 4);
    const unsigned step_bytes = (unsigned)(4 * HW * 4);
    const bool ctail = (g.C & 3) != 0;

    floatx4 acc[NKB][T2];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int f = 0; f < T2; ++f) acc[kb][f] = floatx4{0.f, 0.f, 0.f, 0.f};

    float dA[T2], dB[T2];
    ld.load(make_rsrc(x, xbytes), dA);
    int cs = 0;
    for (; cs + 1 < g.Cs; cs += 2) {
        ld.load(make_rsrc(x + (cs + 1) * 4 * HW, xbytes - (cs + 1) * step_bytes), dB);
        fused_step<M, NKB>(acc, dA, wt, g, kb0, cs, lane, false);
        if (cs + 2 < g.Cs) ld.load(make_rsrc(x + (cs + 2) * 4 * HW, xbytes - (cs + 2) * step_bytes), dA);
        fused_step<M, NKB>(acc, dB, wt, g, kb0, cs + 1, lane,
                           ctail && cs + 1 == g.Cs - 1 && (cs + 1) * 4 + cq >= g.C);
    }
    if (cs < g.Cs)
        fused_step<M, NKB>(acc, dA, wt, g, kb0, cs, lane, ctail && cs * 4 + cq >= g.C);

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
// Fused kernel, shared-transform schedule.  A workgroup (4 waves) is one task of
// R = 16*TB tiles and 64 output channels (Sec. 4).  The channel loop runs in
// stages of CC = 256/R channels; in each stage every thread loads and transforms
// one (tile, channel) input tile and stores its T^2 values in LDS, so the
// left-hand matrices of the stage (the paper's R x C slices, one per frequency)
// are built once and read by all four waves.  Wave w multiplies them by the
// transformed kernels of output-channel block w, which stream from L2 (the
// paper's hot right-hand matrices).  LDS is double-buffered: while a stage's
// products run, the next stage's input tiles are loaded and then transformed
// into the other buffer, with one barrier per stage.  The accumulators (result
// matrices) stay in registers until the output transform.
//
// LDS layout of one buffer, in float4 units: [T^2/4][CC][R] with the four
// frequencies 4*f4 .. 4*f4+3 of (channel, tile) in one float4, so that a wave's
// matrix-core B operand for four frequencies is one contiguous 1 KB read.
template <int M, int TB>
__global__ void __launch_bounds__(256) fused_shared_kernel(const float *__restrict__ x,
                                                           const floatx4 *__restrict__ wt,
                                                           float *__restrict__ y, Geometry g) {
    constexpr int T = M + 2, T2 = T * T, F4 = T2 / 4;
    constexpr int R = 16 * TB;       // tiles per workgroup
    constexpr int CC = 256 / R;      // channels per stage
    constexpr int SS = CC / 4;       // matrix-core channel steps per stage
    constexpr int BUF = F4 * CC * R; // float4s per LDS buffer
    __shared__ floatx4 lds[2 * BUF];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const long long HW = (long long)g.H * g.W;
    const unsigned xbytes = (unsigned)((long long)g.N * g.C * HW * 4);
    const int tile0 = blockIdx.x * R;

    // transform role: thread -> (tile tile0 + tr, channel cl of the stage)
    const int tr = tid % R;
    const int cl = tid / R;
    BufTile<M, (M <= 2)> ld;
    ld.init(g, decode_tile(g, tile0 + tr), cl);
    const int stages = (g.C + CC - 1) / CC;
    const bool ctail = (g.C % CC) != 0;

    // matrix-core role: wave -> output-channel block kb
    const int kb = blockIdx.y * 4 + wave;
    const floatx4 *wk = wt + (long long)kb * g.Cs * F4 * 64 + lane;

    floatx4 acc[TB][T2];
#pragma unroll
    for (int t = 0; t < TB; ++t)
#pragma unroll
        for (int f = 0; f < T2; ++f) acc[t][f] = floatx4{0.f, 0.f, 0.f, 0.f};

    float d[T2];
    auto transform_store = [&](int stage, floatx4 *buf) {
        float u[T2];
        input_tile_transform<M>(d, u);
        if (ctail && stage == stages - 1 && stage * CC + cl >= g.C) {
#pragma unroll
            for (int f = 0; f < T2; ++f) u[f] = 0.0f;
        }
#pragma unroll
        for (int f4 = 0; f4 < F4; ++f4)
            buf[(f4 * CC + cl) * R + tr] = floatx4{u[4 * f4], u[4 * f4 + 1], u[4 * f4 + 2], u[4 * f4 + 3]};
    };

    ld.load(make_rsrc(x, xbytes), d);
    transform_store(0, lds);
    __syncthreads();

    for (int j = 0; j < stages; ++j) {
        const bool next = j + 1 < stages;
        if (next) {
            const long long cbase = (long long)(j + 1) * CC * HW;
            ld.load(make_rsrc(x + cbase, xbytes - (unsigned)(cbase * 4)), d);
        }
        const floatx4 *cur = lds + (j & 1) * BUF;
#pragma unroll
        for (int s = 0; s < SS; ++s) {
            const int cs = j * SS + s;
            if (cs < g.Cs) {
                const floatx4 *wp = wk + (long long)cs * F4 * 64;
                const floatx4 *bp = cur + (4 * s + (lane >> 4)) * R + (lane & 15);
#pragma unroll
                for (int f4 = 0; f4 < F4; ++f4) {
                    const floatx4 a = wp[f4 * 64];
#pragma unroll
                    for (int t = 0; t < TB; ++t) {
                        const floatx4 b = bp[f4 * CC * R + t * 16];
#pragma unroll
                        for (int q = 0; q < 4; ++q)
                            acc[t][4 * f4 + q] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                a[q], b[q], acc[t][4 * f4 + q], 0, 0, 0);
                    }
                }
            }
        }
        if (next) transform_store(j + 1, lds + ((j + 1) & 1) * BUF);
        __syncthreads();
    }

    // Output transform Y = A^T Mm A per (output channel, tile), clipped to H x W.
#pragma unroll
    for (int t = 0; t < TB; ++t) {
        const TileIdx ti = decode_tile(g, tile0 + t * 16 + (lane & 15));
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int k = kb * 16 + (lane >> 4) * 4 + v;
            float mm[T2];
#pragma unroll
            for (int f = 0; f < T2; ++f) mm[f] = acc[t][f][v];
            float yy[M * M];
            output_tile_transform<M>(mm, yy);
            if (ti.ok && k < g.K) {
                float *yp = y + ((long long)ti.n * g.K + k) * HW;
#pragma unroll
                for (int i = 0; i < M; ++i) {
                    const int h = ti.ty * M + i;
                    if (h < g.H) {
#pragma unroll
                        for (int jj = 0; jj < M; ++jj) {
                            const int w = ti.tx * M + jj;
                            if (w < g.W) __builtin_nontemporal_store(yy[i * M + jj], yp + (long long)h * g.W + w);
                        }
                    }
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Store one m x m output tile that lies wholly inside the image, its first element
// at yp (16-byte aligned for m = 4, 8-byte for m = 2, 6), rows ld floats apart.
template <int M>
__device__ __forceinline__ void store_rows(float *__restrict__ yp, const float *yy, int ld) {
#pragma unroll
    for (int i = 0; i < M; ++i) {
        float *row = yp + (long long)i * ld;
        if constexpr (M == 4) {
            *reinterpret_cast<floatx4 *>(row) = floatx4{yy[i * M], yy[i * M + 1], yy[i * M + 2], yy[i * M + 3]};
        } else {
#pragma unroll
            for (int jj = 0; jj < M; jj += 2)
                *reinterpret_cast<floatx2 *>(row + jj) = floatx2{yy[i * M + jj], yy[i * M + jj + 1]};
        }
    }
}

// The same through a buffer resource over y: the tile's first element at byte
// offset voff (per lane) + soff (uniform), rows rowb bytes apart (uniform), so the
// per-row and per-channel steps are scalar adds.
template <int M, bool STREAM>
__device__ __forceinline__ void store_rows_buf(int32x4 yrs, unsigned voff, unsigned soff, unsigned rowb,
                                               const float *yy) {
    constexpr int kAux = STREAM ? kStream : 0;
#pragma unroll
    for (int i = 0; i < M; ++i) {
        const unsigned so = soff + (unsigned)i * rowb;
        if constexpr (M == 4) {
            buffer_store_f32x4(floatx4{yy[i * M], yy[i * M + 1], yy[i * M + 2], yy[i * M + 3]}, yrs, voff, so, kAux);
        } else if constexpr (M == 5) {  // 4-byte aligned vector store + one float
            buffer_store_f32x4(floatx4{yy[i * M], yy[i * M + 1], yy[i * M + 2], yy[i * M + 3]}, yrs, voff, so, kAux);
            buffer_store_f32(yy[i * M + 4], yrs, voff + 16u, so, kAux);
        } else {
#pragma unroll
            for (int jj = 0; jj < M; jj += 2)
                buffer_store_f32x2(floatx2{yy[i * M + jj], yy[i * M + jj + 1]}, yrs, voff + 4u * jj, so, kAux);
        }
    }
}

// Store one m x m output tile of plane yp (clipped to H x W).  vec: rows may be
// written with m-float vector stores (16-byte aligned for m = 4, 8-byte for m = 2, 6;
// m = 5 always stores element by element here).
template <int M>
__device__ __forceinline__ void store_tile(float *__restrict__ yp, const float *yy, int h0, int w0,
                                           const Geometry &g, bool vec) {
#pragma unroll
    for (int i = 0; i < M; ++i) {
        const int h = h0 + i;
        if (h >= g.H) break;
        float *row = yp + (long long)h * g.W + w0;
        if (M != 5 && vec && w0 + M <= g.W) {
            if constexpr (M == 4) {
                *reinterpret_cast<floatx4 *>(row) =
                    floatx4{yy[i * M], yy[i * M + 1], yy[i * M + 2], yy[i * M + 3]};
            } else if constexpr (M != 5) {
                #pragma unroll
                for (int jj = 0; jj < M; jj += 2)
                    *reinterpret_cast<floatx2 *>(row + jj) = floatx2{yy[i * M + jj], yy[i * M + jj + 1]};
            }
        } else {
#pragma unroll
            for (int jj = 0; jj < M; ++jj)
                if (w0 + jj < g.W) row[jj] = yy[i * M + jj];
        }
    }
}

// ---------------------------------------------------------------------------
// Fused kernel, warp-specialised schedule.  A workgroup of 8 waves is one task of
// R = 16*TB tiles and 64/FS output channels (Sec. 4).
//
// Waves 4..7 are producers: per stage of CC = 256/R channels each lane loads one
// (tile, channel) input tile, transforms it (B^T d B) and writes its T^2 values to
// LDS; the loads of the next stage are issued before the transform, so their
// latency hides behind it and behind the barrier.
//
// Waves 0..3 are consumers on the matrix cores.  With FS = 1, wave w owns output
// block w and all T^2 frequencies.  With FS = 2 (F(6), whose 64 frequencies would
// need 256 accumulators), waves 2b and 2b+1 share output block b and each owns
// half of the transform-domain rows; by linearity of the output transform each
// inverse-transforms its own rows and the two partial tiles are added through a
// small LDS slot of the pair.  The kernel operands of the next 4-channel step
// are loaded while the current step runs.
//
// Two waves per SIMD (a producer and a consumer) let the producers' vector work
// overlap the matrix cores.  LDS holds two stage buffers with one barrier per
// stage; the layout of a buffer is that of fused_shared_kernel.

// Transform-domain rows owned by frequency group G of FS (bit i = row i).  Each
// group is closed under the (+p, -p) row pairs and covers whole float4s of
// frequencies: F(6) (T = 8, a row is two float4s): rows {0,1,2,7} and {3,4,5,6};
// F(5) (T = 7): rows {0..3} = frequencies 0..27 = float4s 0..6 and rows {4,5,6} =
// float4s 7..12 (the last padded).
template <int M, int FS, int G>
constexpr unsigned group_rows() {
    if constexpr (FS == 1) return (1u << (M + 2)) - 1u;
    else if constexpr (M == 5) return G == 0 ? 0x0fu : 0x70u;
    else return G == 0 ? 0x87u : 0x78u;
}

// Global float4 frequency indices of the group's float4s (those holding a
// frequency of the group's rows), as a compile-time table.
template <int M, int FS, int G>
struct GroupF4 {
    static constexpr int T = M + 2;
    static constexpr int Q = freq_quads<M>();
    static constexpr int count() {
        int n = 0;
        for (int q = 0; q < Q; ++q)
            if ((group_rows<M, FS, G>() >> ((4 * q) / T)) & 1u) ++n;
        return n;
    }
    static constexpr int N = count();
    int f4[N];
    // accumulator index (4 * position of the float4 + offset) of frequency f
    constexpr int index(int f) const {
        for (int i = 0; i < N; ++i)
            if (f4[i] == f / 4) return 4 * i + f % 4;
        return -1;
    }
    constexpr GroupF4() : f4{} {
        int n = 0;
        for (int q = 0; q < Q; ++q)
            if ((group_rows<M, FS, G>() >> ((4 * q) / T)) & 1u) f4[n++] = q;
    }
    // every float4 lies within the group's rows (the group splits on float4 bounds)
    static constexpr bool whole() {
        for (int q = 0; q < Q; ++q) {
            const unsigned r0 = (group_rows<M, FS, G>() >> ((4 * q) / T)) & 1u;
            for (int e = 1; e < 4; ++e) {
                const int f = 4 * q + e;
                if (f < T * T && ((group_rows<M, FS, G>() >> (f / T)) & 1u) != r0) return false;
            }
        }
        return true;
    }
};

// Frequency-split (FS = 2) epilogue: the partial output tiles of the two waves of
// a block pair are added one output channel of the four (v) at a time through an
// LDS slot per pair.  The pair synchronises through two counters next to the
// slot (partials written, partials read) rather than workgroup barriers, so the
// epilogue never waits for the producer waves.  A wait gives up after kSpinLimit
// polls, so a broken handshake ends the kernel with wrong output instead of
// hanging it.
constexpr unsigned kSpinLimit = 1u << 22;

__device__ __forceinline__ void wait_counter(const unsigned *c, unsigned target) {
    for (unsigned n = 0; n < kSpinLimit; ++n) {
        if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) == target) return;
        __builtin_amdgcn_s_sleep(1);
    }
}

// Stage ring of the warp-specialised kernel: per LDS buffer (slot) a count of
// producer waves that have filled it and of consumer waves that have drained
// it, both only growing.  The g-th filling of a slot is complete when its fill
// count reaches 4(g+1); the slot may be filled again once its drain count
// reaches 4(g+1).  Waits give up after kSpinLimit polls like wait_counter.
__device__ __forceinline__ void wait_at_least(const unsigned *c, unsigned target) {
    for (unsigned n = 0; n < kSpinLimit; ++n) {
        if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= target) return;
        __builtin_amdgcn_s_sleep(1);
    }
}

// LDS stage buffers of the warp-specialised kernel: three where they fit (the
// producers may then run up to two stages ahead), two for F(6).
template <int M>
constexpr int ws_slots() { return M <= 4 ? 3 : 2; }

// One wave's +1 on counter c, ordered after all of the wave's LDS accesses.
__device__ __forceinline__ void signal_wave(unsigned *c) {
    if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Items of a persistent workgroup: first + i * stride, i < count.  Items are
// numbered with the output-channel group fastest; each XCD takes one contiguous
// range of them and its workgroups take items from it round-robin (workgroup b
// runs on XCD b % 8 as its (b / 8)-th workgroup), so the workgroups of an XCD
// work on neighbouring items at any time.
struct ItemRange {
    int first, stride, count;
};

__device__ __forceinline__ ItemRange item_range(int n_items) {
    constexpr int kXcds = 8;
    const int nwg = gridDim.x;
    const int xcd = blockIdx.x % kXcds, j = blockIdx.x / kXcds;
    const int per = nwg / kXcds, extra = nwg % kXcds;
    const int wg_on_xcd = per + (xcd < extra ? 1 : 0);
    const int wg_before = xcd * per + (xcd < extra ? xcd : extra);
    const int xcd_first = (int)((long long)n_items * wg_before / nwg);
    const int xcd_end = (int)((long long)n_items * (wg_before + wg_on_xcd) / nwg);
    ItemRange r;
    r.first = xcd_first + j;
    r.stride = wg_on_xcd;
    r.count = r.first < xcd_end ? (xcd_end - r.first + r.stride - 1) / r.stride : 0;
    return r;
}

// Work of one persistent workgroup of the warp-specialised kernel, as one
// sequence of (item, channel stage) pairs shared by its producers and consumers:
// first its whole items (taken as by item_range from the first n_whole items),
// then its pieces of split items.  Each split item is cut into P pieces of L
// consecutive channel stages (the last one shorter when L does not divide the
// stages); the pieces ("split units", unit u is piece u % P of split item u / P)
// are distributed as by item_range.  Splitting only the items of a last, partly
// filled round spreads that round over compute units that would otherwise idle;
// splitting every item computes the layer as P convolutions over subsets of the
// input channels whose outputs are added (Sec. 7).  A workgroup's sequence falls
// into segments, one per whole item or piece; a piece yields a partial output,
// and the partial outputs of an item are added by whichever of its P
// contributors finishes last.
// Item numbering of the warp-specialised kernel: with KM false the output-channel
// group varies fastest (items = tile groups x groups, the groups of one tile group
// adjacent: its input tiles are shared in L2); with KM true the tile group varies
// fastest (the tile groups of one output-channel group adjacent: its transformed
// kernels are shared in L2).  n_inner is the count of the fastest index.
template <bool KM>
__device__ __forceinline__ int item_tgroup(int it, int n_inner) { return KM ? it % n_inner : it / n_inner; }
template <bool KM>
__device__ __forceinline__ int item_kgroup(int it, int n_inner) { return KM ? it / n_inner : it % n_inner; }

struct WsSplit {
    int n_whole;          // items distributed whole (item_range over the first n_whole)
    int tail_first;       // first split item
    int n_units;          // split items x P
    int P;                // pieces per split item (contributors)
    int piece;            // stages per piece (L)
    float *part;          // partial outputs, [split item][contributor][part_floats]
    unsigned *cnt;        // contributors arrived, per split item (zero between calls)
    int part_floats;      // floats of one partial output
};

struct WsSeq {
    int first, stride, nfull;     // whole items first + i * stride, i < nfull
    int pfirst, pstride, npiece;  // split units pfirst + i * pstride, i < npiece
    int S;                        // stages per item
    int n_items;
    int tail_first, P, L;         // as in WsSplit
    int nseg;                     // segments: nfull whole items, then npiece pieces

    __device__ __forceinline__ void init(const WsSplit &sp, int n_items_, int stages, bool split) {
        S = stages;
        n_items = n_items_;
        const ItemRange ir = item_range(sp.n_whole);
        first = ir.first;
        stride = ir.stride;
        nfull = ir.count;
        pfirst = 0;
        pstride = 1;
        npiece = 0;
        tail_first = sp.tail_first;
        P = sp.P > 0 ? sp.P : 1;
        L = sp.piece > 0 ? sp.piece : stages;
        if (split) {
            const ItemRange pr = item_range(sp.n_units);
            pfirst = pr.first;
            pstride = pr.stride;
            npiece = pr.count;
        }
        nseg = nfull + npiece;
    }
    __device__ __forceinline__ int length() const {
        // stages of the pieces: L each, except those that are the last of their item
        int n = nfull * S;
        for (int i = 0; i < npiece; ++i) {
            int item, sb, se;
            segment(nfull + i, item, sb, se);
            n += se - sb;
        }
        return n;
    }
    __device__ __forceinline__ int segments() const { return nseg; }
    // segment k: item and its stages [sb, se); k past the end repeats the last one
    __device__ __forceinline__ void segment(int k, int &item, int &sb, int &se) const {
        k = k < nseg ? k : nseg - 1;
        if (k < nfull) {
            item = first + k * stride;
            sb = 0;
            se = S;
        } else {
            const int u = pfirst + (k - nfull) * pstride;
            const int t = u / P;
            item = tail_first + t;
            sb = (u - t * P) * L;
            se = sb + L < S ? sb + L : S;
        }
    }
    // A walker over the sequence, one stage at a time.
    struct Cursor {
        int k, item, st, se;
    };
    __device__ __forceinline__ Cursor start() const {
        Cursor c{0, n_items, 0, 1};
        if (nseg > 0) {
            int sb;
            segment(0, c.item, sb, c.se);
            c.st = sb;
        }
        return c;
    }
    // next stage; past the end, an item that does not exist
    __device__ __forceinline__ void advance(Cursor &c) const {
        if (++c.st < c.se) return;
        if (++c.k < nseg) {
            int sb;
            segment(c.k, c.item, sb, c.se);
            c.st = sb;
        } else {
            c.item = n_items;
            c.st = 0;
            c.se = 1;
        }
    }
};

// Consumer of the persistent warp-specialised kernel: the workgroup's segments,
// as one continuous sequence of stages shared with the producers.
template <int M, int TB, int FS, int G, bool SPLIT, bool KM>
__device__ __forceinline__ void ws_consume(const floatx4 *lds, float *comb, unsigned *pairc, unsigned *ring,  // shared memory, written by other waves
                                           unsigned *skc,
                                           const floatx4 *__restrict__ wt, float *__restrict__ y,
                                           const Geometry &g, const WsSeq &sq, const WsSplit &sp,
                                           int n_inner, int kbl, int lane, int vec, bool ystream) {
    constexpr int T = M + 2, F4 = freq_quads<M>();
    constexpr int R = 16 * TB, CC = 256 / R, SS = CC / 4, BUF = F4 * CC * R;
    constexpr int NSLOT = ws_slots<M>();
    constexpr GroupF4<M, FS, G> gm{};
    constexpr int NF4 = gm.N;  // float4s of frequencies this wave multiplies
    constexpr int KBW = 4 / FS;
    constexpr int MM = M * M;
    constexpr int MMP = (MM + 3) / 4 * 4;  // output tile padded to whole float4s
    constexpr unsigned ROWS = group_rows<M, FS, G>();
    static_assert(FS == 1 || T >= 7, "frequency split is built for F(5) and F(6)");
    static_assert(gm.whole() && rows_pair_closed<M, ROWS>(), "groups split on float4 and pair bounds");
    const long long HW = (long long)g.H * g.W;
    const int32x4 yrs = make_rsrc(y, (unsigned)((long long)g.N * g.K * HW * 4));
    const unsigned hwb = (unsigned)(HW * 4), rowb = (unsigned)g.W * 4u;

    static_assert(SS % 2 == 0, "channel steps are processed in pairs");
    // Kernel operands alternate between two register sets over channel steps (set
    // a for even steps, b for odd ones): the loads of step u+1 are issued before
    // the products of step u.  Every stage runs all SS steps: channels past C hold
    // zero input tiles in LDS (and their operand indices are clamped to the last
    // step), so a segment's step sequence has an even length and the loads past
    // its end fetch the next segment's first steps, which arrive during the
    // epilogue.  The loads are unconditional, so that the wait for an operand never
    // has to include loads issued after it.
    // Operands are read with buffer loads: the lane's offset in a VGPR, the
    // (uniform) offset of a step of the wave's output block in an SGPR.
    kbl = __builtin_amdgcn_readfirstlane(kbl);
    constexpr unsigned SB = F4 * 1024u;  // bytes of one channel step of one output block
    const int32x4 wrs = make_rsrc(reinterpret_cast<const float *>(wt),
                                  (unsigned)g.Kb_alloc * (unsigned)g.Cs * SB);
    const unsigned vo = (unsigned)lane * 16u;
    // partial outputs of a contributor: [kbl][t][v][lane][element] floats, so a
    // lane's output tile is contiguous (16-byte accesses)
    const unsigned vlane = (unsigned)lane * MMP * 4u;
    auto poff = [&](int t, int v) { return (unsigned)((((kbl * TB + t) * 4 + v) * 64) * MMP) * 4u; };
    auto wbase = [&](int it) { return (unsigned)((item_kgroup<KM>(it, n_inner) * KBW + kbl) * g.Cs) * SB; };
    auto wload = [&](unsigned soff, int lf) { return buffer_load_f32x4(wrs, vo, soff + gm.f4[lf] * 1024u, 0); };
    const int last = g.Cs - 1;
    const int nseg = sq.segments();
    floatx4 wa[NF4], wb[NF4];
    int item = 0, sb = 0, se = 0;
    if (nseg > 0) {
        sq.segment(0, item, sb, se);
        const unsigned c0 = (unsigned)(sb * SS < last ? sb * SS : last);
#pragma unroll
        for (int lf = 0; lf < NF4; ++lf) wa[lf] = wload(wbase(item) + c0 * SB, lf);
    }

    int q = 0;  // position in the stage sequence (selects the LDS buffer)
    unsigned seq = 0;  // partial tiles exchanged so far by this wave pair (FS = 2)
    unsigned nsk = 0;  // partial-output epilogues so far
    int slot = 0;      // LDS buffer of stage q
    unsigned gen = 0;  // fillings of that buffer before stage q
    for (int k = 0; k < nseg; ++k) {
        if (k > 0) sq.segment(k, item, sb, se);
        int item2, sb2, se2;
        sq.segment(k + 1, item2, sb2, se2);
        const int nsteps = (se - sb) * SS;
        const unsigned bk = wbase(item), bn = wbase(item2);
        // operands of step u of this segment (u >= nsteps: the next segment's)
        auto wsrc = [&](int u) {
            const bool cur = u < nsteps;
            int c = cur ? sb * SS + u : sb2 * SS + (u - nsteps);
            c = c < last ? c : last;
            return (cur ? bk : bn) + (unsigned)c * SB;
        };

        floatx4 acc[TB][NF4 * 4];
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
            for (int f = 0; f < NF4 * 4; ++f) acc[t][f] = floatx4{0.f, 0.f, 0.f, 0.f};

        // products of one channel step: operands w, transformed tiles from LDS step s
        auto step = [&](const floatx4 (&w)[NF4], const floatx4 *cur, int s) {
            const floatx4 *bp = cur + (4 * s + (lane >> 4)) * R + (lane & 15);
#pragma unroll
            for (int lf = 0; lf < NF4; ++lf) {
#pragma unroll
                for (int t = 0; t < TB; ++t) {
                    const floatx4 b = bp[gm.f4[lf] * CC * R + t * 16];
#pragma unroll
                    for (int qq = 0; qq < 4; ++qq)
                        acc[t][4 * lf + qq] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            w[lf][qq], b[qq], acc[t][4 * lf + qq], 0, 0, 0);
                }
            }
        };
        auto load_w = [&](floatx4 (&w)[NF4], unsigned src) {
#pragma unroll
            for (int lf = 0; lf < NF4; ++lf) w[lf] = wload(src, lf);
        };
        for (int j = 0; j < se - sb; ++j, ++q) {
            wait_at_least(ring + slot, 4u * (gen + 1));  // the producers have filled it
            const floatx4 *cur = lds + slot * BUF;
#pragma unroll
            for (int s = 0; s < SS; s += 2) {
                const int u = j * SS + s;
                load_w(wb, wsrc(u + 1));
                __builtin_amdgcn_sched_barrier(0);
                step(wa, cur, s);
                load_w(wa, wsrc(u + 2));
                __builtin_amdgcn_sched_barrier(0);
                step(wb, cur, s + 1);
            }
            signal_wave(ring + NSLOT + slot);  // drained
            if (++slot == NSLOT) {
                slot = 0;
                ++gen;
            }
        }

        // Output transform Y = A^T Mm A per (output channel, tile), clipped to H x W,
        // into yy; emit(t, v, k, ti, yy) consumes each finished output tile.
        const int tile0 = item_tgroup<KM>(item, n_inner) * R;
        const int kb = item_kgroup<KM>(item, n_inner) * KBW + kbl;
        auto out_tiles = [&](auto emit) {
#pragma unroll
            for (int t = 0; t < TB; ++t) {
                const TileIdx ti = decode_tile(g, tile0 + t * 16 + (lane & 15));
                // P = Mm A, one transform-domain row i at a time for the lane's four
                // output channels, so the accumulators of a row are dead once it is done
                float pm[4][T][M];  // [v][i][c]; rows outside ROWS are not used
#pragma unroll
                for (int i = 0; i < T; ++i) {
                    if (!((ROWS >> i) & 1u)) continue;
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        float row[T];
#pragma unroll
                        for (int jj = 0; jj < T; ++jj) row[jj] = acc[t][gm.index(i * T + jj)][v];
                        at_1d<M, 1, 1>(row, pm[v][i]);
                    }
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    // Y = A^T P, column by column
                    float yy[MM];
#pragma unroll
                    for (int c = 0; c < M; ++c) at_1d_rows<M, M, M, ROWS>(&pm[v][0][c], yy + c);
                    if constexpr (FS == 2) {
                        float *cslot = comb + (long long)kbl * MM * 64 + lane;
                        unsigned *written = pairc + 2 * kbl, *read = pairc + 2 * kbl + 1;
                        if constexpr (G == 1) {
                            wait_counter(read, seq);  // the slot's previous partial has been read
#pragma unroll
                            for (int e = 0; e < MM; ++e) cslot[e * 64] = yy[e];
                            __hip_atomic_store(written, seq + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
                        } else {
                            wait_counter(written, seq + 1);
#pragma unroll
                            for (int e = 0; e < MM; ++e) yy[e] += cslot[e * 64];
                            __hip_atomic_store(read, seq + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
                        }
                        ++seq;
                    }
                    if constexpr (G == 0) emit(t, v, kb * 16 + (lane >> 4) * 4 + v, ti, yy);
                }
            }
        };
        // Whole tiles: buffer stores at the byte offset of output channel k_out - v
        // (per lane, y is below 2^31 bytes) plus v planes (scalar).
        auto store = [&](const TileIdx &ti, int k_out, int v, const float *yy, bool whole) {
            if (whole) {
                const unsigned vb = (unsigned)((((long long)ti.n * g.K + (k_out - v)) * HW +
                                                (long long)ti.ty * M * g.W + ti.tx * M) * 4);
                if (ystream)
                    store_rows_buf<M, true>(yrs, vb, (unsigned)v * hwb, rowb, yy);
                else
                    store_rows_buf<M, false>(yrs, vb, (unsigned)v * hwb, rowb, yy);
            } else if (ti.ok && k_out < g.K)
                store_tile<M>(y + ((long long)ti.n * g.K + k_out) * HW, yy, ti.ty * M, ti.tx * M, g, vec != 0);
        };
        // When every tile of the wave lies wholly inside the image and all 16 output
        // channels of the block exist (a wave-uniform test), rows are stored unclipped.
        auto whole_of = [&](const TileIdx &ti) {
            const bool inside = ti.ok && ti.ty * M + M <= g.H && ti.tx * M + M <= g.W;
            return vec != 0 && (kb + 1) * 16 <= g.K && __builtin_amdgcn_ballot_w64(!inside) == 0;
        };
        // the last contributor of a split item: y = sum of the partials in order
        auto sum_partials = [&](const float *pbase_, int ncontrib_) {
            const int32x4 all = make_rsrc_uniform(pbase_, (unsigned)(ncontrib_ * sp.part_floats) * 4u);
            for (int t = 0; t < TB; ++t) {
                const TileIdx ti = decode_tile(g, tile0 + t * 16 + (lane & 15));
                const bool whole = whole_of(ti);
                for (int v = 0; v < 4; ++v) {
                    float yy[MMP];
#pragma unroll
                    for (int e = 0; e < MMP; ++e) yy[e] = 0.0f;
                    // CH contributors' partials are loaded before any is added (one
                    // memory round trip per CH contributors); the additions keep
                    // contributor order
                    constexpr int CH = MMP >= 28 ? 2 : 4;
                    for (int jc0 = 0; jc0 < ncontrib_; jc0 += CH) {
                        floatx4 pv[CH][MMP / 4];
#pragma unroll
                        for (int c = 0; c < CH; ++c) {
                            const int jc = jc0 + c < ncontrib_ ? jc0 + c : ncontrib_ - 1;
                            const unsigned o = (unsigned)(jc * sp.part_floats) * 4u + poff(t, v);
#pragma unroll
                            for (int e = 0; e < MMP / 4; ++e) pv[c][e] = buffer_load_f32x4(all, vlane, o + e * 16u, kDeviceCoherent);
                        }
#pragma unroll
                        for (int c = 0; c < CH; ++c) {
                            if (jc0 + c < ncontrib_) {
#pragma unroll
                                for (int e = 0; e < MM; ++e) yy[e] += pv[c][e / 4][e % 4];
                            }
                        }
                    }
                    store(ti, kb * 16 + (lane >> 4) * 4 + v, v, yy, whole);
                }
            }
        };
        // A segment that covers only part of its item's stages yields a partial
        // output (Sec. 3: the output transform is linear, so partial sums over
        // channels can be inverse-transformed separately and added).  Each
        // contributor writes its partial; the one that arrives last adds all
        // partials in contributor order (a fixed order, so the result is
        // reproducible) and stores y.  Partials are written and read with
        // device-coherent accesses; a writer's stores have completed before its
        // arrival is counted.
        const bool partial = SPLIT && !(sb == 0 && se == sq.S);
        const unsigned t_split = (unsigned)__builtin_amdgcn_readfirstlane(item - sp.tail_first);
        int ncontrib = 0;
        const float *pbase = sp.part;
        int32x4 mine{};
        if (partial) {
            // contributor index: the piece's position in stage order
            ncontrib = sq.P;
            pbase = sp.part + (long long)t_split * sq.P * sp.part_floats;
            mine = make_rsrc_uniform(pbase + (long long)(sb / sq.L) * sp.part_floats,
                                     (unsigned)sp.part_floats * 4u);
        }
        out_tiles([&](int t, int v, int k_out, const TileIdx &ti, const float *yy) {
            if (!partial) {
                store(ti, k_out, v, yy, whole_of(ti));
            } else {
#pragma unroll
                for (int e = 0; e < MMP; e += 4)
                    buffer_store_f32x4(floatx4{yy[e], e + 1 < MM ? yy[e + 1] : 0.0f, e + 2 < MM ? yy[e + 2] : 0.0f,
                                               e + 3 < MM ? yy[e + 3] : 0.0f},
                                       mine, vlane, poff(t, v) + e * 4u, kDeviceCoherent);
            }
        });
        if (partial) {
            if constexpr (G == 0) {
                unsigned *written = skc, *decided = skc + 1, *flag = skc + 2;
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's partial is stored
                signal_wave(written);
                if (kbl == 0) {
                    wait_at_least(written, (unsigned)KBW * (nsk + 1));
                    if (lane == 0) {
                        const unsigned old = __hip_atomic_fetch_add(sp.cnt + t_split, 1u, __ATOMIC_RELAXED,
                                                                    __HIP_MEMORY_SCOPE_AGENT);
                        const unsigned is_last = (old + 1 == (unsigned)ncontrib) ? 1u : 0u;
                        if (is_last) __hip_atomic_store(sp.cnt + t_split, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        flag[nsk & 1u] = is_last;
                    }
                    signal_wave(decided);
                }
                wait_at_least(decided, nsk + 1);
                if (__builtin_amdgcn_readfirstlane(flag[nsk & 1u]) != 0) sum_partials(pbase, ncontrib);
            }
            ++nsk;
        }

        // next segment's first operands are in wa (loaded as step nsteps)
    }
}

// Persistent warp-specialised fused kernel: one workgroup per compute unit
// (register and LDS use allow one).  Items (tile group, output-channel group)
// are numbered with the output-channel group fastest; the whole items of a
// workgroup come from one contiguous range per XCD, taken round-robin by its
// workgroups, so at any time the workgroups of an XCD work on neighbouring items:
// the groups that re-read one tile group's input, and the tile groups whose input
// tiles share halo rows and columns, find those in the XCD's L2.  The remaining
// items are split stage-wise across all workgroups (WsSeq).  Each workgroup runs
// its stages as one sequence, so the next item's first input tiles load and
// transform while the consumers finish the current item's output transform and
// stores.
template <int M, int TB, int FS, bool VX, bool SPLIT, bool KM>
__global__ void __launch_bounds__(512) fused_ws_kernel(const float *__restrict__ x,
                                                       const floatx4 *__restrict__ wt,
                                                       float *__restrict__ y, Geometry g, int vec,
                                                       int n_inner, int n_items, WsSplit sp, int ystream) {
    constexpr int T = M + 2, T2 = T * T, F4 = freq_quads<M>();
    constexpr int R = 16 * TB;
    constexpr int CC = 256 / R;
    constexpr int BUF = F4 * CC * R;
    constexpr int NSLOT = ws_slots<M>();
    // float4s of the combine slots and the pair counters (FS = 2)
    constexpr int COMB = FS == 1 ? 0 : 2 * M * M * 64 / 4 + 1;
    constexpr int NCNT = 2 * NSLOT + 4;        // ring counters, then split-output counters
    constexpr int RING = (NCNT + 3) / 4;        // float4s of the counters
    __shared__ floatx4 lds[NSLOT * BUF + COMB + RING];
    float *comb = reinterpret_cast<float *>(lds + NSLOT * BUF);
    unsigned *pairc = FS == 2 ? reinterpret_cast<unsigned *>(comb + 2 * M * M * 64) : nullptr;
    unsigned *ring = reinterpret_cast<unsigned *>(lds + NSLOT * BUF + COMB);  // fill counts, then drain counts
    unsigned *skc = ring + 2 * NSLOT;  // split outputs: written, decided, flag[2]

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    if (tid < NCNT) ring[tid] = 0u;
    if (FS == 2 && tid >= 64 && tid < 68) pairc[tid - 64] = 0u;
    __syncthreads();
    const long long HW = (long long)g.H * g.W;
    const int stages = (g.C + CC - 1) / CC;
    WsSeq sq;
    sq.init(sp, n_items, stages, SPLIT);
    const int nrounds = sq.length();  // stages this workgroup processes

    if (wave >= 4) {
        // ---------------- producer: load + input transform -> LDS ----------------
        const int pt = tid - 256;
        const int tr = pt % R;
        const int cl = pt / R;
        // VX: row-vector loads with DPP halo exchange; otherwise one load per element
        using Loader = typename std::conditional<VX, RowTile<M>, BufTile<M, (M <= 2)>>::type;
        Loader ld;
        int cur_item = -1;
        // cursors of the stage being loaded (PD ahead) and of the stage transformed
        WsSeq::Cursor cl_load = sq.start(), cl_proc = sq.start();
        const bool maskcols = (g.W % M) != 0;
        const unsigned xbytes = (unsigned)((long long)g.N * g.C * HW * 4);
        const bool ctail = (g.C % CC) != 0;
        // load the next stage of the sequence (its item's tiles are located when the
        // item changes)
        auto load_stage = [&](float *d, unsigned &fl) {
            const int it = cl_load.item, st = cl_load.st;
            sq.advance(cl_load);
            if (it != cur_item) {
                cur_item = it;
                const int t0 = item_tgroup<KM>(it, n_inner) * R;
                const TileIdx ti = decode_tile(g, t0 + tr);
                if constexpr (VX) {
                    TileIdx rf, rl;
                    row_edges<TB>(g, t0, tr, rf, rl);
                    ld.init(g, ti, rf, rl, cl, lane & 15);
                } else {
                    ld.init(g, ti, cl);
                }
            }
            const long long cbase = (long long)st * CC * HW;
            const int32x4 rs = make_rsrc(x + cbase, xbytes - (unsigned)(cbase * 4));
            if constexpr (VX) {
                ld.issue(rs, d);
                fl = ld.flags();
            } else {
                ld.load(rs, d);
            }
        };
        // round r: issue the loads of stage r+PD, wait until buffer r % NSLOT is
        // drained, finish and transform stage r into it, and count it filled.
        // PD = 2 (three rotating register sets) keeps two stages of input loads in
        // flight where registers allow (m <= 4), else PD = 1.
        constexpr int PD = (M <= 4) ? 2 : 1;
        // The loads of round r + PD are issued unconditionally (past the last stage
        // they address tiles outside every image: no memory access), so that the
        // wait for a stage's data never has to cover loads issued after it.
        auto round = [&](int r, float *dcur, unsigned fcur, float *dnext, unsigned &fnext) {
            load_stage(dnext, fnext);
            if (r < nrounds) {
                const int slot = r % NSLOT;
                const unsigned gen = (unsigned)(r / NSLOT);
                if constexpr (VX) RowTile<M>::finish(dcur, fcur, maskcols);
                if (gen > 0) wait_at_least(ring + NSLOT + slot, 4u * gen);
                const int st = cl_proc.st;
                sq.advance(cl_proc);
                // channels past C (last stage only, when C % CC != 0) transform zeros
                if (ctail && st == stages - 1) {
                    asm volatile("");  // keeps this a branch instead of selects run every stage
                    if (st * CC + cl >= g.C) {
#pragma unroll
                        for (int f = 0; f < T2; ++f) dcur[f] = 0.0f;
                    }
                }
                floatx4 *buf = lds + slot * BUF + cl * R + tr;
                input_tile_transform_emit<M>(dcur, [&](int f4, float a, float b, float c, float e) {
                    buf[f4 * CC * R] = floatx4{a, b, c, e};
                });
                signal_wave(ring + slot);
            }
        };
        int r = 0;
        if constexpr (PD == 1) {
            float d0[T2], d1[T2];
            unsigned f0 = 0, f1 = 0;
            load_stage(d0, f0);
            for (; r + 1 < nrounds; r += 2) {
                round(r, d0, f0, d1, f1);
                round(r + 1, d1, f1, d0, f0);
            }
            if (r < nrounds) round(r, d0, f0, d1, f1);
        } else {
            float d0[T2], d1[T2], d2[T2];
            unsigned f0 = 0, f1 = 0, f2 = 0;
            load_stage(d0, f0);
            load_stage(d1, f1);
            for (; r + 2 < nrounds; r += 3) {
                round(r, d0, f0, d2, f2);
                round(r + 1, d1, f1, d0, f0);
                round(r + 2, d2, f2, d1, f1);
            }
            if (r < nrounds) round(r, d0, f0, d2, f2);
            if (r + 1 < nrounds) round(r + 1, d1, f1, d0, f0);
        }
        return;
    }

    // ---------------- consumers ----------------
    const int kbl = wave / FS;
    if constexpr (FS == 1) {
        ws_consume<M, TB, 1, 0, SPLIT, KM>(lds, comb, pairc, ring, skc, wt, y, g, sq, sp, n_inner, kbl, lane, vec, ystream != 0);
    } else {
        if ((wave % FS) == 0) ws_consume<M, TB, FS, 0, SPLIT, KM>(lds, comb, pairc, ring, skc, wt, y, g, sq, sp, n_inner, kbl, lane, vec, ystream != 0);
        else ws_consume<M, TB, FS, 1, SPLIT, KM>(lds, comb, pairc, ring, skc, wt, y, g, sq, sp, n_inner, kbl, lane, vec, ystream != 0);
    }
}

// ---------------------------------------------------------------------------
// Persistent fused kernel, one wave per SIMD.  On this GPU the matrix cores'
// fp32 products and the vector ALU's fp32 arithmetic do not run concurrently on
// one SIMD, so dedicating waves to the input transform gains no overlap; it
// only halves the registers of the wave that holds the accumulators.  Here the
// four waves of a workgroup each do both jobs with the full register file, which
// allows R = 16*TB = 32 (F(4)) or 64 (F(2)) tiles per item: twice or four times
// the reuse of every transformed-kernel operand read from L2.
//
// A stage is CC = 8 channels.  In stage q every wave (1) multiplies the input
// tiles of stage q (LDS buffer q&1) by its output block's kernel operands, two
// 4-channel steps with ping-pong operand registers as in ws_consume, (2) finishes
// and transforms its NT tile-channels of stage q+1, whose loads were issued one
// stage earlier, into the other buffer, (3) issues the loads of stage q+2, and
// (4) meets the others at the one barrier of the stage.  The stages of all the
// workgroup's items form one sequence, so the input of an item's first stage is
// transformed during the previous item's last stage.  Items are as in
// fused_ws_kernel; the accumulators of TB tile blocks x T^2 frequencies stay in
// registers until the output transform.
template <int M, int TB, bool VX>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
fused_1w_kernel(const float *__restrict__ x, const floatx4 *__restrict__ wt, float *__restrict__ y,
                Geometry g, int vec, int n_kgroups, int n_items) {
    constexpr int T = M + 2, T2 = T * T, F4 = T2 / 4;
    constexpr int R = 16 * TB, CC = 8, SS = CC / 4, NT = R * CC / 256;
    constexpr int BUF = F4 * CC * R;
    static_assert(NT >= 1 && R * CC == 256 * NT, "whole tile-channels per lane");
    static_assert(SS == 2, "one pair of channel steps per stage");
    __shared__ floatx4 lds[2 * BUF];

    // An (empty) use of an accumulation register: the compiler then keeps the
    // matrix-core accumulators in the accumulation registers rather than in the
    // vector registers the transforms need.
    asm volatile("" ::: "a0");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ItemRange ir = item_range(n_items);
    const long long HW = (long long)g.H * g.W;
    const int stages = (g.C + CC - 1) / CC;

    // ---- input role: the lane's NT (tile, channel) pairs of a stage ----
    using Loader = typename std::conditional<VX, RowTile<M>, BufTile<M, (M <= 2)>>::type;
    Loader ld[NT];
    int tr[NT], cl[NT];
#pragma unroll
    for (int n = 0; n < NT; ++n) {
        tr[n] = (tid + 256 * n) % R;
        cl[n] = (tid + 256 * n) / R;
    }
    const bool maskcols = (g.W % M) != 0;
    const unsigned xbytes = (unsigned)((long long)g.N * g.C * HW * 4);
    const bool ctail = (g.C % CC) != 0;
    float xd[NT][T2];
    unsigned xf[NT];
    // Issue the loads of stage q of the sequence (item ir.first + (q / stages) *
    // ir.stride, channel stage q % stages).  Unconditional: past the sequence the
    // tiles are those of later items, or outside the image (no memory access).
    auto issue = [&](int q) {
        const int st = q % stages;
        if (st == 0) {
            const int it = ir.first + (q / stages) * ir.stride;
#pragma unroll
            for (int n = 0; n < NT; ++n) {
                const int t0 = (it / n_kgroups) * R;
                const TileIdx ti = decode_tile(g, t0 + tr[n]);
                if constexpr (VX) {
                    TileIdx rf, rl;
                    row_edges<TB>(g, t0, tr[n], rf, rl);
                    ld[n].init(g, ti, rf, rl, cl[n], lane & 15);
                } else {
                    ld[n].init(g, ti, cl[n]);
                }
            }
        }
        const long long cbase = (long long)st * CC * HW;
        const int32x4 rs = make_rsrc(x + cbase, xbytes - (unsigned)(cbase * 4));
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            if constexpr (VX) {
                ld[n].issue(rs, xd[n]);
                xf[n] = ld[n].flags();
            } else {
                ld[n].load(rs, xd[n]);
            }
        }
    };
    // B^T d B of the lane's tiles of stage q into LDS buffer buf
    auto transform = [&](int q, floatx4 *buf) {
        const int st = q % stages;
#pragma unroll
        for (int n = 0; n < NT; ++n) {
            if constexpr (VX) RowTile<M>::finish(xd[n], xf[n], maskcols);
            // channels past C (last stage only, when C % CC != 0) transform zeros
            if (ctail && st == stages - 1) {
                asm volatile("");  // keeps this a branch instead of selects run every stage
                if (st * CC + cl[n] >= g.C) {
#pragma unroll
                    for (int f = 0; f < T2; ++f) xd[n][f] = 0.0f;
                }
            }
            floatx4 *b = buf + cl[n] * R + tr[n];
            input_tile_transform_emit<M>(xd[n], [&](int f4, float a, float bb, float c, float e) {
                b[f4 * CC * R] = floatx4{a, bb, c, e};
            });
        }
    };

    // ---- matrix role: the wave's output block of the item's group ----
    constexpr unsigned SB = F4 * 1024u;  // bytes of one channel step of one output block
    const int32x4 wrs = make_rsrc(reinterpret_cast<const float *>(wt),
                                  (unsigned)g.Kb_alloc * (unsigned)g.Cs * SB);
    const unsigned vo = (unsigned)lane * 16u;
    auto wbase = [&](int it) { return (unsigned)(((it % n_kgroups) * 4 + wave) * g.Cs) * SB; };
    auto wload = [&](unsigned soff, int f4) { return buffer_load_f32x4(wrs, vo, soff + (unsigned)f4 * 1024u, 0); };
    auto load_w = [&](floatx4 (&w)[F4], unsigned src) {
#pragma unroll
        for (int f4 = 0; f4 < F4; ++f4) w[f4] = wload(src, f4);
    };
    const int last = g.Cs - 1, nsteps = stages * SS;
    floatx4 wa[F4], wb[F4];

    // prologue: stage 0 into buffer 0, the loads of stage 1 in flight
    issue(0);
    transform(0, lds);
    issue(1);
    if (ir.count > 0) load_w(wa, wbase(ir.first));
    __syncthreads();

    int q = 0;  // position in the stage sequence
    for (int i = 0; i < ir.count; ++i) {
        const int it = ir.first + i * ir.stride;
        const int tile0 = (it / n_kgroups) * R;
        const int kb = (it % n_kgroups) * 4 + wave;
        const unsigned bk = wbase(it), bn = wbase(i + 1 < ir.count ? it + ir.stride : it);
        // operands of step u of this item's sequence (u >= nsteps: the next item's)
        auto wsrc = [&](int u) {
            const unsigned base = u < nsteps ? bk : bn;
            u = u < nsteps ? u : u - nsteps;
            u = u < last ? u : last;
            return base + (unsigned)u * SB;
        };

        floatx4 acc[TB][T2];
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
            for (int f = 0; f < T2; ++f) acc[t][f] = floatx4{0.f, 0.f, 0.f, 0.f};

        // products of one channel step: operands w, transformed tiles of LDS step s
        auto step = [&](const floatx4 (&w)[F4], const floatx4 *cur, int s) {
            const floatx4 *bp = cur + (4 * s + (lane >> 4)) * R + (lane & 15);
#pragma unroll
            for (int f4 = 0; f4 < F4; ++f4) {
#pragma unroll
                for (int t = 0; t < TB; ++t) {
                    const floatx4 b = bp[f4 * CC * R + t * 16];
#pragma unroll
                    for (int qq = 0; qq < 4; ++qq)
                        acc[t][4 * f4 + qq] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                            w[f4][qq], b[qq], acc[t][4 * f4 + qq], 0, 0, 0);
                }
            }
        };
        for (int j = 0; j < stages; ++j, ++q) {
            const floatx4 *cur = lds + (q & 1) * BUF;
            const int u = j * SS;
            load_w(wb, wsrc(u + 1));
            __builtin_amdgcn_sched_barrier(0);
            step(wa, cur, 0);
            load_w(wa, wsrc(u + 2));
            __builtin_amdgcn_sched_barrier(0);
            step(wb, cur, 1);
            __builtin_amdgcn_sched_barrier(0);
            transform(q + 1, lds + ((q + 1) & 1) * BUF);
            issue(q + 2);
            __syncthreads();
        }

        // Output transform Y = A^T Mm A per (output channel, tile), as in ws_consume.
#pragma unroll
        for (int t = 0; t < TB; ++t) {
            const TileIdx ti = decode_tile(g, tile0 + t * 16 + (lane & 15));
            const bool inside = ti.ok && ti.ty * M + M <= g.H && ti.tx * M + M <= g.W;
            const bool whole = vec != 0 && (kb + 1) * 16 <= g.K &&
                               __builtin_amdgcn_ballot_w64(!inside) == 0;
            float pm[4][T][M];  // P = Mm A, [v][i][c]
#pragma unroll
            for (int i2 = 0; i2 < T; ++i2) {
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float row[T];
#pragma unroll
                    for (int jj = 0; jj < T; ++jj) row[jj] = acc[t][i2 * T + jj][v];
                    at_1d<M, 1, 1>(row, pm[v][i2]);
                }
            }
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int k = kb * 16 + (lane >> 4) * 4 + v;
                float yy[M * M];
#pragma unroll
                for (int c = 0; c < M; ++c) at_1d<M, M, M>(&pm[v][0][c], yy + c);
                if (whole)
                    store_rows<M>(y + ((long long)ti.n * g.K + k) * HW + (long long)ti.ty * M * g.W + ti.tx * M,
                                  yy, g.W);
                else if (ti.ok && k < g.K)
                    store_tile<M>(y + ((long long)ti.n * g.K + k) * HW, yy, ti.ty * M, ti.tx * M, g, vec != 0);
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

hipError_t launch_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s) {
    const long long total = (long long)g.Kb_alloc * g.Cs * 64;
    dim3 block(256), grid((unsigned)((total + 255) / 256));
    WINO_DISPATCH_M(g.m, hipLaunchKernelGGL(weight_transform_kernel<MM>, grid, block, 0, s, w,
                                            reinterpret_cast<floatx4 *>(wt), g));
    return hipGetLastError();
}

bool fused_cfg_supported(int m, const FusedCfg &cfg) {
    if (m != 2 && m != 4 && m != 5 && m != 6) return false;
    if (cfg.schedule == kSchedSpecialised) return true;
    if (m == 5) return false;  // F(5) runs only the warp-specialised kernel
    if (cfg.schedule == kSchedPersistent) return m == 2;
    if (cfg.schedule == kSchedShared) return cfg.tb == 1 || (cfg.tb == 2 && m <= 4);
    if (cfg.schedule != kSchedPerWave) return false;
    if (cfg.waves < 1 || cfg.waves > 4) return false;
    switch (m) {
        case 2: return cfg.nkb == 1 || cfg.nkb == 2 || cfg.nkb == 4;
        case 4: return cfg.nkb == 1 || cfg.nkb == 2;
        default: return cfg.nkb == 1;
    }
}

FusedCfg fused_cfg_default(const Geometry &g) {
    FusedCfg c;
    c.schedule = kSchedSpecialised;
    c.num_cus = 256;  // replaced by the device's count at plan time
    c.tb = (g.m == 2) ? 2 : 1;
    c.waves = 4;
    c.csplit = 0;
    switch (g.m) {
        case 2: c.nkb = g.Kb >= 4 ? 4 : (g.Kb >= 2 ? 2 : 1); break;
        case 4: c.nkb = g.Kb >= 2 ? 2 : 1; break;
        default: c.nkb = 1; break;
    }
    return c;
}

// Split plan of the warp-specialised kernel (see WsSeq): grid size, whole items
// per workgroup, the split items and the partial-output buffer they need.
// csplit > 1 splits every item into that many channel pieces (at most one per
// stage); otherwise only a last, partly filled round may be split.
template <int M, int TB, int FS>
static SplitInfo ws_split_info(const Geometry &g, int num_cus, int csplit) {
    constexpr int R = 16 * TB, CC = 256 / R, KBW = 4 / FS;
    SplitInfo si{};
    const int n_tgroups = (g.ntiles + R - 1) / R;
    si.n_kgroups = (g.Kb + KBW - 1) / KBW;
    si.n_items = n_tgroups * si.n_kgroups;
    si.stages = (g.C + CC - 1) / CC;
    const int cus = num_cus < 1 ? 1 : num_cus;
    si.nfull = si.n_items / cus;
    si.grid = si.n_items < cus ? si.n_items : cus;
    si.part_floats = KBW * TB * 4 * ((M * M + 3) / 4 * 4) * 64;  // output tiles padded to float4s
    si.tail_first = si.n_items;  // every item whole unless split below
    si.n_tail = 0;
    si.n_units = 0;
    si.piece = si.stages;
    si.maxc = 0;
    if (csplit > 1 && si.stages > 1) {
        // every item in P pieces of L stages: L = ceil(stages / csplit), P =
        // ceil(stages / L) (P < csplit when csplit does not divide the stages)
        const int want = csplit < si.stages ? csplit : si.stages;
        const int L = (si.stages + want - 1) / want;
        const int P = (si.stages + L - 1) / L;
        si.nfull = 0;
        si.tail_first = 0;
        si.n_tail = si.n_items;
        si.piece = L;
        si.maxc = P;
        si.n_units = si.n_items * P;
        si.grid = si.n_units < cus ? si.n_units : cus;
        return si;
    }
    // Split the items of a last, partly filled round into P pieces (P <= 4,
    // dividing the stages) when at least half of the compute units would idle in
    // it otherwise.  A piece costs its workgroup a partial-output epilogue
    // (output transform, device-coherent stores, arrival count) and the last
    // contributor a sum, which keeps P small; with four or more full rounds the
    // imbalance is small and items stay whole.
    constexpr int kMaxPieces = 4, kMaxSplitRounds = 4;
    const int tail = si.n_items - si.nfull * cus;
    if (si.nfull >= kMaxSplitRounds || tail == 0 || 2 * tail > cus) return si;
    int P = cus / tail < kMaxPieces ? cus / tail : kMaxPieces;
    while (P > 1 && si.stages % P != 0) --P;
    if (P < 2) return si;
    si.tail_first = si.nfull * cus;
    si.n_tail = tail;
    si.piece = si.stages / P;
    si.n_units = tail * P;
    si.maxc = P;
    si.grid = si.nfull > 0 ? cus : tail * P;
    return si;
}

SplitInfo fused_split_info(const Geometry &g, const FusedCfg &cfg) {
    if (cfg.schedule != kSchedSpecialised) return SplitInfo{};
    switch (g.m) {
        case 2: return ws_split_info<2, 2, 1>(g, cfg.num_cus, cfg.csplit);
        case 4: return ws_split_info<4, 1, 1>(g, cfg.num_cus, cfg.csplit);
        case 5: return ws_split_info<5, 1, 2>(g, cfg.num_cus, cfg.csplit);
        default: return ws_split_info<6, 1, 2>(g, cfg.num_cus, cfg.csplit);
    }
}

template <int M, int TB, int FS>
static void launch_ws_t(const Geometry &g, const float *x, const float *wt, float *y, bool vec,
                        int num_cus, int csplit, const SplitBuffers &sb, hipStream_t s) {
    const SplitInfo si = ws_split_info<M, TB, FS>(g, num_cus, csplit);
    WsSplit sp;
    sp.n_whole = si.tail_first;
    sp.tail_first = si.tail_first;
    sp.n_units = si.n_units;
    sp.P = si.maxc;
    sp.piece = si.piece;
    sp.part = sb.part;
    sp.cnt = sb.cnt;
    sp.part_floats = si.part_floats;
    dim3 block(512), grid((unsigned)si.grid);
    // row-vector input loads need every row start aligned to the vector width
    // (m = 5: 4-byte aligned vector loads)
    const unsigned vw = (M == 4) ? 16u : (M == 5) ? 4u : 8u;
    const bool vx = (reinterpret_cast<uintptr_t>(x) % vw == 0) && ((unsigned)g.W * 4u) % vw == 0;
    // Item order: when the transformed kernels outweigh the input (deep layers),
    // the tile groups of one output-channel group are numbered adjacently, so the
    // workgroups of an XCD share that group's transformed kernels in L2.
    const bool km = si.n_kgroups > 1 &&
                    (double)g.T2 * g.C * g.K > (double)g.N * g.C * g.H * g.W;
    const int n_inner = km ? si.n_items / si.n_kgroups : si.n_kgroups;
    const int ystream = (long long)g.N * g.K * g.H * g.W * 4 >= kStreamOutputBytes ? 1 : 0;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, block, 0, s, x, reinterpret_cast<const floatx4 *>(wt), y, g, vec ? 1 : 0,
                           n_inner, si.n_items, sp, ystream);
    };
    // layers whose items all stay whole run an instantiation without the split path
    const bool split = si.n_tail > 0;
    if (vx) {
        if (split) km ? go(fused_ws_kernel<M, TB, FS, true, true, true>) : go(fused_ws_kernel<M, TB, FS, true, true, false>);
        else km ? go(fused_ws_kernel<M, TB, FS, true, false, true>) : go(fused_ws_kernel<M, TB, FS, true, false, false>);
    } else {
        if (split) km ? go(fused_ws_kernel<M, TB, FS, false, true, true>) : go(fused_ws_kernel<M, TB, FS, false, true, false>);
        else km ? go(fused_ws_kernel<M, TB, FS, false, false, true>) : go(fused_ws_kernel<M, TB, FS, false, false, false>);
    }
}

template <int M, int TB>
static void launch_1w_t(const Geometry &g, const float *x, const float *wt, float *y, bool vec,
                        int num_cus, hipStream_t s) {
    const int n_tgroups = (g.ntiles + 16 * TB - 1) / (16 * TB);
    const int n_kgroups = (g.Kb + 3) / 4;
    const int n_items = n_tgroups * n_kgroups;
    const int nwg = n_items < num_cus ? n_items : num_cus;
    dim3 block(256), grid((unsigned)nwg);
    const unsigned vw = (M == 4) ? 16u : 8u;
    const bool vx = (reinterpret_cast<uintptr_t>(x) % vw == 0) && ((unsigned)g.W * 4u) % vw == 0;
    if (vx)
        hipLaunchKernelGGL((fused_1w_kernel<M, TB, true>), grid, block, 0, s, x,
                           reinterpret_cast<const floatx4 *>(wt), y, g, vec ? 1 : 0, n_kgroups, n_items);
    else
        hipLaunchKernelGGL((fused_1w_kernel<M, TB, false>), grid, block, 0, s, x,
                           reinterpret_cast<const floatx4 *>(wt), y, g, vec ? 1 : 0, n_kgroups, n_items);
}

template <int M, int TB>
static void launch_shared_t(const Geometry &g, const float *x, const float *wt, float *y,
                            hipStream_t s) {
    dim3 block(256);
    dim3 grid((unsigned)((g.ntiles + 16 * TB - 1) / (16 * TB)), (unsigned)((g.Kb + 3) / 4));
    hipLaunchKernelGGL((fused_shared_kernel<M, TB>), grid, block, 0, s, x,
                       reinterpret_cast<const floatx4 *>(wt), y, g);
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
                        float *y, const SplitBuffers &sb, hipStream_t s) {
    if (!fused_cfg_supported(g.m, cfg)) return hipErrorInvalidValue;
    const uintptr_t ya = reinterpret_cast<uintptr_t>(y);
    // rows of whole tiles stored as vectors: 16-byte aligned for m = 4, 8-byte for m =
    // 2, 6; m = 5 uses buffer stores that need only 4-byte alignment
    const bool vec = (g.m == 5) ? true
                     : (g.m == 4) ? (g.W % 4 == 0 && ya % 16 == 0) : (g.W % 2 == 0 && ya % 8 == 0);
    if (cfg.schedule == kSchedPersistent) {
        launch_1w_t<2, 4>(g, x, wt, y, vec, cfg.num_cus, s);
        return hipGetLastError();
    }
    if (cfg.schedule == kSchedSpecialised) {
        switch (g.m) {
            case 2: launch_ws_t<2, 2, 1>(g, x, wt, y, vec, cfg.num_cus, cfg.csplit, sb, s); break;
            case 4: launch_ws_t<4, 1, 1>(g, x, wt, y, vec, cfg.num_cus, cfg.csplit, sb, s); break;
            case 5: launch_ws_t<5, 1, 2>(g, x, wt, y, vec, cfg.num_cus, cfg.csplit, sb, s); break;
            default: launch_ws_t<6, 1, 2>(g, x, wt, y, vec, cfg.num_cus, cfg.csplit, sb, s); break;
        }
        return hipGetLastError();
    }
    if (cfg.schedule == kSchedShared) {
        switch (g.m) {
            case 2:
                if (cfg.tb == 2) launch_shared_t<2, 2>(g, x, wt, y, s);
                else launch_shared_t<2, 1>(g, x, wt, y, s);
                break;
            case 4:
                if (cfg.tb == 2) launch_shared_t<4, 2>(g, x, wt, y, s);
                else launch_shared_t<4, 1>(g, x, wt, y, s);
                break;
            default:
                launch_shared_t<6, 1>(g, x, wt, y, s);
                break;
        }
        return hipGetLastError();
    }
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
        default:
            launch_fused_t<6, 1>(g, cfg.waves, x, wt, y, s);
            break;
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
