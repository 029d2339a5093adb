// Device-side building blocks shared by the Winograd kernels on gfx950: tile
// indexing, raw buffer loads and stores (range-checked, so reads outside a buffer
// return zero), the row-vector input-tile loader with its DPP halo exchange, and
// output-tile stores.
//
// Matrix-core mapping (v_mfma_f32_16x16x4_f32, one 64-lane wave):
//   D[16 x 16] += A[16 x 4] * B[4 x 16]
//   lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] and holds
//   D[4 * (l / 16) + v][l % 16], v = 0..3.
// Every product here is, for one frequency f, D[k][tile] += sum_c W'[f][c][k] U[f][c][tile]
// (Sec. 3, step 2), so A is a 16 (k) x 4 (c) slice of the transformed kernels and
// B a 4 (c) x 16 (tile) slice of the transformed input.
#pragma once

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

// Frequencies are grouped in float4s (four consecutive f) for the matrix-core
// operands; T^2 = 49 (F(5)) ends with a partial group padded with zeros.
template <int M>
constexpr int freq_quads() { return ((M + 2) * (M + 2) + 3) / 4; }

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

// Store one row of m output floats through a buffer resource over y: the row's
// first element at byte offset voff (per lane) + so (uniform).  STREAM: streaming
// (non-temporal) cache policy.
template <int M, bool STREAM>
__device__ __forceinline__ void store_row_buf(int32x4 yrs, unsigned voff, unsigned so, const float *r) {
    constexpr int kAux = STREAM ? kStream : 0;
    if constexpr (M == 4) {
        buffer_store_f32x4(floatx4{r[0], r[1], r[2], r[3]}, yrs, voff, so, kAux);
    } else if constexpr (M == 5) {  // 4-byte aligned vector store + one float
        buffer_store_f32x4(floatx4{r[0], r[1], r[2], r[3]}, yrs, voff, so, kAux);
        buffer_store_f32(r[4], yrs, voff + 16u, so, kAux);
    } else if constexpr (M == 7) {  // 4-byte aligned: 4 + 2 + 1 floats
        buffer_store_f32x4(floatx4{r[0], r[1], r[2], r[3]}, yrs, voff, so, kAux);
        buffer_store_f32x2(floatx2{r[4], r[5]}, yrs, voff + 16u, so, kAux);
        buffer_store_f32(r[6], yrs, voff + 24u, so, kAux);
    } else {
#pragma unroll
        for (int jj = 0; jj < M; jj += 2) buffer_store_f32x2(floatx2{r[jj], r[jj + 1]}, yrs, voff + 4u * jj, so, kAux);
    }
}

// Store one m x m output tile that lies wholly inside the image: its first element
// at byte offset voff (per lane) + soff (uniform), rows rowb bytes apart (uniform),
// so the per-row and per-channel steps are scalar adds.
template <int M, bool STREAM>
__device__ __forceinline__ void store_rows_buf(int32x4 yrs, unsigned voff, unsigned soff, unsigned rowb,
                                               const float *yy) {
#pragma unroll
    for (int i = 0; i < M; ++i) store_row_buf<M, STREAM>(yrs, voff, soff + (unsigned)i * rowb, yy + i * M);
}

// Store one m x m output tile of plane yp (clipped to H x W).  vec: rows may be
// written with m-float vector stores (16-byte aligned for m = 4, 8-byte for m = 2, 6;
// odd m always stores element by element here).
template <int M>
__device__ __forceinline__ void store_tile(float *__restrict__ yp, const float *yy, int h0, int w0,
                                           const Geometry &g, bool vec) {
#pragma unroll
    for (int i = 0; i < M; ++i) {
        const int h = h0 + i;
        if (h >= g.H) break;
        float *row = yp + (long long)h * g.W + w0;
        if (M % 2 == 0 && vec && w0 + M <= g.W) {
            if constexpr (M == 4) {
                *reinterpret_cast<floatx4 *>(row) =
                    floatx4{yy[i * M], yy[i * M + 1], yy[i * M + 2], yy[i * M + 3]};
            } else if constexpr (M % 2 == 0) {
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

}  // namespace wino
